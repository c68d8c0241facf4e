// Pageable-master staging: a memcpy thread pool and the pinned bounce ring.
#include "staging.hpp"

#include <algorithm>
#include <cstring>

namespace wisp {

CopyPool::CopyPool(int threads) {
  for (int i = 0; i < threads; ++i) threads_.emplace_back(&CopyPool::worker, this, i);
}

CopyPool::~CopyPool() {
  {
    std::lock_guard<std::mutex> lk(mu_);
    stop_ = true;
  }
  cv_.notify_all();
  for (auto& t : threads_) t.join();
}

void CopyPool::copy(void* dst, const void* src, size_t bytes) {
  if (threads_.empty() || bytes < (1u << 20)) {
    std::memcpy(dst, src, bytes);
    return;
  }
  std::unique_lock<std::mutex> lk(mu_);
  dst_ = static_cast<uint8_t*>(dst);
  src_ = static_cast<const uint8_t*>(src);
  bytes_ = bytes;
  pending_ = static_cast<int>(threads_.size());
  ++generation_;
  cv_.notify_all();
  done_cv_.wait(lk, [&] { return pending_ == 0; });
}

void CopyPool::worker(int id) {
  uint64_t seen = 0;
  const int n = static_cast<int>(threads_.size());
  for (;;) {
    uint8_t* dst;
    const uint8_t* src;
    size_t bytes;
    {
      std::unique_lock<std::mutex> lk(mu_);
      cv_.wait(lk, [&] { return stop_ || generation_ != seen; });
      if (stop_) return;
      seen = generation_;
      dst = dst_;
      src = src_;
      bytes = bytes_;
    }
    // contiguous share of this worker, in 4 KiB units
    const size_t pages = (bytes + 4095) / 4096;
    const size_t p0 = pages * id / n, p1 = pages * (id + 1) / n;
    const size_t b0 = std::min(bytes, p0 * 4096), b1 = std::min(bytes, p1 * 4096);
    if (b1 > b0) std::memcpy(dst + b0, src + b0, b1 - b0);
    {
      std::lock_guard<std::mutex> lk(mu_);
      if (--pending_ == 0) done_cv_.notify_all();
    }
  }
}

BounceRing::~BounceRing() {
  for (int i = 0; i < kBuffers; ++i) {
    if (used_[i] && ev_[i]) (void)hipEventSynchronize(ev_[i]);
    if (ev_[i]) (void)hipEventDestroy(ev_[i]);
    if (buf_[i]) (void)hipHostFree(buf_[i]);
  }
  delete pool_;
}

hipError_t BounceRing::init(int threads) {
  for (int i = 0; i < kBuffers; ++i) {
    void* p = nullptr;
    // coherent (snooped) pinned memory: the host threads write a piece with ordinary stores right
    // before the DMA engine reads it, so its reads must see the CPU caches
    hipError_t e = hipHostMalloc(&p, kPieceBytes, hipHostMallocCoherent);
    if (e != hipSuccess) return e;
    buf_[i] = static_cast<uint8_t*>(p);
    e = hipEventCreateWithFlags(&ev_[i], hipEventDisableTiming);
    if (e != hipSuccess) return e;
  }
  pool_ = new CopyPool(threads);
  return hipSuccess;
}

hipError_t BounceRing::copy_to_device(void* dst, const uint8_t* src, size_t bytes, hipStream_t st) {
  for (size_t off = 0; off < bytes; off += kPieceBytes) {
    const size_t n = std::min(kPieceBytes, bytes - off);
    const int b = next_;
    next_ = (next_ + 1) % kBuffers;
    if (used_[b]) {
      hipError_t e = hipEventSynchronize(ev_[b]);
      if (e != hipSuccess) return e;
    }
    pool_->copy(buf_[b], src + off, n);
    hipError_t e = hipMemcpyAsync(static_cast<uint8_t*>(dst) + off, buf_[b], n, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return e;
    e = hipEventRecord(ev_[b], st);
    if (e != hipSuccess) return e;
    used_[b] = true;
  }
  return hipSuccess;
}

}  // namespace wisp
