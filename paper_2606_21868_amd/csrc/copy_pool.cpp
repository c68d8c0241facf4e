// A fixed set of host threads that split one memcpy between them.
#include "copy_pool.hpp"

#include <algorithm>
#include <cstring>

namespace wisp {

CopyPool::CopyPool(int threads) {
  // each worker is told the thread count: threads_ is still growing while the first workers run,
  // so a worker must not read its size (one that did could take a share computed for fewer
  // threads and leave part of a copy to nobody)
  threads_.reserve(static_cast<size_t>(threads));
  for (int i = 0; i < threads; ++i) threads_.emplace_back(&CopyPool::worker, this, i, threads);
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

void CopyPool::worker(int id, int n) {
  uint64_t seen = 0;
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

}  // namespace wisp
