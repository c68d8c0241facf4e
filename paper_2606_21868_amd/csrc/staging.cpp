// Pageable-master staging: the pinned bounce ring.
#include "staging.hpp"

#include <algorithm>
#include <cstring>

namespace wisp {

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
    hipError_t e = hipHostMalloc(&p, kPieceBytes, hipHostMallocDefault);
    if (e != hipSuccess) return e;
    buf_[i] = static_cast<uint8_t*>(p);
    e = hipEventCreateWithFlags(&ev_[i], hipEventDisableTiming);
    if (e != hipSuccess) return e;
  }
  pool_ = new CopyPool(threads);
  return hipSuccess;
}

hipError_t BounceRing::copy_to_device(void* dst, const uint8_t* src, size_t bytes, hipStream_t st) {
  // the link is idle when no earlier piece's copy is still pending: then it waits for this copy's
  // first host copy, which is kept small; behind pending copies full pieces keep it busy
  bool idle = true;
  for (int i = 0; i < kBuffers && idle; ++i)
    if (used_[i] && hipEventQuery(ev_[i]) != hipSuccess) idle = false;
  size_t piece = idle ? kFirstPieceBytes : kPieceBytes;
  for (size_t off = 0; off < bytes; off += piece, piece = std::min(kPieceBytes, 2 * piece)) {
    const size_t n = std::min(piece, bytes - off);
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
