// Host->device copies out of pageable host memory, staged through a small pinned bounce ring.
//
// Expert masters normally live in pinned host memory and a fault is one DMA copy.  A machine may
// cap the pinned memory of a process below the size of the master set; the masters then live in
// ordinary pageable memory, and each copy goes piece by piece through pinned bounce buffers:
// host threads copy a piece into a free buffer, a DMA copy on the stream moves it to the device,
// and an event recorded after it frees the buffer again.  The host copy of the next piece overlaps
// the DMA of the previous ones.  A copy that finds the link idle starts with a small piece and
// doubles it up to the buffer size: the link waits for the host copy of the first piece only, so
// that piece is kept short.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "copy_pool.hpp"

namespace wisp {

class BounceRing {
 public:
  static constexpr size_t kPieceBytes = 32ull << 20;        // buffer size, the largest piece
  static constexpr size_t kFirstPieceBytes = 4ull << 20;     // the first piece of a copy from idle
  static constexpr int kBuffers = 4;
  BounceRing() = default;
  ~BounceRing();
  BounceRing(const BounceRing&) = delete;
  BounceRing& operator=(const BounceRing&) = delete;
  hipError_t init(int threads);   // pinned buffers, events and the copy threads
  // Enqueue dst[0, bytes) <- src[0, bytes) on `st`.  Blocks while every buffer still feeds a DMA
  // copy that has not run; all work those copies wait for must already be enqueued.
  hipError_t copy_to_device(void* dst, const uint8_t* src, size_t bytes, hipStream_t st);

 private:
  uint8_t* buf_[kBuffers] = {};
  hipEvent_t ev_[kBuffers] = {};
  bool used_[kBuffers] = {};
  int next_ = 0;
  CopyPool* pool_ = nullptr;
};

}  // namespace wisp
