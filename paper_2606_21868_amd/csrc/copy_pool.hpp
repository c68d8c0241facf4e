// A fixed set of host threads that split one memcpy between them (plain C++: the pageable-master
// staging uses it to fill its pinned bounce buffers).
#pragma once

#include <condition_variable>
#include <cstddef>
#include <cstdint>
#include <mutex>
#include <thread>
#include <vector>

namespace wisp {

class CopyPool {
 public:
  explicit CopyPool(int threads);
  ~CopyPool();
  CopyPool(const CopyPool&) = delete;
  CopyPool& operator=(const CopyPool&) = delete;
  void copy(void* dst, const void* src, size_t bytes);   // returns when the copy is complete

 private:
  void worker(int id, int n);   // n: the number of workers
  std::vector<std::thread> threads_;
  std::mutex mu_;
  std::condition_variable cv_, done_cv_;
  uint8_t* dst_ = nullptr;
  const uint8_t* src_ = nullptr;
  size_t bytes_ = 0;
  uint64_t generation_ = 0;
  int pending_ = 0;
  bool stop_ = false;
};

}  // namespace wisp
