// Host-only check of the staging copy pool: fresh pools (the window right after the worker threads
// start), each asked at once for copies of several sizes into a buffer that holds other bytes; every
// byte of every copy must arrive.  Prints "ok <copies>" or the first bad copy, and exits non-zero on
// a bad one.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "copy_pool.hpp"

int main(int argc, char** argv) {
  const int pools = argc > 1 ? std::atoi(argv[1]) : 200;
  const size_t sizes[] = {(9u << 20) + 4096, 9437184, 3u << 20, (1u << 20) + 12288};
  std::vector<uint8_t> src(10u << 20), dst(10u << 20);
  uint64_t x = 88172645463325252ull;
  for (auto& b : src) { x ^= x << 13; x ^= x >> 7; x ^= x << 17; b = static_cast<uint8_t>(x); }
  long copies = 0;
  for (int p = 0; p < pools; ++p) {
    wisp::CopyPool pool(1 + p % 8);
    for (size_t n : sizes) {
      std::memset(dst.data(), 0xA5 ^ p, dst.size());
      pool.copy(dst.data(), src.data(), n);
      ++copies;
      if (std::memcmp(dst.data(), src.data(), n) != 0) {
        size_t i = 0, j = n;
        while (i < n && dst[i] == src[i]) ++i;
        while (j > i && dst[j - 1] == src[j - 1]) --j;
        std::printf("bad copy: pool %d (%d threads), %zu bytes, bytes [%zu, %zu) differ\n", p, 1 + p % 8, n, i, j);
        return 1;
      }
    }
  }
  std::printf("ok %ld\n", copies);
  return 0;
}
