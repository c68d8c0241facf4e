// wisp_route_topk_noalloc: router scoring and top-k without a context and without allocating.
//
// The router kernels need device scratch beyond their inputs and outputs: the logits [T, N] fp32
// (up to kRouterMaxSplit partial sums of them for token batches) and, for the one-launch path of up
// to four tokens, the tagged logit words of the workgroups that publish logit rows.  Here that
// scratch is the file-scope array `scratch` below, of a fixed size, held by every device the library
// runs on until the process ends.  Host code never passes the array's name to a kernel (in host code it names a host-side stand-in); it passes the device
// address hipGetSymbolAddress returns for the current device, looked up once per device.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <string>

#include "errors.hpp"
#include "kernels.hpp"
#include "wisp.h"

namespace {

constexpr size_t kTagBytes = 4 * 256 * 8;                   // tagged logit words of the one-launch path
// logits [T, N] fp32 of the two-launch path, as up to kRouterMaxSplit partial sums
constexpr size_t kLogitBytes = static_cast<size_t>(wisp::kRouterMaxSplit) * WISP_NOALLOC_MAX_LOGITS * 4;
constexpr size_t kScratchBytes = kTagBytes + kLogitBytes;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::atomic<uint8_t*> g_scratch_dev[kMaxDevices];
std::atomic<uint32_t> g_tag[kMaxDevices];   // tag of the last one-launch router kernel per device
std::mutex g_init;

__global__ void clear_words_kernel(uint32_t* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0u;
}

// The device address of `scratch` on the current device (looked up, and its tag words cleared, on the
// first call on that device).
wisp_status scratch_on_device(hipStream_t st, uint8_t** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return wisp::set_error(WISP_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return wisp::set_error(WISP_E_INVAL, "device ordinal beyond 63");
  uint8_t* p = g_scratch_dev[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lk(g_init);
    p = g_scratch_dev[dev].load(std::memory_order_relaxed);
    if (!p) {
      void* q = nullptr;
      e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !q)
        return wisp::set_error(WISP_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
      p = static_cast<uint8_t*>(q);
      // the tag words must start at zero (tags are never 0); a kernel rather than a memset, so that a
      // caller capturing this stream records no memset node
      hipLaunchKernelGGL(clear_words_kernel, dim3(1), dim3(256), 0, st, reinterpret_cast<uint32_t*>(p),
                         static_cast<int>(kTagBytes / 4));
      e = hipGetLastError();
      if (e != hipSuccess) return wisp::set_error(WISP_E_HIP, std::string("tag clear: ") + hipGetErrorString(e));
      g_scratch_dev[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return WISP_OK;
}

}  // namespace

extern "C" wisp_status wisp_route_topk_noalloc(const float* w_r_dev, const void* x_dev, int32_t x_dtype, int32_t T,
                                               int32_t N, int32_t d, int32_t k, int32_t route, int32_t n_groups,
                                               int32_t topk_groups, int32_t* idx_dev, float* w_dev, void* stream) {
  using wisp::set_error;
  if (!w_r_dev || !x_dev || !idx_dev || !w_dev) return set_error(WISP_E_INVAL, "NULL device pointer");
  if (x_dtype != WISP_F32 && x_dtype != WISP_BF16) return set_error(WISP_E_INVAL, "x_dtype must be f32 or bf16");
  if (N < 1 || N > 256) return set_error(WISP_E_INVAL, "N must be in [1, 256]");
  if (k < 1 || k > 8 || k > N) return set_error(WISP_E_INVAL, "k must be in [1, min(8, N)]");
  if (route < 0 || route > 2) return set_error(WISP_E_INVAL, "unknown route");
  if (route == WISP_ROUTE_SIGMOID_GROUP) {
    if (n_groups < 1 || n_groups > 32 || N % n_groups) return set_error(WISP_E_INVAL, "n_groups must divide N, <= 32");
    if (topk_groups < 1 || topk_groups > n_groups || topk_groups * (N / n_groups) < k)
      return set_error(WISP_E_INVAL, "topk_groups too small for k");
  }
  if (d < 4 || d % 4) return set_error(WISP_E_INVAL, "d must be a positive multiple of 4");
  if (T < 1) return set_error(WISP_E_INVAL, "T must be >= 1");
  if (static_cast<int64_t>(T) * N > WISP_NOALLOC_MAX_LOGITS)
    return set_error(WISP_E_INVAL, "T * N exceeds the static scratch of wisp_route_topk_noalloc (524288 logits)");
  if (T > 8 && !(N % 16 == 0 && d % 16 == 0) && d % 32)
    return set_error(WISP_E_INVAL, "more than 8 tokens need d a multiple of 32");
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* base = nullptr;
  wisp_status s = scratch_on_device(st, &base);
  if (s != WISP_OK) return s;
  uint64_t* tagged = reinterpret_cast<uint64_t*>(base);
  float* logits = reinterpret_cast<float*>(base + kTagBytes);
  hipError_t e;
  if (T <= 4) {
    int dev = 0;
    (void)hipGetDevice(&dev);
    uint32_t tag = g_tag[dev].fetch_add(1, std::memory_order_relaxed) + 1;
    if (tag == 0) tag = g_tag[dev].fetch_add(1, std::memory_order_relaxed) + 1;
    e = wisp::launch_route_select(w_r_dev, x_dev, x_dtype, d, tagged, tag, T, N, k, route, n_groups,
                                  topk_groups, idx_dev, w_dev, nullptr, 0, st, wisp::LaunchTiming{});
  } else {
    int n_split = 1;
    e = wisp::launch_router_logits(w_r_dev, x_dev, x_dtype, T, N, d, logits, &n_split, st, wisp::LaunchTiming{});
    if (e == hipSuccess)
      e = wisp::launch_router_select(logits, n_split, T, N, k, route, n_groups, topk_groups, idx_dev, w_dev, nullptr, 0, st,
                                     wisp::LaunchTiming{});
  }
  if (e != hipSuccess) return set_error(WISP_E_HIP, std::string("router launch: ") + hipGetErrorString(e));
  return WISP_OK;
}
