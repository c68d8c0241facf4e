// Top-k expert selection of up to four tokens by one 256-thread workgroup, shared by the router
// kernel and the device pager kernel.
//
// Scores are kept in LDS as 64-bit keys (0 = not allowed).  Thread e computes the rank of expert
// e — how many allowed experts order before it on (logit desc, id asc) — as a count of larger
// keys over the token's LDS row, and the expert of rank j < k goes to slot j.  The logit orders
// experts exactly as softmax or sigmoid do (both are increasing) without ties introduced by
// rounding them.  Group-limited routing first scores each
// group by the sum of its two largest sigmoids and keeps the topk_groups best groups (score
// desc, group asc).  Gates: softmax over the chosen logits (equal to renormalising a softmax over
// all N) or the chosen sigmoids divided by their sum.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace wisp {

enum { R_SOFTMAX_RENORM = 0, R_TOPK_SOFTMAX = 1, R_SIGMOID_GROUP = 2 };

struct SelectShared {
  uint64_t key[4][256];   // (order-preserving logit << 32 | 255 - id), 0 = not allowed
  float z[4][256];
  float gam[4][32];
  int sel[4][8];
  float gate[4][8];
};

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float sel_sigmoid(float z) { return 1.0f / (1.0f + __expf(-z)); }

// Tokens t0 .. t0+3 (those < T) of logits [T, N]; all 256 threads must call it.  Thread e owns
// expert e of every token (N <= 256).  A key packs the order-preserving bits of the logit above
// 255 - id, so (logit desc, id asc) is plain unsigned order and every allowed key is distinct:
// the rank of an expert is the number of larger keys.  COHERENT: the logits were written by other
// workgroups of the running kernel, so they are read at device scope.
template <bool COHERENT = false>
__device__ __forceinline__ void select_tokens(const float* __restrict__ logits, int t0, int T, int N, int k, int route,
                                              int n_groups, int topk_groups, SelectShared& sh) {
  const int tid = threadIdx.x;
  const int nt = min(4, T - t0);
  const int e = tid;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t >= nt) break;
    const float* zp = logits + static_cast<size_t>(t0 + t) * N + e;
    float z = 0.f;
    if (e < N) z = COHERENT ? __hip_atomic_load(zp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : *zp;
    sh.z[t][e] = z;
    sh.key[t][e] = e < N ? (static_cast<uint64_t>(order_key(z)) << 32) | static_cast<uint32_t>(255 - e) : 0ull;
  }
  __syncthreads();
  if (route == R_SIGMOID_GROUP) {
    const int gs = N / n_groups;
    // group score: the sum of the sigmoids of the group's two largest logits
    if (tid < nt * n_groups) {
      const int t = tid / n_groups, q = tid - t * n_groups;
      uint64_t k1 = 0, k2 = 0;
      int b1 = -1, b2 = -1;
      for (int i = q * gs; i < (q + 1) * gs; ++i) {
        const uint64_t ki = sh.key[t][i];
        if (ki > k1) { k2 = k1; b2 = b1; k1 = ki; b1 = i; }
        else if (ki > k2) { k2 = ki; b2 = i; }
      }
      sh.gam[t][q] = sel_sigmoid(sh.z[t][b1]) + (b2 >= 0 ? sel_sigmoid(sh.z[t][b2]) : 0.f);
    }
    __syncthreads();
    // keep the topk_groups best groups (score desc, group asc)
    bool drop[4] = {false, false, false, false};
    if (e < N) {
      const int q = e / gs;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (t >= nt) break;
        int grank = 0;
        const float b = sh.gam[t][q];
        for (int q2 = 0; q2 < n_groups; ++q2) {
          const float a = sh.gam[t][q2];
          grank += (a > b || (a == b && q2 < q)) ? 1 : 0;
        }
        drop[t] = grank >= topk_groups;
      }
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (t < nt && drop[t]) sh.key[t][e] = 0ull;
    __syncthreads();
  }
  if (e < N) {
    const int n_pad = (N + 15) & ~15;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (t >= nt) break;
      const uint64_t ke = sh.key[t][e];
      if (ke == 0ull) continue;
      int rank = 0;
      for (int e2 = 0; e2 < n_pad; e2 += 16) {
#pragma unroll
        for (int q = 0; q < 16; ++q) rank += sh.key[t][e2 + q] > ke ? 1 : 0;   // broadcast reads
      }
      if (rank < k) sh.sel[t][rank] = e;
    }
  }
  __syncthreads();
  if (tid < nt) {
    const int t = tid;
    float g[8];
    float den = 0.f;
    const float z0 = sh.z[t][sh.sel[t][0]];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j >= k) break;
      const float zj = sh.z[t][sh.sel[t][j]];
      g[j] = route == R_SIGMOID_GROUP ? sel_sigmoid(zj) : __expf(zj - z0);
      den += g[j];
    }
    const float inv = 1.0f / den;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j >= k) break;
      sh.gate[t][j] = g[j] * inv;
    }
  }
  __syncthreads();
}

}  // namespace wisp
