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

constexpr int kSelectMaxSplit = 8;   // partial sums of a logit the selection adds (kRouterMaxSplit)

struct SelectShared {
  uint64_t key[4][256];   // (order-preserving logit << 32 | 255 - id), 0 = not allowed
  float z[4][256];
  int cnt[4][256];        // partial ranks (N <= 128: threads e and e + 128 count halves)
  float gam[4][32];
  int sel[4][8];
  float term[4][8];       // exp(z_j - z_0) or sigmoid(z_j) of rank j
  float gate[4][8];
};

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float sel_sigmoid(float z) { return 1.0f / (1.0f + __expf(-z)); }

// A logit published by another workgroup of the running kernel: one 64-bit word, the launch's tag
// above the fp32 bits, written by a single atomic store.
__device__ __forceinline__ uint64_t tag_logit(uint32_t tag, float z) {
  return (static_cast<uint64_t>(tag) << 32) | __float_as_uint(z);
}

// Spins (bounded) until the word carries `tag`.  Atomic accesses to one location are coherent, so once
// the publishing workgroup's store is visible the word holds this launch's logit.  Only the reading
// workgroup waits; every publisher computes its row and stores it without waiting for anything, so
// each store is issued once the publisher has been dispatched, whether or not all workgroups fit on
// the chip at once.  After kTagSpins polls (seconds) the word is used as it is.
constexpr int kTagSpins = 1 << 22;
__device__ __forceinline__ float read_tagged_logit(const uint64_t* p, uint32_t tag) {
  uint64_t v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (int i = 0; static_cast<uint32_t>(v >> 32) != tag && i < kTagSpins; ++i) {
    __builtin_amdgcn_s_sleep(1);
    v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return __uint_as_float(static_cast<uint32_t>(v));
}

// Tokens t0 .. t0+3 (those < T) of logits [T, N]; all 256 threads must call it.  Thread e owns
// expert e of every token (N <= 256).  A key packs the order-preserving bits of the logit above
// 255 - id, so (logit desc, id asc) is plain unsigned order and every allowed key is distinct:
// the rank of an expert is the number of larger keys.  TAGGED: the logits are 64-bit tagged words
// published by other workgroups of the running kernel (tag_logit), read until they carry `tag`;
// otherwise plain fp32 written by an earlier kernel, as n_split partial sums (split s at s * split_stride
// floats), added in split order.
template <bool TAGGED = false>
__device__ __forceinline__ void select_tokens(const void* __restrict__ logits, uint32_t tag, int t0, int T, int N,
                                              int k, int route, int n_groups, int topk_groups, SelectShared& sh,
                                              int n_split = 1, size_t split_stride = 0) {
  const int tid = threadIdx.x;
  const int nt = min(4, T - t0);
  const int e = tid;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t >= nt) break;
    const size_t at = static_cast<size_t>(t0 + t) * N + e;
    float z = 0.f;
    if (e < N) {
      if (TAGGED) {
        z = read_tagged_logit(static_cast<const uint64_t*>(logits) + at, tag);
      } else {
        // the slices' loads go out together, then they are added in slice order
        const float* f = static_cast<const float*>(logits);
        float part[kSelectMaxSplit];
#pragma unroll
        for (int q = 0; q < kSelectMaxSplit; ++q) part[q] = q < n_split ? f[q * split_stride + at] : 0.f;
        z = part[0];
#pragma unroll
        for (int q = 1; q < kSelectMaxSplit; ++q)
          if (q < n_split) z += part[q];
      }
    }
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
  // rank of expert e = the number of larger keys.  Up to 128 experts, threads e and e + 128 each
  // count over one half of the (16-padded) row and the halves are added; beyond, thread e counts
  // the whole row.
  const int n_pad = (N + 15) & ~15;
  const bool split = N <= 128;
  const int ex = split ? (tid & 127) : tid;
  const int h_mid = split ? ((n_pad + 31) >> 5) << 4 : n_pad;   // a multiple of 16
  const int r0 = split && tid >= 128 ? h_mid : 0, r1 = split && tid < 128 ? h_mid : n_pad;
  if (ex < N) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (t >= nt) break;
      const uint64_t ke = sh.key[t][ex];
      int rank = 0;
      if (ke != 0ull) {
        for (int e2 = r0; e2 < r1; e2 += 16) {
#pragma unroll
          for (int q = 0; q < 16; ++q) rank += sh.key[t][e2 + q] > ke ? 1 : 0;   // broadcast reads
        }
      }
      sh.cnt[t][tid] = rank;
    }
  }
  __syncthreads();
  if (e < N) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (t >= nt) break;
      if (sh.key[t][e] == 0ull) continue;
      const int rank = split ? sh.cnt[t][e] + sh.cnt[t][e + 128] : sh.cnt[t][e];
      if (rank < k) sh.sel[t][rank] = e;
    }
  }
  __syncthreads();
  // gates: the terms of all ranks in parallel, then one thread per token sums them in rank order
  // and each rank's gate is its term times the reciprocal (the same operations as a serial loop)
  {
    const int t = tid >> 3, j = tid & 7;
    if (t < nt && j < k) {
      const float zj = sh.z[t][sh.sel[t][j]];
      sh.term[t][j] = route == R_SIGMOID_GROUP ? sel_sigmoid(zj) : __expf(zj - sh.z[t][sh.sel[t][0]]);
    }
  }
  __syncthreads();
  if (tid < nt) {
    const int t = tid;
    float den = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j >= k) break;
      den += sh.term[t][j];
    }
    const float inv = 1.0f / den;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j >= k) break;
      sh.gate[t][j] = sh.term[t][j] * inv;
    }
  }
  __syncthreads();
}

}  // namespace wisp
