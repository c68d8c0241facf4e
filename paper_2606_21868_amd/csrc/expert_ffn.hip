// Slot-indirected expert FFN for decode-sized token counts (gfx950).
//
// The expert is o = W2 (silu(W1 x) * (W3 x)).  At decode sizes every weight byte is used once
// per token, so the work is a streaming GEMV bound by HBM bandwidth, not a contraction worth
// MFMA tiles.  Each launch covers a batch of "items" (an expert blob in its slot plus the up to
// four tokens that chose it), so an expert is read once however many tokens use it.
//
// Layout of the work: a group of LPR lanes owns one weight row; lane l of the group reads the
// 16-byte chunks l, l + LPR, ... of the row (coalesced across the group), decodes them (fp32 /
// bf16 bit shifts; fp8 E4M3 with the hardware packed conversion, times the bf16 scale of the
// chunk's 128x128 block), and multiplies them with the matching input elements read from LDS,
// where the workgroup has staged the item's input rows.  Group partial sums are reduced with
// cross-lane shuffles.  Phase 1 (gate/up) reads the W1 and W3 rows of the same output index
// together and writes h = silu(a) * b; phase 2 (down) reads W2 rows and writes the per-(token,
// rank) outputs that the combine kernel sums in rank order.  Both phases give every item its own
// row blocks (a grid of items x row blocks): many waves with few loads each hide HBM latency
// better than few waves that each walk every expert.  Every (token, rank) result is
// computed by the same instructions in the same order whatever the batch composition, so a
// paged run is bit-identical to a fully resident one.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.hpp"

namespace wisp {

BlobLayout make_blob_layout(int d, int I, int w_dtype) {
  BlobLayout L;
  L.d = d;
  L.I = I;
  L.w_dtype = w_dtype;
  L.elem = w_dtype == DT_F32 ? 4 : w_dtype == DT_BF16 ? 2 : 1;
  const size_t n = static_cast<size_t>(d) * I;
  L.off_w1 = 0;
  L.off_w3 = n * L.elem;
  L.off_w2 = 2 * n * L.elem;
  L.bytes = 3 * n * L.elem;
  if (w_dtype == DT_FP8) {
    const size_t nb = static_cast<size_t>(d / 128) * (I / 128);
    L.off_s1 = 3 * n;
    L.off_s3 = L.off_s1 + 2 * nb;
    L.off_s2 = L.off_s3 + 2 * nb;
    L.bytes = 3 * n + 6 * nb;
  }
  return L;
}

namespace {

enum { MODE_GATEUP = 0, MODE_DOWN = 1 };

template <int WT> struct WFmt;
template <> struct WFmt<DT_F32> { static constexpr int EPL = 4; };
template <> struct WFmt<DT_BF16> { static constexpr int EPL = 8; };
template <> struct WFmt<DT_FP8> { static constexpr int EPL = 16; };

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

// Four E4M3 codes (little-endian bytes of w) to fp32 with the gfx950 packed conversion.
__device__ __forceinline__ void fp8x4(uint32_t w, float* o) {
  auto lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), false);
  auto hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w), true);
  o[0] = lo[0];
  o[1] = lo[1];
  o[2] = hi[0];
  o[3] = hi[1];
}

template <int WT>
__device__ __forceinline__ void decode_chunk(const uint4 v, float* o) {
  if constexpr (WT == DT_F32) {
    o[0] = __uint_as_float(v.x); o[1] = __uint_as_float(v.y);
    o[2] = __uint_as_float(v.z); o[3] = __uint_as_float(v.w);
  } else if constexpr (WT == DT_BF16) {
    o[0] = bf16_lo(v.x); o[1] = bf16_hi(v.x); o[2] = bf16_lo(v.y); o[3] = bf16_hi(v.y);
    o[4] = bf16_lo(v.z); o[5] = bf16_hi(v.z); o[6] = bf16_lo(v.w); o[7] = bf16_hi(v.w);
  } else {
    fp8x4(v.x, o); fp8x4(v.y, o + 4); fp8x4(v.z, o + 8); fp8x4(v.w, o + 12);
  }
}

// EPL consecutive input elements starting at element col of an LDS row.
template <int IT, int EPL>
__device__ __forceinline__ void lds_chunk(const uint8_t* row, int col, float* o) {
  if constexpr (IT == DT_F32) {
    static_assert(EPL % 4 == 0, "");
    const float4* p = reinterpret_cast<const float4*>(row + static_cast<size_t>(col) * 4);
#pragma unroll
    for (int q = 0; q < EPL / 4; ++q) {
      const float4 v = p[q];
      o[4 * q] = v.x; o[4 * q + 1] = v.y; o[4 * q + 2] = v.z; o[4 * q + 3] = v.w;
    }
  } else {
    static_assert(EPL % 8 == 0, "");
    const uint4* p = reinterpret_cast<const uint4*>(row + static_cast<size_t>(col) * 2);
#pragma unroll
    for (int q = 0; q < EPL / 8; ++q) {
      const uint4 v = p[q];
      o[8 * q + 0] = bf16_lo(v.x); o[8 * q + 1] = bf16_hi(v.x); o[8 * q + 2] = bf16_lo(v.y); o[8 * q + 3] = bf16_hi(v.y);
      o[8 * q + 4] = bf16_lo(v.z); o[8 * q + 5] = bf16_hi(v.z); o[8 * q + 6] = bf16_lo(v.w); o[8 * q + 7] = bf16_hi(v.w);
    }
  }
}

// The same EPL input elements from 16-byte chunks held in registers.
template <int IT, int EPL>
__device__ __forceinline__ void reg_chunk(const uint4* q, float* o) {
  if constexpr (IT == DT_F32) {
#pragma unroll
    for (int c = 0; c < EPL / 4; ++c) {
      o[4 * c] = __uint_as_float(q[c].x); o[4 * c + 1] = __uint_as_float(q[c].y);
      o[4 * c + 2] = __uint_as_float(q[c].z); o[4 * c + 3] = __uint_as_float(q[c].w);
    }
  } else {
#pragma unroll
    for (int c = 0; c < EPL / 8; ++c) {
      o[8 * c + 0] = bf16_lo(q[c].x); o[8 * c + 1] = bf16_hi(q[c].x); o[8 * c + 2] = bf16_lo(q[c].y);
      o[8 * c + 3] = bf16_hi(q[c].y); o[8 * c + 4] = bf16_lo(q[c].z); o[8 * c + 5] = bf16_hi(q[c].z);
      o[8 * c + 6] = bf16_lo(q[c].w); o[8 * c + 7] = bf16_hi(q[c].w);
    }
  }
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// acc + w.lo * x.lo + w.hi * x.hi on two packed bf16 pairs (one v_dot2c_f32_bf16).
__device__ __forceinline__ float dot2_bf16(uint32_t w, uint32_t x, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w), __builtin_bit_cast(bf16x2_t, x), acc, false);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Rows [r_begin, r_end) of one item, by one workgroup.  Weights and fp8 scales are read from the
// blob at `rd`; if `wr` is not null every loaded 16-byte chunk is also stored at the same offset
// of `wr` (a faulted expert streamed from its host master into its slot while being used).
// K = inner (row) length, R = rows; off0/off1: byte offsets of the matrix (matrices) in the blob;
// soff0/soff1: fp8 scale tables.  The arithmetic is the same whatever rd / wr are.
template <int WT, int IT, int MODE, int LPR, int NLT>
__device__ __forceinline__ void rows_body(const FfnItem& it, const uint8_t* rd, uint8_t* wr,
                                          const uint8_t* __restrict__ vin, int vin_stride, int K, int R, int r_begin,
                                          int r_end, uint32_t off0, uint32_t off1, uint32_t soff0, uint32_t soff1,
                                          uint8_t* __restrict__ out, int out_stride, uint8_t* lds) {
  constexpr int EPL = WFmt<WT>::EPL;
  constexpr int RPW = 64 / LPR;                 // rows a wave covers at once
  constexpr int IS = IT == DT_F32 ? 4 : 2;      // input element bytes
  constexpr int U = NLT > 0 ? NLT : 4;          // chunks in flight per lane
  const int ntok = it.ntok;
  const int row_bytes = K * IS;

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int sub = lane / LPR;
  const int sl = lane - sub * LPR;
  const int NL = NLT > 0 ? NLT : (K / EPL) / LPR;
  const uint8_t* wbase0 = rd + off0;
  const uint8_t* wbase1 = rd + off1;
  const uint16_t* sc0 = reinterpret_cast<const uint16_t*>(rd + soff0);
  const uint16_t* sc1 = reinterpret_cast<const uint16_t*>(rd + soff1);
  const int scols = K / 128;
  const size_t row_stride_b = static_cast<size_t>(K) * (WT == DT_F32 ? 4 : WT == DT_BF16 ? 2 : 1);

  // Single-token items of the unrolled shapes keep the lane's slice of the input row in registers:
  // a lane reads the same columns of every row it processes, so the slice is loaded once, before
  // the weights, and no LDS staging or barrier is needed.  Other items stage their input rows in
  // LDS.  The multiply-add sequence is the same either way.
  constexpr int XQ = NLT > 0 ? EPL * IS / 16 : 1;          // 16-byte input chunks per weight chunk
  constexpr bool kXreg = NLT > 0 && !(WT == DT_FP8 && NLT > 4);
  const bool xreg = kXreg && ntok == 1;
  uint4 xr[kXreg ? NLT * XQ : 1];
  const int rbase0 = r_begin + wave * RPW;
  const uint8_t* xrow = vin + static_cast<size_t>(MODE == MODE_GATEUP ? it.tok[0] : it.out[0]) * vin_stride * IS;
  if (!xreg) {
    // stage the item's input rows (x for gate/up, h for down) in LDS
    for (int t = 0; t < ntok; ++t) {
      const int src_row = MODE == MODE_GATEUP ? it.tok[t] : it.out[t];
      const uint4* src = reinterpret_cast<const uint4*>(vin + static_cast<size_t>(src_row) * vin_stride * IS);
      uint4* dst = reinterpret_cast<uint4*>(lds + t * row_bytes);
      for (int i = threadIdx.x; i < row_bytes / 16; i += 256) dst[i] = src[i];
    }
    __syncthreads();
  }

  for (int rbase = rbase0; rbase < r_end; rbase += 4 * RPW) {
    const int r = rbase + sub;
    const bool valid = r < r_end;
    const int rr = valid ? r : r_begin;   // keep addresses in range for idle row groups
    float acc0[kMaxTokPerItem], acc1[kMaxTokPerItem];
#pragma unroll
    for (int t = 0; t < kMaxTokPerItem; ++t) { acc0[t] = 0.f; acc1[t] = 0.f; }
    const uint4* row0 = reinterpret_cast<const uint4*>(wbase0 + rr * row_stride_b);
    const uint4* row1 = reinterpret_cast<const uint4*>(wbase1 + rr * row_stride_b);

    for (int m0 = 0; m0 < NL; m0 += U) {
      uint4 a[U], b[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int m = m0 + u;
        if (NLT > 0 || m < NL) {
          a[u] = row0[m * LPR + sl];
          if constexpr (MODE == MODE_GATEUP) b[u] = row1[m * LPR + sl];
        }
      }
      if (xreg && m0 == 0) {
        // the input slice is read after the weight loads are issued, through an address the
        // compiler cannot see as loop-invariant, so neither the load nor its conversion is hoisted
        // ahead of the weight loads (which would put two memory round trips in a row)
        uint32_t opaque = 0;
        asm volatile("" : "+s"(opaque));
        const uint8_t* xp = xrow + opaque;
#pragma unroll
        for (int m = 0; m < (NLT > 0 ? NLT : 1); ++m)
#pragma unroll
          for (int q = 0; q < XQ; ++q)
            xr[m * XQ + q] = reinterpret_cast<const uint4*>(xp + static_cast<size_t>((m * LPR + sl) * EPL) * IS)[q];
      }
      if (wr && valid) {
        uint4* w0 = reinterpret_cast<uint4*>(wr + off0 + rr * row_stride_b);
        uint4* w1 = reinterpret_cast<uint4*>(wr + off1 + rr * row_stride_b);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int m = m0 + u;
          if (NLT > 0 || m < NL) {
            w0[m * LPR + sl] = a[u];
            if constexpr (MODE == MODE_GATEUP) w1[m * LPR + sl] = b[u];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int m = m0 + u;
        if (!(NLT > 0 || m < NL)) continue;
        const int col = (m * LPR + sl) * EPL;
        if constexpr (WT == DT_BF16 && IT == DT_BF16) {
          // packed bf16 pairs straight into v_dot2c_f32_bf16: a*b products of bf16 values are exact in
          // fp32, so only the sums round; no unpacking of weights or inputs
#pragma unroll
          for (int t = 0; t < kMaxTokPerItem; ++t) {
            if (t >= ntok) break;
            const uint4 xq = xreg ? xr[(NLT > 0 ? m : 0) * XQ]
                                  : *reinterpret_cast<const uint4*>(lds + t * row_bytes + col * 2);
            acc0[t] = dot2_bf16(a[u].x, xq.x, acc0[t]);
            acc0[t] = dot2_bf16(a[u].y, xq.y, acc0[t]);
            acc0[t] = dot2_bf16(a[u].z, xq.z, acc0[t]);
            acc0[t] = dot2_bf16(a[u].w, xq.w, acc0[t]);
            if constexpr (MODE == MODE_GATEUP) {
              acc1[t] = dot2_bf16(b[u].x, xq.x, acc1[t]);
              acc1[t] = dot2_bf16(b[u].y, xq.y, acc1[t]);
              acc1[t] = dot2_bf16(b[u].z, xq.z, acc1[t]);
              acc1[t] = dot2_bf16(b[u].w, xq.w, acc1[t]);
            }
          }
          continue;
        }
        float wa[EPL], wb[EPL];
        decode_chunk<WT>(a[u], wa);
        if constexpr (MODE == MODE_GATEUP) decode_chunk<WT>(b[u], wb);
        float s0 = 1.f, s1 = 1.f;
        if constexpr (WT == DT_FP8) {
          const int sidx = (rr / 128) * scols + col / 128;
          s0 = __uint_as_float(static_cast<uint32_t>(sc0[sidx]) << 16);
          if constexpr (MODE == MODE_GATEUP) s1 = __uint_as_float(static_cast<uint32_t>(sc1[sidx]) << 16);
        }
#pragma unroll
        for (int t = 0; t < kMaxTokPerItem; ++t) {
          if (t >= ntok) break;
          float xv[EPL];
          if (xreg) reg_chunk<IT, EPL>(&xr[(NLT > 0 ? m : 0) * XQ], xv);
          else lds_chunk<IT, EPL>(lds + t * row_bytes, col, xv);
          if constexpr (WT == DT_FP8) {
            float pa = 0.f, pb = 0.f;
#pragma unroll
            for (int e = 0; e < EPL; ++e) {
              pa = fmaf(wa[e], xv[e], pa);
              if constexpr (MODE == MODE_GATEUP) pb = fmaf(wb[e], xv[e], pb);
            }
            acc0[t] = fmaf(s0, pa, acc0[t]);
            if constexpr (MODE == MODE_GATEUP) acc1[t] = fmaf(s1, pb, acc1[t]);
          } else {
#pragma unroll
            for (int e = 0; e < EPL; ++e) {
              acc0[t] = fmaf(wa[e], xv[e], acc0[t]);
              if constexpr (MODE == MODE_GATEUP) acc1[t] = fmaf(wb[e], xv[e], acc1[t]);
            }
          }
        }
      }
    }
    // reduce over the LPR lanes of the row group
#pragma unroll
    for (int t = 0; t < kMaxTokPerItem; ++t) {
      if (t >= ntok) break;
#pragma unroll
      for (int off = LPR / 2; off > 0; off >>= 1) {
        acc0[t] += __shfl_xor(acc0[t], off, 64);
        if constexpr (MODE == MODE_GATEUP) acc1[t] += __shfl_xor(acc1[t], off, 64);
      }
    }
    if (valid && sl == 0) {
      for (int t = 0; t < ntok; ++t) {
        const size_t o = static_cast<size_t>(it.out[t]) * out_stride + r;
        if constexpr (MODE == MODE_GATEUP) {
          const float a = acc0[t];
          const float h = a / (1.0f + __expf(-a)) * acc1[t];
          if constexpr (IT == DT_F32) reinterpret_cast<float*>(out)[o] = h;
          else reinterpret_cast<uint16_t*>(out)[o] = f32_to_bf16_rne(h);
        } else {
          reinterpret_cast<float*>(out)[o] = acc0[t];
        }
      }
    }
  }
}

// Host-planned launch: blockIdx.x = item * blocks_per_item + row block; the items come with the
// launch (kernel arguments).
template <int WT, int IT, int MODE, int LPR, int NLT>
__global__ void __launch_bounds__(256) ffn_rows(const FfnBatch B, const uint8_t* __restrict__ vin, int vin_stride,
                                                int K, int R, int rows_per_wg, int blocks_per_item, uint32_t off0,
                                                uint32_t off1, uint32_t soff0, uint32_t soff1,
                                                uint8_t* __restrict__ out, int out_stride) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int item_idx = blockIdx.x / blocks_per_item;
  const int rb = blockIdx.x - item_idx * blocks_per_item;
  const FfnItem& it = B.items[item_idx];
  const int r_begin = rb * rows_per_wg;
  rows_body<WT, IT, MODE, LPR, NLT>(it, it.w, nullptr, vin, vin_stride, K, R, r_begin, min(R, r_begin + rows_per_wg),
                                    off0, off1, soff0, soff1, out, out_stride, lds);
}

// Device-planned gate/up: the item list was written to HBM by the device pager of this layer.
// Per item slot, bpi workgroups: a resident expert uses them as row blocks of rows_hit rows; a
// faulted expert uses fault_wgs of them to stream its W1/W3 rows from the host master (computing
// h and filling the slot) and copy_wgs more to copy the rest of its blob (W2 and fp8 scales)
// host -> slot; the others exit.  The PCIe stream needs few workgroups, which leaves the CUs to
// the resident experts meanwhile.
template <int WT, int IT, int LPR, int NLT>
__global__ void __launch_bounds__(256) ffn_gateup_dev(const FfnBatch* __restrict__ P, const uint8_t* __restrict__ vin,
                                                      int d, int I, int bpi, int rows_hit, int fault_wgs, int copy_wgs,
                                                      uint32_t off1, uint32_t off3, uint32_t soff1, uint32_t soff3,
                                                      uint32_t copy_off, uint32_t copy_bytes, uint8_t* __restrict__ h) {
  extern __shared__ __align__(16) uint8_t lds[];
  constexpr int RPW = 64 / LPR;
  const int item_idx = blockIdx.x / bpi;
  const int j = blockIdx.x - item_idx * bpi;
  if (item_idx >= P->n_items) return;
  const FfnItem& it = P->items[item_idx];
  if (!it.fault) {
    const int r_begin = j * rows_hit;
    if (r_begin >= I) return;
    rows_body<WT, IT, MODE_GATEUP, LPR, NLT>(it, it.w, nullptr, vin, d, d, I, r_begin, min(I, r_begin + rows_hit),
                                             off1, off3, soff1, soff3, h, I, lds);
  } else if (j < fault_wgs) {
    int rows = (I + fault_wgs - 1) / fault_wgs;
    rows = (rows + 4 * RPW - 1) / (4 * RPW) * (4 * RPW);
    const int r_begin = j * rows;
    if (r_begin >= I) return;
    rows_body<WT, IT, MODE_GATEUP, LPR, NLT>(it, it.src, const_cast<uint8_t*>(it.w), vin, d, d, I, r_begin,
                                             min(I, r_begin + rows), off1, off3, soff1, soff3, h, I, lds);
  } else if (j < fault_wgs + copy_wgs) {
    // copy [copy_off, copy_off + copy_bytes) host -> slot, four 16-byte loads in flight per thread
    const int q = j - fault_wgs;
    const size_t n16 = copy_bytes / 16;
    const size_t per = (n16 + copy_wgs - 1) / copy_wgs;
    const size_t c0 = static_cast<size_t>(q) * per;
    const size_t c1 = c0 + per < n16 ? c0 + per : n16;
    const uint4* src = reinterpret_cast<const uint4*>(it.src + copy_off);
    uint4* dst = reinterpret_cast<uint4*>(const_cast<uint8_t*>(it.w) + copy_off);
    size_t i = c0 + threadIdx.x;
    for (; i + 768 < c1; i += 1024) {
      const uint4 a = src[i], b = src[i + 256], c = src[i + 512], e = src[i + 768];
      dst[i] = a; dst[i + 256] = b; dst[i + 512] = c; dst[i + 768] = e;
    }
    for (; i < c1; i += 256) dst[i] = src[i];
    if (q == copy_wgs - 1) {
      for (size_t b = n16 * 16 + threadIdx.x; b < copy_bytes; b += 256)
        const_cast<uint8_t*>(it.w)[copy_off + b] = it.src[copy_off + b];
    }
  }
}

// Device-planned down projection: per item slot, row blocks of W2 (every expert of the step is
// resident by now; faulted ones were filled by the gate/up kernel).
template <int WT, int IT, int LPR, int NLT>
__global__ void __launch_bounds__(256) ffn_down_dev(const FfnBatch* __restrict__ P, const uint8_t* __restrict__ h,
                                                    int d, int I, int bpi, int rows_per_wg, uint32_t off2,
                                                    uint32_t soff2, float* __restrict__ buf) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int item_idx = blockIdx.x / bpi;
  const int rb = blockIdx.x - item_idx * bpi;
  if (item_idx >= P->n_items) return;
  const FfnItem& it = P->items[item_idx];
  const int r_begin = rb * rows_per_wg;
  if (r_begin >= d) return;
  rows_body<WT, IT, MODE_DOWN, LPR, NLT>(it, it.w, nullptr, h, I, I, d, r_begin, min(d, r_begin + rows_per_wg), off2,
                                         off2, soff2, soff2, reinterpret_cast<uint8_t*>(buf), d, lds);
}

// Single-token launches with bf16 weights and inputs (every decode launch at batch 1): a lean copy
// of rows_body for this case.  All weight loads of a row group are issued first and the input slice
// after them, and each row is the same chain of v_dot2c_f32_bf16
// over the lane's chunks followed by the same shuffle reduction as rows_body, so a row's result has
// the same bits whichever of the two kernels computes it.
struct FfnT1Batch {
  const uint8_t* w[kMaxItems];
  int32_t row[kMaxItems];    // input row: the token (gate/up) or the h row (down)
  int32_t out[kMaxItems];    // output row
  int32_t n_items;
};

// A 16-byte weight load with the non-temporal hint: every weight of a layer-step is read once, so
// its lines need not displace anything in the caches (3 % faster on the gate/up launches).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// One row pass of the single-token body, split so that the weight loads can be issued early: the
// lane's NL 16-byte chunks of row rr of the first (and, for gate/up, second) matrix ...
template <int MODE, int LPR, int NL>
__device__ __forceinline__ void t1_load(const uint8_t* w, uint32_t off0, uint32_t off1, size_t row_b, int rr, int sl,
                                        uint4* a, uint4* b) {
  const uint4* row0 = reinterpret_cast<const uint4*>(w + off0 + rr * row_b);
  const uint4* row1 = reinterpret_cast<const uint4*>(w + off1 + rr * row_b);
#pragma unroll
  for (int m = 0; m < NL; ++m) {
    a[m] = load_stream(row0 + m * LPR + sl);
    if constexpr (MODE == MODE_GATEUP) b[m] = load_stream(row1 + m * LPR + sl);
  }
}

// ... the lane's input chunks (issued after the weights) ...
template <int LPR, int NL>
__device__ __forceinline__ void t1_input(const uint4* xrow, int sl, uint4* xr) {
#pragma unroll
  for (int m = 0; m < NL; ++m) xr[m] = xrow[m * LPR + sl];
}

// ... and the row's dot products: one v_dot2c_f32_bf16 chain over the lane's chunks, then the
// shuffle reduction over the LPR lanes of the row group.  Every single-token kernel computes a row
// through this function, so a row has the same bits whichever kernel computes it.
template <int MODE, int LPR, int NL>
__device__ __forceinline__ void t1_dot(const uint4* a, const uint4* b, const uint4* xr, float& acc0, float& acc1) {
  acc0 = 0.f;
  acc1 = 0.f;
#pragma unroll
  for (int m = 0; m < NL; ++m) {
    acc0 = dot2_bf16(a[m].x, xr[m].x, acc0);
    acc0 = dot2_bf16(a[m].y, xr[m].y, acc0);
    acc0 = dot2_bf16(a[m].z, xr[m].z, acc0);
    acc0 = dot2_bf16(a[m].w, xr[m].w, acc0);
    if constexpr (MODE == MODE_GATEUP) {
      acc1 = dot2_bf16(b[m].x, xr[m].x, acc1);
      acc1 = dot2_bf16(b[m].y, xr[m].y, acc1);
      acc1 = dot2_bf16(b[m].z, xr[m].z, acc1);
      acc1 = dot2_bf16(b[m].w, xr[m].w, acc1);
    }
  }
#pragma unroll
  for (int off = LPR / 2; off > 0; off >>= 1) {
    acc0 += __shfl_xor(acc0, off, 64);
    if constexpr (MODE == MODE_GATEUP) acc1 += __shfl_xor(acc1, off, 64);
  }
}

__device__ __forceinline__ uint16_t swiglu_bf16(float a, float b) {
  return f32_to_bf16_rne(a / (1.0f + __expf(-a)) * b);
}

// One pass of the single-token body over rows [rbase, rbase + RPW) of the item's matrix.
template <int MODE, int LPR, int NL>
__device__ __forceinline__ void t1_pass(const uint8_t* w, const uint4* xrow, int K, int rbase, int r_end, int r_first,
                                        uint32_t off0, uint32_t off1, uint8_t* __restrict__ out, size_t out_row) {
  constexpr int RPW = 64 / LPR;
  const int lane = threadIdx.x & 63;
  const int sub = lane / LPR, sl = lane - sub * LPR;
  const size_t row_b = static_cast<size_t>(K) * 2;
  const int r = rbase + sub;
  const bool valid = r < r_end;
  const int rr = valid ? r : r_first;
  uint4 a[NL], b[NL], xr[NL];
  t1_load<MODE, LPR, NL>(w, off0, off1, row_b, rr, sl, a, b);
  t1_input<LPR, NL>(xrow, sl, xr);
  float acc0, acc1;
  t1_dot<MODE, LPR, NL>(a, b, xr, acc0, acc1);
  if (valid && sl == 0) {
    if constexpr (MODE == MODE_GATEUP)
      reinterpret_cast<uint16_t*>(out)[out_row + r] = swiglu_bf16(acc0, acc1);
    else
      reinterpret_cast<float*>(out)[out_row + r] = acc0;
  }
  (void)RPW;
}

// Grid (row blocks, items): the item is blockIdx.y.  A kernel that follows another kernel starts
// with cold instruction and scalar caches, so every dependent round trip before its first weight
// load shows in its duration.  With ONE_PASS (a workgroup's rows_per_wg = 4 * RPW rows, one pass of
// its four waves: every batch-1 decode launch) the body is straight-line, and the workgroup's
// scalar loads, its item's blob address among them, go out together before anything waits.
template <int MODE, int LPR, int NL, bool ONE_PASS>
__global__ void __launch_bounds__(256) ffn_rows_t1(const FfnT1Batch B, const uint8_t* __restrict__ vin, int vin_stride,
                                                   int K, int R, int rows_per_wg, uint32_t off0, uint32_t off1,
                                                   uint8_t* __restrict__ out, int out_stride) {
  constexpr int RPW = 64 / LPR;
  const int item = blockIdx.y;
  const int wave = threadIdx.x >> 6;
  const uint8_t* w = B.w[item];
  const uint4* xrow = reinterpret_cast<const uint4*>(vin + static_cast<size_t>(B.row[item]) * vin_stride * 2);
  const size_t out_row = static_cast<size_t>(B.out[item]) * out_stride;
  if constexpr (ONE_PASS) {
    // K = LPR * NL chunks of 8 bf16 and rows_per_wg = 4 * RPW are fixed by the instantiation, so
    // nothing but R waits on a kernel argument before the addresses are formed
    constexpr int KC = LPR * NL * 8;
    const int r_begin = blockIdx.x * 4 * RPW;
    t1_pass<MODE, LPR, NL>(w, xrow, KC, r_begin + wave * RPW, min(R, r_begin + 4 * RPW), r_begin, off0, off1, out,
                           out_row);
    (void)K;
    (void)rows_per_wg;
  } else {
    const int r_begin = blockIdx.x * rows_per_wg, r_end = min(R, r_begin + rows_per_wg);
    for (int rbase = r_begin + wave * RPW; rbase < r_end; rbase += 4 * RPW)
      t1_pass<MODE, LPR, NL>(w, xrow, K, rbase, r_end, r_begin, off0, off1, out, out_row);
  }
}

// ------------------------------------------------------------------------------------------
// Down projection fused with the gate-weighted combine, for single-token steps with bf16 weights
// (every decode layer-step at batch 1).  A workgroup owns RPW output rows for all of the step's
// experts: wave w computes o_j for the experts w, w + 4, ... (W2 rows first, then the h slices),
// the outputs meet in LDS and y = sum_j g_j o_j (+ the shared expert) is formed in rank order.  The
// separate down kernel writes every o_j to HBM for a combine launch to read back; here it never
// leaves the chip, and a layer-step needs one launch less.  Each o_j is t1_dot's chain and the sum
// is the combine kernel's fmaf chain, so y has the same bits as down + combine.
// ------------------------------------------------------------------------------------------
// Where the items of a single-token down + combine come from: the launch's kernel argument (host
// pager) or the plan the device pager wrote to HBM (read straight from there: a scalar load of
// memory another kernel wrote is coherent, since every kernel starts with its caches invalidated).
struct ArgItems {
  const FusedT1Items& b;
  __device__ int n() const { return b.n_items; }
  __device__ const uint8_t* w(int i) const { return b.w[i]; }
  __device__ int32_t rank(int i) const { return b.rank[i]; }
};
struct PlanItems {
  const FfnBatch* p;
  __device__ int n() const { return p->n_items; }
  __device__ const uint8_t* w(int i) const { return p->items[i].w; }
  __device__ int32_t rank(int i) const { return p->items[i].out[0]; }   // single-token items: the rank
};

template <int LPR, int NL, int MAXW, typename Items>
__device__ __forceinline__ void down_combine_t1(const Items& items, const uint8_t* h, const float* __restrict__ gates,
                                                float* __restrict__ y, int d, int I, int k, int has_shared,
                                                uint32_t off2, float* o_lds) {
  constexpr int RPW = 64 / LPR;
  static_assert(4 * MAXW <= kMaxItems, "the item arrays hold every index read below");
  static_assert(MAXW == 3, "the scalar hold below names three experts per wave");
  // The wave index is uniform, so the experts' addresses and ranks are scalar values.  They are read
  // (entries past n exist in both item arrays and are never dereferenced) together with the other scalars
  // the loads need, and held in scalar registers by one empty asm statement, so the workgroup waits
  // once for all of them; otherwise the compiler sinks each into its branch below and the branches
  // wait one after the other.  I is LPR * NL * 8 for every instantiation (the launcher's shapes).
  constexpr size_t row_b = static_cast<size_t>(LPR) * NL * 16;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int sub = lane / LPR, sl = lane - sub * LPR;
  uint32_t lo[MAXW], hi[MAXW];
  int32_t rq[MAXW];
#pragma unroll
  for (int q = 0; q < MAXW; ++q) {
    const uint64_t p = reinterpret_cast<uint64_t>(items.w(wave + 4 * q));
    lo[q] = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p));
    hi[q] = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p >> 32));
    rq[q] = __builtin_amdgcn_readfirstlane(items.rank(wave + 4 * q));
  }
  int n_s = __builtin_amdgcn_readfirstlane(items.n()), d_s = d;
  uint32_t off2_s = off2;
  asm volatile("" : "+s"(lo[0]), "+s"(hi[0]), "+s"(rq[0]), "+s"(lo[1]), "+s"(hi[1]), "+s"(rq[1]), "+s"(lo[2]),
               "+s"(hi[2]), "+s"(rq[2]), "+s"(n_s), "+s"(d_s), "+s"(off2_s));
  typedef const __attribute__((address_space(1))) uint8_t* global_bytes;
  const uint8_t* wq[MAXW];
#pragma unroll
  for (int q = 0; q < MAXW; ++q)   // back to global-memory pointers, so the loads stay global loads
    wq[q] = (const uint8_t*)reinterpret_cast<global_bytes>((static_cast<uint64_t>(hi[q]) << 32) | lo[q]);
  const int r0 = blockIdx.x * RPW;
  const int r = r0 + sub;
  const int rr = r < d_s ? r : r0;
  (void)I;
  uint4 a[MAXW][NL], xr[MAXW][NL];
#pragma unroll
  for (int q = 0; q < MAXW; ++q) {
    const int i = wave + 4 * q;
    if (i < n_s) t1_load<MODE_DOWN, LPR, NL>(wq[q], off2_s, off2_s, row_b, rr, sl, a[q], a[q]);
  }
#pragma unroll
  for (int q = 0; q < MAXW; ++q) {
    const int i = wave + 4 * q;
    if (i < n_s) t1_input<LPR, NL>(reinterpret_cast<const uint4*>(h + static_cast<size_t>(rq[q]) * row_b), sl, xr[q]);
  }
#pragma unroll
  for (int q = 0; q < MAXW; ++q) {
    const int i = wave + 4 * q;
    if (i >= n_s) continue;
    float acc0, acc1;
    t1_dot<MODE_DOWN, LPR, NL>(a[q], a[q], xr[q], acc0, acc1);
    if (sl == 0) o_lds[rq[q] * RPW + sub] = acc0;
  }
  __syncthreads();
  if (tid < RPW && r0 + tid < d) {
    float acc = 0.f;
    for (int j = 0; j < k; ++j) acc = fmaf(gates[j], o_lds[j * RPW + tid], acc);
    if (has_shared) acc += o_lds[k * RPW + tid];
    y[r0 + tid] = acc;
  }
}

// host-planned: the experts come with the launch
template <int LPR, int NL, int MAXW>
__global__ void __launch_bounds__(256) ffn_down_combine_t1(const FusedT1Items B, const uint8_t* __restrict__ h,
                                                           const float* __restrict__ gates, float* __restrict__ y,
                                                           int d, int I, int k, int has_shared, uint32_t off2) {
  __shared__ float o_lds[9 * 64];
  down_combine_t1<LPR, NL, MAXW>(ArgItems{B}, h, gates, y, d, I, k, has_shared, off2, o_lds);
}

// device-planned: the experts of the plan the device pager wrote (single-token items; the output
// row of token 0 is the rank)
template <int LPR, int NL, int MAXW>
__global__ void __launch_bounds__(256) ffn_down_combine_dev(const FfnBatch* __restrict__ P, const uint8_t* __restrict__ h,
                                                            const float* __restrict__ gates, float* __restrict__ y,
                                                            int d, int I, int k, int has_shared, uint32_t off2) {
  __shared__ float o_lds[9 * 64];
  down_combine_t1<LPR, NL, MAXW>(PlanItems{P}, h, gates, y, d, I, k, has_shared, off2, o_lds);
}

using T1Kernel = void (*)(const FfnT1Batch, const uint8_t*, int, int, int, int, uint32_t, uint32_t, uint8_t*, int);

T1Kernel pick_t1(int mode, int lpr, int nl, bool one_pass) {
#define WISP_T1(M, L, N) \
  if (mode == M && lpr == L && nl == N) return one_pass ? &ffn_rows_t1<M, L, N, true> : &ffn_rows_t1<M, L, N, false>;
  WISP_T1(MODE_GATEUP, 64, 4) WISP_T1(MODE_GATEUP, 64, 8) WISP_T1(MODE_DOWN, 32, 3) WISP_T1(MODE_DOWN, 64, 28)
  WISP_T1(MODE_DOWN, 32, 1) WISP_T1(MODE_DOWN, 16, 1) WISP_T1(MODE_DOWN, 16, 3) WISP_T1(MODE_GATEUP, 32, 1)
  WISP_T1(MODE_GATEUP, 16, 3)
#undef WISP_T1
  return nullptr;
}

using RowsKernel = void (*)(const FfnBatch, const uint8_t*, int, int, int, int, int, uint32_t, uint32_t, uint32_t,
                            uint32_t, uint8_t*, int);

template <int WT, int IT, int MODE>
RowsKernel pick_kernel(int lpr, int nl) {
#define WISP_K(L, N) \
  if (lpr == L && nl == N) return &ffn_rows<WT, IT, MODE, L, N>;
  // shapes of the benchmarked and tested workloads, fully unrolled
  if constexpr (WT == DT_F32) {
    WISP_K(64, 1) WISP_K(64, 2)
  } else if constexpr (WT == DT_BF16) {
    WISP_K(64, 4) WISP_K(64, 8) WISP_K(32, 3) WISP_K(64, 28) WISP_K(32, 1) WISP_K(16, 1) WISP_K(16, 3)
  } else {
    WISP_K(64, 7) WISP_K(64, 2) WISP_K(16, 1)
  }
  // any other shape: runtime chunk count
  WISP_K(64, 0) WISP_K(32, 0) WISP_K(16, 0) WISP_K(8, 0)
#undef WISP_K
  return nullptr;
}

int pick_lpr(int chunks) {
  if (chunks % 64 == 0) return 64;
  if (chunks % 32 == 0) return 32;
  if (chunks % 16 == 0) return 16;
  if (chunks % 8 == 0) return 8;
  return 0;
}

hipError_t launch_rows(int mode, const FfnBatch& b, const FfnShape& s, const void* vin, int vin_stride, void* out,
                       int out_stride, hipStream_t st, const LaunchTiming& tm) {
  if (b.n_items <= 0) return hipSuccess;
  const BlobLayout& L = s.blob;
  const int WT = L.w_dtype;
  const int IT = mode == MODE_GATEUP ? s.x_dtype : s.h_dtype;
  const int K = mode == MODE_GATEUP ? L.d : L.I;
  const int R = mode == MODE_GATEUP ? L.I : L.d;
  const int EPL = WT == DT_F32 ? 4 : WT == DT_BF16 ? 8 : 16;
  if (K % EPL != 0) return hipErrorInvalidValue;
  const int chunks = K / EPL;
  const int lpr = pick_lpr(chunks);
  if (lpr == 0) return hipErrorInvalidValue;
  int nl = chunks / lpr;
  RowsKernel k = nullptr;
  auto pick = [&](int n) -> RowsKernel {
    if (WT == DT_F32 && IT == DT_F32)
      return mode == MODE_GATEUP ? pick_kernel<DT_F32, DT_F32, MODE_GATEUP>(lpr, n)
                                 : pick_kernel<DT_F32, DT_F32, MODE_DOWN>(lpr, n);
    if (WT == DT_BF16 && IT == DT_BF16)
      return mode == MODE_GATEUP ? pick_kernel<DT_BF16, DT_BF16, MODE_GATEUP>(lpr, n)
                                 : pick_kernel<DT_BF16, DT_BF16, MODE_DOWN>(lpr, n);
    if (WT == DT_FP8 && IT == DT_BF16)
      return mode == MODE_GATEUP ? pick_kernel<DT_FP8, DT_BF16, MODE_GATEUP>(lpr, n)
                                 : pick_kernel<DT_FP8, DT_BF16, MODE_DOWN>(lpr, n);
    return nullptr;
  };
  k = pick(nl);
  if (!k) k = pick(0);
  if (!k) return hipErrorInvalidValue;

  const int rpw = 64 / lpr;
  const int step = 4 * rpw;  // rows per workgroup pass
  // about 2048 workgroups per launch (8 per CU), each a whole number of passes
  int bpi = (2048 + b.n_items - 1) / b.n_items;
  const int max_bpi = (R + step - 1) / step;
  if (bpi > max_bpi) bpi = max_bpi;
  if (bpi < 1) bpi = 1;
  int rows_per_wg = (R + bpi - 1) / bpi;
  rows_per_wg = (rows_per_wg + step - 1) / step * step;
  bpi = (R + rows_per_wg - 1) / rows_per_wg;

  const int isz = IT == DT_F32 ? 4 : 2;
  const size_t lds = static_cast<size_t>(b.max_ntok) * K * isz;
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (e != hipSuccess) return e;
  }
  const uint32_t off0 = static_cast<uint32_t>(mode == MODE_GATEUP ? L.off_w1 : L.off_w2);
  const uint32_t off1 = static_cast<uint32_t>(mode == MODE_GATEUP ? L.off_w3 : L.off_w2);
  if (b.max_ntok == 1 && WT == DT_BF16 && IT == DT_BF16) {
    if (T1Kernel k1 = pick_t1(mode, lpr, nl, rows_per_wg == step)) {
      FfnT1Batch t1;
      t1.n_items = b.n_items;
      for (int i = 0; i < b.n_items; ++i) {
        t1.w[i] = b.items[i].w;
        t1.row[i] = mode == MODE_GATEUP ? b.items[i].tok[0] : b.items[i].out[0];
        t1.out[i] = b.items[i].out[0];
      }
      dim3 grid(static_cast<unsigned>(bpi), static_cast<unsigned>(b.n_items)), block(256);
      hipExtLaunchKernelGGL(k1, grid, block, 0, st, tm.start, tm.stop, 0, t1, static_cast<const uint8_t*>(vin),
                            vin_stride, K, R, rows_per_wg, off0, off1, static_cast<uint8_t*>(out), out_stride);
      return hipGetLastError();
    }
  }
  const uint32_t soff0 = static_cast<uint32_t>(mode == MODE_GATEUP ? L.off_s1 : L.off_s2);
  const uint32_t soff1 = static_cast<uint32_t>(mode == MODE_GATEUP ? L.off_s3 : L.off_s2);
  dim3 grid(static_cast<unsigned>(b.n_items * bpi)), block(256);
  hipExtLaunchKernelGGL(k, grid, block, static_cast<uint32_t>(lds), st, tm.start, tm.stop, 0, b,
                        static_cast<const uint8_t*>(vin), vin_stride, K, R, rows_per_wg, bpi, off0, off1, soff0, soff1,
                        static_cast<uint8_t*>(out), out_stride);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ffn_gateup(const FfnBatch& b, const FfnShape& s, const void* x, void* h, hipStream_t st,
                             const LaunchTiming& tm) {
  return launch_rows(MODE_GATEUP, b, s, x, s.blob.d, h, s.blob.I, st, tm);
}

hipError_t launch_ffn_down(const FfnBatch& b, const FfnShape& s, const void* h, float* buf, hipStream_t st,
                           const LaunchTiming& tm) {
  return launch_rows(MODE_DOWN, b, s, h, s.blob.I, buf, s.blob.d, st, tm);
}

namespace {
// (lanes per row, 16-byte loads per lane) of the down rows of a single-token bf16 step, or false
bool dc_shape(const FfnShape& s, int* lpr, int* nl) {
  const BlobLayout& L = s.blob;
  if (L.w_dtype != DT_BF16 || s.h_dtype != DT_BF16 || L.I % 8) return false;
  *lpr = pick_lpr(L.I / 8);
  if (!*lpr) return false;
  *nl = L.I / 8 / *lpr;
  return (*lpr == 32 && *nl == 3) || (*lpr == 16 && *nl == 1) || (*lpr == 16 && *nl == 3) || (*lpr == 64 && *nl == 2);
}

template <int LPR, int NL>
hipError_t dc_launch(bool dev, const void* items, const FfnShape& s, const void* h, const float* gates, float* y, int k,
                     int has_shared, int max_items, hipStream_t st, const LaunchTiming& tm) {
  const BlobLayout& L = s.blob;
  const dim3 grid((L.d + 64 / LPR - 1) / (64 / LPR)), block(256);
  const uint32_t off2 = static_cast<uint32_t>(L.off_w2);
  // three experts per wave: a single-token step has at most k + 1 <= 9 experts
  if (max_items > 12) return hipErrorInvalidValue;
  if (dev)
    hipExtLaunchKernelGGL(ffn_down_combine_dev<LPR, NL, 3>, grid, block, 0, st, tm.start, tm.stop, 0,
                          static_cast<const FfnBatch*>(items), static_cast<const uint8_t*>(h), gates, y, L.d, L.I, k,
                          has_shared, off2);
  else
    hipExtLaunchKernelGGL(ffn_down_combine_t1<LPR, NL, 3>, grid, block, 0, st, tm.start, tm.stop, 0,
                          *static_cast<const FusedT1Items*>(items), static_cast<const uint8_t*>(h), gates, y, L.d, L.I,
                          k, has_shared, off2);
  return hipGetLastError();
}

hipError_t dc_dispatch(bool dev, const void* items, const FfnShape& s, const void* h, const float* gates, float* y,
                       int k, int has_shared, int max_items, hipStream_t st, const LaunchTiming& tm) {
  int lpr = 0, nl = 0;
  if (!dc_shape(s, &lpr, &nl)) return hipErrorNotSupported;
  if (max_items < 1 || max_items > 12 || k < 1 || k > 8) return hipErrorInvalidValue;
  if (lpr == 32 && nl == 3) return dc_launch<32, 3>(dev, items, s, h, gates, y, k, has_shared, max_items, st, tm);
  if (lpr == 16 && nl == 1) return dc_launch<16, 1>(dev, items, s, h, gates, y, k, has_shared, max_items, st, tm);
  if (lpr == 16 && nl == 3) return dc_launch<16, 3>(dev, items, s, h, gates, y, k, has_shared, max_items, st, tm);
  return dc_launch<64, 2>(dev, items, s, h, gates, y, k, has_shared, max_items, st, tm);
}
}  // namespace

bool down_combine_supported(const FfnShape& s) {
  int lpr = 0, nl = 0;
  return dc_shape(s, &lpr, &nl);
}

hipError_t launch_down_combine_t1(const FusedT1Items& items, const FfnShape& s, const void* h, const float* gates,
                                  float* y, int k, int has_shared, hipStream_t st, const LaunchTiming& tm) {
  if (items.n_items < 1 || items.n_items > kMaxItems) return hipErrorInvalidValue;
  for (int i = 0; i < items.n_items; ++i)
    if (items.rank[i] < 0 || items.rank[i] > k || (items.rank[i] == k && !has_shared)) return hipErrorInvalidValue;
  return dc_dispatch(false, &items, s, h, gates, y, k, has_shared, items.n_items, st, tm);
}

hipError_t launch_down_combine_dev(const FfnBatch* plan, int max_items, const FfnShape& s, const void* h,
                                   const float* gates, float* y, int k, int has_shared, hipStream_t st,
                                   const LaunchTiming& tm) {
  return dc_dispatch(true, plan, s, h, gates, y, k, has_shared, max_items, st, tm);
}

namespace {
// Shapes with a device-planned path: (w dtype, h dtype, d lanes/loads, I lanes/loads).
struct DevShape { int lpr_g, nl_g, lpr_d, nl_d; };
bool dev_shape(const FfnShape& s, DevShape* o) {
  const BlobLayout& L = s.blob;
  const int EPL = L.w_dtype == DT_F32 ? 4 : L.w_dtype == DT_BF16 ? 8 : 16;
  o->lpr_g = pick_lpr(L.d / EPL);
  o->lpr_d = pick_lpr(L.I / EPL);
  if (!o->lpr_g || !o->lpr_d) return false;
  o->nl_g = L.d / EPL / o->lpr_g;
  o->nl_d = L.I / EPL / o->lpr_d;
  return true;
}
}  // namespace

hipError_t launch_ffn_dev(const FfnBatch* plan, int max_items, const FfnShape& s, const void* x, void* h,
                          float* buf, bool with_down, hipStream_t st, const LaunchTiming& tm_gateup,
                          const LaunchTiming& tm_down) {
  const BlobLayout& L = s.blob;
  DevShape ds;
  if (!dev_shape(s, &ds)) return hipErrorNotSupported;
  const int WT = L.w_dtype, XT = s.x_dtype, HT = s.h_dtype;
  using GK = void (*)(const FfnBatch*, const uint8_t*, int, int, int, int, int, int, uint32_t, uint32_t, uint32_t,
                      uint32_t, uint32_t, uint32_t, uint8_t*);
  using DK = void (*)(const FfnBatch*, const uint8_t*, int, int, int, int, uint32_t, uint32_t, float*);
  GK gk = nullptr;
  DK dk = nullptr;
#define WISP_G(W, X, LP, N) \
  if (WT == W && XT == X && ds.lpr_g == LP && ds.nl_g == N) gk = &ffn_gateup_dev<W, X, LP, N>;
#define WISP_DD(W, X, LP, N) \
  if (WT == W && HT == X && ds.lpr_d == LP && ds.nl_d == N) dk = &ffn_down_dev<W, X, LP, N>;
  WISP_G(DT_BF16, DT_BF16, 64, 4)   // d = 2048
  WISP_G(DT_BF16, DT_BF16, 32, 1)   // d = 256
  WISP_G(DT_BF16, DT_BF16, 16, 3)   // d = 384
  WISP_G(DT_FP8, DT_BF16, 64, 7)    // d = 7168
  WISP_G(DT_FP8, DT_BF16, 16, 1)    // d = 256
  WISP_G(DT_F32, DT_F32, 64, 1)     // d = 256
  WISP_DD(DT_BF16, DT_BF16, 32, 3)  // I = 768
  WISP_DD(DT_BF16, DT_BF16, 16, 1)  // I = 128
  WISP_DD(DT_BF16, DT_BF16, 8, 3)   // I = 192
  WISP_DD(DT_FP8, DT_BF16, 64, 2)   // I = 2048
  WISP_DD(DT_FP8, DT_BF16, 16, 1)   // I = 256
  WISP_DD(DT_F32, DT_F32, 64, 2)    // I = 512
#undef WISP_G
#undef WISP_DD
  if (!gk || !dk) return hipErrorNotSupported;
  // gate/up: per item slot, one row pass per workgroup for resident experts, and at least the
  // streaming workgroups of a fault
  const int rows_hit = 4 * (64 / ds.lpr_g);
  const int fault_wgs = 32, copy_wgs = 16;
  int bpi = (L.I + rows_hit - 1) / rows_hit;
  if (bpi < fault_wgs + copy_wgs) bpi = fault_wgs + copy_wgs;
  const int xs = XT == DT_F32 ? 4 : 2, hs = HT == DT_F32 ? 4 : 2;
  const size_t lds_g = static_cast<size_t>(kMaxTokPerItem) * L.d * xs;
  if (lds_g > 64 * 1024) return hipErrorNotSupported;
  hipExtLaunchKernelGGL(gk, dim3(max_items * bpi), dim3(256), static_cast<uint32_t>(lds_g), st, tm_gateup.start,
                        tm_gateup.stop, 0, plan, static_cast<const uint8_t*>(x), L.d, L.I, bpi, rows_hit, fault_wgs,
                        copy_wgs, static_cast<uint32_t>(L.off_w1), static_cast<uint32_t>(L.off_w3),
                        static_cast<uint32_t>(L.off_s1), static_cast<uint32_t>(L.off_s3),
                        static_cast<uint32_t>(L.off_w2), static_cast<uint32_t>(L.bytes - L.off_w2),
                        static_cast<uint8_t*>(h));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !with_down) return e;
  // down: per item slot, one row pass per workgroup
  const int rows_d = 4 * (64 / ds.lpr_d);
  const int bpi_d = (L.d + rows_d - 1) / rows_d;
  const size_t lds_d = static_cast<size_t>(kMaxTokPerItem) * L.I * hs;
  if (lds_d > 64 * 1024) return hipErrorNotSupported;
  hipExtLaunchKernelGGL(dk, dim3(max_items * bpi_d), dim3(256), static_cast<uint32_t>(lds_d), st, tm_down.start,
                        tm_down.stop, 0, plan, static_cast<const uint8_t*>(h), L.d, L.I, bpi_d, rows_d,
                        static_cast<uint32_t>(L.off_w2), static_cast<uint32_t>(L.off_s2), buf);
  return hipGetLastError();
}

bool ffn_dev_supported(const FfnShape& s, int T, int k, int has_shared) {
  DevShape ds;
  if (!dev_shape(s, &ds)) return false;
  const BlobLayout& L = s.blob;
  const int WT = L.w_dtype;
  const bool g = (WT == DT_BF16 && ((ds.lpr_g == 64 && ds.nl_g == 4) || (ds.lpr_g == 32 && ds.nl_g == 1) ||
                                    (ds.lpr_g == 16 && ds.nl_g == 3))) ||
                 (WT == DT_FP8 && ((ds.lpr_g == 64 && ds.nl_g == 7) || (ds.lpr_g == 16 && ds.nl_g == 1))) ||
                 (WT == DT_F32 && ds.lpr_g == 64 && ds.nl_g == 1);
  const bool dn = (WT == DT_BF16 && ((ds.lpr_d == 32 && ds.nl_d == 3) || (ds.lpr_d == 16 && ds.nl_d == 1) ||
                                     (ds.lpr_d == 8 && ds.nl_d == 3))) ||
                  (WT == DT_FP8 && ((ds.lpr_d == 64 && ds.nl_d == 2) || (ds.lpr_d == 16 && ds.nl_d == 1))) ||
                  (WT == DT_F32 && ds.lpr_d == 64 && ds.nl_d == 2);
  const int hs = s.h_dtype == DT_F32 ? 4 : 2, xs = s.x_dtype == DT_F32 ? 4 : 2;
  (void)k;
  (void)has_shared;
  return g && dn && T <= kMaxTokPerItem && static_cast<size_t>(kMaxTokPerItem) * L.d * xs <= 64 * 1024 &&
         static_cast<size_t>(kMaxTokPerItem) * L.I * hs <= 64 * 1024;
}

// ------------------------------------------------------------------------------------------
// fp8 decode probe: the same conversion as the FFN kernels, for checking all codes on device.
// ------------------------------------------------------------------------------------------
namespace {
__global__ void decode_fp8_kernel(const uint8_t* __restrict__ codes, float* __restrict__ out, int n) {
  const int i = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i + 3 < n) {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(codes + i);
    float o[4];
    fp8x4(w, o);
    out[i] = o[0]; out[i + 1] = o[1]; out[i + 2] = o[2]; out[i + 3] = o[3];
  } else {
    for (int j = i; j < n; ++j) {
      float o[4];
      fp8x4(static_cast<uint32_t>(codes[j]), o);
      out[j] = o[0];
    }
  }
}
}  // namespace

hipError_t launch_decode_fp8(const uint8_t* codes, float* out, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int threads = (n + 3) / 4;
  hipLaunchKernelGGL(decode_fp8_kernel, dim3((threads + 255) / 256), dim3(256), 0, st, codes, out, n);
  return hipGetLastError();
}

}  // namespace wisp
