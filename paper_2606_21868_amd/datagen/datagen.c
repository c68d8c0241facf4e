/*
 * Seeded synthetic inputs for the paged MoE layer.
 *
 * This module only produces input bytes: expert weights, router weights and hidden states.
 * It holds none of the MoE method's arithmetic.  Both the HIP path and the CPU oracle read
 * the bytes it writes; neither links against the other.
 *
 * Random numbers: Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3" (SC'11).  Every value is a pure function of
 * (seed, tensor kind, layer, expert, element index), so any expert can be regenerated alone and
 * generation parallelises over any partition.
 *   key     = (seed, kind << 24 | layer << 12 | expert)
 *   counter = (q mod 2^32, q >> 32, 0, 0) for element block q = index / 4
 * The four 32-bit outputs of block q feed two Box-Muller pairs, giving the normals of
 * elements 4q .. 4q+3.  Box-Muller's log/sin/cos are evaluated with fixed fp32 polynomials
 * (series of atanh, sin and cos on reduced ranges) so the bytes do not depend on the host's
 * libm or CPU features.  The series truncation errors are below 1e-8; the resulting normals
 * are fp32 values, clipped at |z| <= 5.77 by the 23-bit uniform.
 *
 * Encodings, written from the format definitions:
 *   bf16: the upper 16 bits of an IEEE binary32 value after round-to-nearest-even.
 *   fp8 E4M3FN (OCP 8-bit floating point, 2023): 1 sign, 4 exponent bits (bias 7), 3 mantissa
 *   bits, subnormals, no infinities, S.1111.111 = NaN, largest finite 448.  Encoding rounds to
 *   nearest-even and saturates to +-448.
 * fp8 block quantisation: each 128x128 block gets a bf16 scale s = bf16(amax / 448) (1.0 for an
 * all-zero block) and codes q = e4m3(w / s); a weight then decodes as e4m3(q) * s.
 */
#include <stdint.h>
#include <string.h>
#include <stdlib.h>
#include <math.h>
#include <immintrin.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------------------------ */
/* Philox4x32-10                                                                               */
/* ------------------------------------------------------------------------------------------ */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void wdg_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
    uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    uint32_t n1 = (uint32_t)p1;
    uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    uint32_t n3 = (uint32_t)p0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += PHILOX_W0; k1 += PHILOX_W1;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Tensor kinds used in the key. */
enum { WDG_W1 = 1, WDG_W3 = 2, WDG_W2 = 3, WDG_WR = 4, WDG_XAR = 5, WDG_XIID = 6 };
#define WDG_SHARED_EXPERT 4095

static inline uint32_t make_key1(int kind, int layer, int expert) {
  return ((uint32_t)kind << 24) | (((uint32_t)layer & 0xFFFu) << 12) | ((uint32_t)expert & 0xFFFu);
}

/* 16 Philox blocks (64 normals) starting at block q0, AVX2, 8 blocks per vector.
 * 32x32->64 products: _mm256_mul_epu32 on even lanes and on odd lanes shifted down. */
#define NB 16
static inline void mulhilo8(__m256i a, __m256i m, __m256i* hi, __m256i* lo) {
  __m256i pe = _mm256_mul_epu32(a, m);
  __m256i po = _mm256_mul_epu32(_mm256_srli_epi64(a, 32), m);
  *lo = _mm256_blend_epi32(pe, _mm256_slli_epi64(po, 32), 0xAA);
  *hi = _mm256_blend_epi32(_mm256_srli_epi64(pe, 32), po, 0xAA);
}

/* Box-Muller on 8 uniform pairs: zc = r cos(theta), zs = r sin(theta). */
static inline void box_muller8(__m256i ua, __m256i ub, __m256* zc, __m256* zs) {
  const __m256 half = _mm256_set1_ps(0.5f), one = _mm256_set1_ps(1.0f), two = _mm256_set1_ps(2.0f);
  /* u1 = ((ua >> 9) + 0.5) * 2^-23 in [2^-24, 1 - 2^-24], exact */
  __m256 u1 = _mm256_mul_ps(_mm256_add_ps(_mm256_cvtepi32_ps(_mm256_srli_epi32(ua, 9)), half),
                            _mm256_set1_ps(1.0f / 8388608.0f));
  __m256i bits = _mm256_castps_si256(u1);
  __m256i e = _mm256_sub_epi32(_mm256_srli_epi32(bits, 23), _mm256_set1_epi32(127));
  __m256 m = _mm256_castsi256_ps(_mm256_or_si256(_mm256_and_si256(bits, _mm256_set1_epi32(0x007FFFFF)),
                                                 _mm256_set1_epi32(0x3F800000)));
  __m256 big = _mm256_cmp_ps(m, _mm256_set1_ps(1.41421356237309505f), _CMP_GT_OQ);
  m = _mm256_blendv_ps(m, _mm256_mul_ps(m, half), big);
  e = _mm256_sub_epi32(e, _mm256_castps_si256(big));          /* mask is -1 where big */
  __m256 s = _mm256_div_ps(_mm256_sub_ps(m, one), _mm256_add_ps(m, one));
  __m256 s2 = _mm256_mul_ps(s, s);
  __m256 p = _mm256_set1_ps(1.0f / 9.0f);
  p = _mm256_add_ps(_mm256_mul_ps(p, s2), _mm256_set1_ps(1.0f / 7.0f));
  p = _mm256_add_ps(_mm256_mul_ps(p, s2), _mm256_set1_ps(1.0f / 5.0f));
  p = _mm256_add_ps(_mm256_mul_ps(p, s2), _mm256_set1_ps(1.0f / 3.0f));
  p = _mm256_add_ps(_mm256_mul_ps(p, s2), one);
  __m256 lnm = _mm256_mul_ps(_mm256_mul_ps(two, s), p);
  __m256 lnu = _mm256_add_ps(_mm256_mul_ps(_mm256_cvtepi32_ps(e), _mm256_set1_ps(0.693147180559945309f)), lnm);
  __m256 r = _mm256_sqrt_ps(_mm256_mul_ps(_mm256_set1_ps(-2.0f), lnu));
  /* theta = 2 pi u2 = q pi/2 + pi/4 + phi, q = top two bits, phi in [-pi/4, pi/4) */
  __m256i q = _mm256_srli_epi32(ub, 30);
  __m256 f = _mm256_mul_ps(_mm256_cvtepi32_ps(_mm256_and_si256(_mm256_srli_epi32(ub, 8), _mm256_set1_epi32(0x3FFFFF))),
                           _mm256_set1_ps(1.0f / 4194304.0f));
  __m256 phi = _mm256_mul_ps(_mm256_sub_ps(f, half), _mm256_set1_ps(1.57079632679489662f));
  __m256 p2 = _mm256_mul_ps(phi, phi);
  __m256 sp = _mm256_set1_ps(1.0f / 362880.0f);
  sp = _mm256_sub_ps(_mm256_set1_ps(1.0f / 5040.0f), _mm256_mul_ps(p2, sp));
  sp = _mm256_sub_ps(_mm256_set1_ps(1.0f / 120.0f), _mm256_mul_ps(p2, sp));
  sp = _mm256_sub_ps(_mm256_set1_ps(1.0f / 6.0f), _mm256_mul_ps(p2, sp));
  sp = _mm256_sub_ps(one, _mm256_mul_ps(p2, sp));
  sp = _mm256_mul_ps(phi, sp);
  __m256 cp = _mm256_set1_ps(1.0f / 3628800.0f);
  cp = _mm256_sub_ps(_mm256_set1_ps(1.0f / 40320.0f), _mm256_mul_ps(p2, cp));
  cp = _mm256_sub_ps(_mm256_set1_ps(1.0f / 720.0f), _mm256_mul_ps(p2, cp));
  cp = _mm256_sub_ps(_mm256_set1_ps(1.0f / 24.0f), _mm256_mul_ps(p2, cp));
  cp = _mm256_sub_ps(half, _mm256_mul_ps(p2, cp));
  cp = _mm256_sub_ps(one, _mm256_mul_ps(p2, cp));
  const __m256 rs = _mm256_set1_ps(0.707106781186547524f);
  __m256 sa = _mm256_mul_ps(_mm256_add_ps(sp, cp), rs);   /* sin(pi/4 + phi) */
  __m256 ca = _mm256_mul_ps(_mm256_sub_ps(cp, sp), rs);   /* cos(pi/4 + phi) */
  /* quadrant rotation: q=0 (sa, ca), 1 (ca, -sa), 2 (-sa, -ca), 3 (-ca, sa) as (sin, cos) */
  __m256 odd = _mm256_castsi256_ps(_mm256_cmpeq_epi32(_mm256_and_si256(q, _mm256_set1_epi32(1)), _mm256_set1_epi32(1)));
  __m256 st = _mm256_blendv_ps(sa, ca, odd);
  __m256 ct = _mm256_blendv_ps(ca, sa, odd);
  __m256i sgn_s = _mm256_slli_epi32(_mm256_srli_epi32(q, 1), 31);                              /* q >= 2 */
  __m256i sgn_c = _mm256_slli_epi32(_mm256_and_si256(_mm256_xor_si256(q, _mm256_srli_epi32(q, 1)),
                                                     _mm256_set1_epi32(1)), 31);              /* q = 1, 2 */
  st = _mm256_xor_ps(st, _mm256_castsi256_ps(sgn_s));
  ct = _mm256_xor_ps(ct, _mm256_castsi256_ps(sgn_c));
  *zc = _mm256_mul_ps(r, ct);
  *zs = _mm256_mul_ps(r, st);
}

static void normals64(uint32_t seed, uint32_t key1, uint64_t q0, float* z) {
  const __m256i M0 = _mm256_set1_epi32((int)PHILOX_M0), M1 = _mm256_set1_epi32((int)PHILOX_M1);
  for (int g = 0; g < NB / 8; ++g) {
    uint32_t lo[8], hi[8];
    for (int i = 0; i < 8; ++i) {
      uint64_t q = q0 + (uint64_t)(g * 8 + i);
      lo[i] = (uint32_t)q; hi[i] = (uint32_t)(q >> 32);
    }
    __m256i c0 = _mm256_loadu_si256((const __m256i*)lo);
    __m256i c1 = _mm256_loadu_si256((const __m256i*)hi);
    __m256i c2 = _mm256_setzero_si256(), c3 = _mm256_setzero_si256();
    uint32_t k0 = seed, k1 = key1;
    for (int r = 0; r < 10; ++r) {
      __m256i hi0, lo0, hi1, lo1;
      mulhilo8(c0, M0, &hi0, &lo0);
      mulhilo8(c2, M1, &hi1, &lo1);
      __m256i n0 = _mm256_xor_si256(_mm256_xor_si256(hi1, c1), _mm256_set1_epi32((int)k0));
      __m256i n2 = _mm256_xor_si256(_mm256_xor_si256(hi0, c3), _mm256_set1_epi32((int)k1));
      c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
      k0 += PHILOX_W0; k1 += PHILOX_W1;
    }
    __m256 zc0, zs0, zc1, zs1;
    box_muller8(c0, c1, &zc0, &zs0);
    box_muller8(c2, c3, &zc1, &zs1);
    float a[8], b[8], c[8], d[8];
    _mm256_storeu_ps(a, zc0); _mm256_storeu_ps(b, zs0); _mm256_storeu_ps(c, zc1); _mm256_storeu_ps(d, zs1);
    for (int i = 0; i < 8; ++i) {
      float* o = z + 4 * (g * 8 + i);
      o[0] = a[i]; o[1] = b[i]; o[2] = c[i]; o[3] = d[i];
    }
  }
}

/* Normals for elements [start, start + n) of stream (seed, kind, layer, expert). */
void wdg_normals(uint32_t seed, int kind, int layer, int expert, uint64_t start, uint64_t n, float* out) {
  uint32_t key1 = make_key1(kind, layer, expert);
  float buf[4 * NB];
  uint64_t i = 0;
  while (i < n) {
    uint64_t idx = start + i;
    uint64_t base = idx & ~(uint64_t)(4 * NB - 1);
    uint64_t off = idx - base;
    uint64_t take = 4 * NB - off;
    if (take > n - i) take = n - i;
    normals64(seed, key1, base / 4, buf);
    memcpy(out + i, buf + off, take * sizeof(float));
    i += take;
  }
}

/* ------------------------------------------------------------------------------------------ */
/* Encodings                                                                                   */
/* ------------------------------------------------------------------------------------------ */
static inline uint16_t f32_to_bf16_rne(float v) {
  uint32_t u; memcpy(&u, &v, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
static inline float bf16_bits_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16; float v; memcpy(&v, &u, 4); return v;
}

/* E4M3FN, round to nearest even, saturate to +-448; NaN input -> 0x7F.
 * Normal range (|v| >= 2^-6): round the binary32 significand to 3 bits on the bit pattern
 * (a carry moves into the exponent), then rebias 127 -> 7.  Below 2^-6 the code is the integer
 * rint(|v| * 2^9) (8 = the smallest normal), computed with the 2^23 addition trick. */
static inline uint8_t f32_to_e4m3_rne_sat(float v) {
  uint32_t u; memcpy(&u, &v, 4);
  uint8_t sign = (uint8_t)((u >> 24) & 0x80u);
  uint32_t a = u & 0x7FFFFFFFu;
  if (a > 0x7F800000u) return 0x7F;                       /* NaN */
  if (a >= 0x43E00000u) return sign | 0x7E;               /* |v| >= 448 */
  if (a >= 0x3C800000u) {                                 /* |v| >= 2^-6 */
    uint32_t r = a + 0x7FFFFu + ((a >> 20) & 1u);
    uint32_t code = (r >> 20) - ((127u - 7u) << 3);
    if (code > 0x7Eu) code = 0x7Eu;
    return sign | (uint8_t)code;
  }
  float af; memcpy(&af, &a, 4);
  float n = (af * 512.0f + 8388608.0f) - 8388608.0f;     /* exact scaling, RNE to integer */
  return sign | (uint8_t)n;
}

uint16_t wdg_f32_to_bf16(float v) { return f32_to_bf16_rne(v); }
uint8_t wdg_f32_to_e4m3(float v) { return f32_to_e4m3_rne_sat(v); }

void wdg_f32_to_bf16_array(const float* in, uint16_t* out, uint64_t n) {
  for (uint64_t i = 0; i < n; ++i) out[i] = f32_to_bf16_rne(in[i]);
}
void wdg_f32_to_e4m3_array(const float* in, uint8_t* out, uint64_t n) {
  for (uint64_t i = 0; i < n; ++i) out[i] = f32_to_e4m3_rne_sat(in[i]);
}

/* ------------------------------------------------------------------------------------------ */
/* Weight matrices                                                                             */
/* ------------------------------------------------------------------------------------------ */
/* dtype codes: 0 = fp32, 1 = bf16, 2 = fp8 E4M3 with bf16 scales per 128x128 block */

/* rows x cols row-major matrix, element (r,c) = std * z[r*cols + c]. */
void wdg_matrix_f32(uint32_t seed, int kind, int layer, int expert, int rows, int cols, float stdv, float* out) {
  wdg_normals(seed, kind, layer, expert, 0, (uint64_t)rows * cols, out);
  uint64_t n = (uint64_t)rows * cols;
  for (uint64_t i = 0; i < n; ++i) out[i] = stdv * out[i];
}

static void matrix_bf16_rows(uint32_t seed, int kind, int layer, int expert, int r0, int r1, int cols,
                             float stdv, uint16_t* out /* whole matrix */) {
  float* tmp = (float*)malloc(sizeof(float) * (size_t)cols);
  for (int r = r0; r < r1; ++r) {
    wdg_normals(seed, kind, layer, expert, (uint64_t)r * cols, (uint64_t)cols, tmp);
    uint16_t* o = out + (size_t)r * cols;
    for (int c = 0; c < cols; ++c) o[c] = f32_to_bf16_rne(stdv * tmp[c]);
  }
  free(tmp);
}

void wdg_matrix_bf16(uint32_t seed, int kind, int layer, int expert, int rows, int cols, float stdv, uint16_t* out) {
  matrix_bf16_rows(seed, kind, layer, expert, 0, rows, cols, stdv, out);
}

/* One 128x128 block (br, bc) of an fp8 matrix: codes into out (row-major, full matrix) and the
 * block's bf16 scale into scales[br * (cols/128) + bc]. */
static void matrix_fp8_block(uint32_t seed, int kind, int layer, int expert, int cols, int br, int bc,
                             float stdv, uint8_t* out, uint16_t* scales, float* tmp /* 128*128 */) {
  float amax = 0.0f;
  for (int rr = 0; rr < 128; ++rr) {
    int r = br * 128 + rr;
    float* t = tmp + rr * 128;
    wdg_normals(seed, kind, layer, expert, (uint64_t)r * cols + (uint64_t)bc * 128, 128, t);
    for (int c = 0; c < 128; ++c) {
      t[c] = stdv * t[c];
      float a = fabsf(t[c]);
      amax = a > amax ? a : amax;
    }
  }
  uint16_t sb = amax > 0.0f ? f32_to_bf16_rne(amax / 448.0f) : f32_to_bf16_rne(1.0f);
  float s = bf16_bits_to_f32(sb);
  scales[(size_t)br * (cols / 128) + bc] = sb;
  for (int rr = 0; rr < 128; ++rr) {
    uint8_t* o = out + (size_t)(br * 128 + rr) * cols + (size_t)bc * 128;
    const float* t = tmp + rr * 128;
    for (int c = 0; c < 128; ++c) o[c] = f32_to_e4m3_rne_sat(t[c] / s);
  }
}

void wdg_matrix_fp8(uint32_t seed, int kind, int layer, int expert, int rows, int cols, float stdv,
                    uint8_t* out, uint16_t* scales) {
  float* tmp = (float*)malloc(sizeof(float) * 128 * 128);
  for (int br = 0; br < rows / 128; ++br)
    for (int bc = 0; bc < cols / 128; ++bc)
      matrix_fp8_block(seed, kind, layer, expert, cols, br, bc, stdv, out, scales, tmp);
  free(tmp);
}

/* ------------------------------------------------------------------------------------------ */
/* Expert blobs                                                                                */
/* ------------------------------------------------------------------------------------------ */
/* Blob layout (a data format read independently by the HIP path and by the oracle):
 *   W1 [I, d] row-major | W3 [I, d] row-major | W2 [d, I] row-major
 *   fp8 only, after the codes: S1 [I/128, d/128] | S3 [I/128, d/128] | S2 [d/128, I/128], bf16.
 * Element sizes: fp32 4, bf16 2, fp8 1.  Weights ~ N(0, std^2) before encoding. */
uint64_t wdg_blob_bytes(int dtype, int d, int I) {
  uint64_t n = (uint64_t)d * I;
  if (dtype == 0) return 3 * n * 4;
  if (dtype == 1) return 3 * n * 2;
  return 3 * n + 2ull * 3ull * (uint64_t)(d / 128) * (uint64_t)(I / 128);
}

/* Work unit: one of the three matrices, rows [r0, r1) (fp8: block rows [r0/128, r1/128)). */
static void blob_part(uint32_t seed, int layer, int expert, int dtype, int d, int I, float stdv,
                      void* blob, int which, int r0, int r1, float* tmp) {
  int kind = which == 0 ? WDG_W1 : which == 1 ? WDG_W3 : WDG_W2;
  int rows = which == 2 ? d : I, cols = which == 2 ? I : d;
  uint64_t n = (uint64_t)d * I;
  if (dtype == 0) {
    float* m = (float*)blob + (uint64_t)which * n;
    for (int r = r0; r < r1; ++r) {
      wdg_normals(seed, kind, layer, expert, (uint64_t)r * cols, (uint64_t)cols, m + (uint64_t)r * cols);
      for (int c = 0; c < cols; ++c) m[(uint64_t)r * cols + c] *= stdv;
    }
  } else if (dtype == 1) {
    uint16_t* m = (uint16_t*)blob + (uint64_t)which * n;
    matrix_bf16_rows(seed, kind, layer, expert, r0, r1, cols, stdv, m);
  } else {
    uint8_t* m = (uint8_t*)blob + (uint64_t)which * n;
    uint64_t sblk = (uint64_t)(d / 128) * (uint64_t)(I / 128);
    uint16_t* sc = (uint16_t*)((uint8_t*)blob + 3 * n) + (uint64_t)which * sblk;
    for (int br = r0 / 128; br < r1 / 128; ++br)
      for (int bc = 0; bc < cols / 128; ++bc)
        matrix_fp8_block(seed, kind, layer, expert, cols, br, bc, stdv, m, sc, tmp);
  }
  (void)rows;
}

void wdg_expert_blob(uint32_t seed, int layer, int expert, int dtype, int d, int I, float stdv, void* blob) {
  float* tmp = (float*)malloc(sizeof(float) * 128 * 128);
  for (int which = 0; which < 3; ++which) {
    int rows = which == 2 ? d : I;
    blob_part(seed, layer, expert, dtype, d, I, stdv, blob, which, 0, rows, tmp);
  }
  free(tmp);
}

/* Fill many blobs in parallel.  blobs[i] receives expert experts[i] of layer layers[i]. */
void wdg_expert_blobs(uint32_t seed, int count, const int32_t* layers, const int32_t* experts, void* const* blobs,
                      int dtype, int d, int I, float stdv, int threads) {
  /* work units of 128 rows of one matrix */
  int units_I = (I + 127) / 128, units_d = (d + 127) / 128;
  int per_blob = 2 * units_I + units_d;
  int64_t total = (int64_t)count * per_blob;
#ifdef _OPENMP
  if (threads <= 0) threads = omp_get_max_threads();
#pragma omp parallel num_threads(threads)
#endif
  {
    float* tmp = (float*)malloc(sizeof(float) * 128 * 128);
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 4)
#endif
    for (int64_t u = 0; u < total; ++u) {
      int b = (int)(u / per_blob);
      int w = (int)(u % per_blob);
      int which, blk;
      if (w < units_I) { which = 0; blk = w; }
      else if (w < 2 * units_I) { which = 1; blk = w - units_I; }
      else { which = 2; blk = w - 2 * units_I; }
      int rows = which == 2 ? d : I;
      int r0 = blk * 128, r1 = r0 + 128 < rows ? r0 + 128 : rows;
      blob_part(seed, layers[b], experts[b], dtype, d, I, stdv, blobs[b], which, r0, r1, tmp);
    }
    free(tmp);
  }
  (void)threads;
}

/* Router weights W_r [N, d] fp32, std = d^-1/2. */
void wdg_router(uint32_t seed, int layer, int N, int d, float* out) {
  float stdv = (float)(1.0 / sqrt((double)d));
  wdg_matrix_f32(seed, WDG_WR, layer, 0, N, d, stdv, out);
}

/* ------------------------------------------------------------------------------------------ */
/* Hidden states                                                                               */
/* ------------------------------------------------------------------------------------------ */
/* AR(1) chain for (layer, batch row): x_0 = eps_0, x_t = rho x_{t-1} + sqrt(1 - rho^2) eps_t,
 * eps_t ~ N(0, I_d) from stream (seed, XAR, layer, row), element index t*d + i.  The chain is
 * carried in fp64; each x_t is stored rounded (via fp32) to the output dtype (0 fp32, 1 bf16).
 * out holds steps rows of d elements with row stride out_stride elements. */
void wdg_ar1_chain(uint32_t seed, int layer, int row, int steps, int d, double rho, int dtype,
                   void* out, int64_t out_stride) {
  double* h = (double*)malloc(sizeof(double) * (size_t)d);
  float* eps = (float*)malloc(sizeof(float) * (size_t)d);
  double a = sqrt(1.0 - rho * rho);
  for (int t = 0; t < steps; ++t) {
    wdg_normals(seed, WDG_XAR, layer, row, (uint64_t)t * d, (uint64_t)d, eps);
    for (int i = 0; i < d; ++i) h[i] = (t == 0) ? (double)eps[i] : rho * h[i] + a * (double)eps[i];
    if (dtype == 0) {
      float* o = (float*)out + (int64_t)t * out_stride;
      for (int i = 0; i < d; ++i) o[i] = (float)h[i];
    } else {
      uint16_t* o = (uint16_t*)out + (int64_t)t * out_stride;
      for (int i = 0; i < d; ++i) o[i] = f32_to_bf16_rne((float)h[i]);
    }
  }
  free(h); free(eps);
}

/* All AR(1) inputs of a decode run: out[l][t][b][:] for layers L, steps S, batch rows T. */
void wdg_decode_inputs(uint32_t seed, int L, int S, int T, int d, double rho, int dtype, void* out, int threads) {
  size_t es = dtype == 0 ? 4 : 2;
#ifdef _OPENMP
  if (threads <= 0) threads = omp_get_max_threads();
#pragma omp parallel for num_threads(threads) schedule(dynamic, 1) collapse(2)
#endif
  for (int l = 0; l < L; ++l)
    for (int b = 0; b < T; ++b) {
      char* base = (char*)out + (((size_t)l * S) * T + b) * d * es;
      wdg_ar1_chain(seed, l, b, S, d, rho, dtype, base, (int64_t)T * d);
    }
  (void)threads;
}

/* i.i.d. N(0, I) inputs for a prefill pass: out[l][t][:], stream (seed, XIID, layer, 0). */
void wdg_prefill_inputs(uint32_t seed, int L, int T, int d, int dtype, void* out, int threads) {
  size_t es = dtype == 0 ? 4 : 2;
#ifdef _OPENMP
  if (threads <= 0) threads = omp_get_max_threads();
#pragma omp parallel for num_threads(threads) schedule(dynamic, 1)
#endif
  for (int l = 0; l < L; ++l) {
    float* tmp = (float*)malloc(sizeof(float) * (size_t)T * d);
    wdg_normals(seed, WDG_XIID, l, 0, 0, (uint64_t)T * d, tmp);
    char* base = (char*)out + (size_t)l * T * d * es;
    if (dtype == 0) memcpy(base, tmp, sizeof(float) * (size_t)T * d);
    else wdg_f32_to_bf16_array(tmp, (uint16_t*)base, (uint64_t)T * d);
    free(tmp);
  }
  (void)threads;
}
