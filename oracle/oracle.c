/*
 * ORACLE — test infrastructure, not part of the product.
 *
 * A plain, slow, fp64 CPU reference for the paged MoE layer of WiSP (arXiv 2606.21868).
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no code, header, table or helper with the HIP path; the only thing both sides share is the
 * input bytes written by the seeded generator.
 *
 * What it computes:
 *  - The paper's exactness invariant (Sec. 3.2, the paragraph after Algorithm 1; Sec. 5.1) says
 *    paging changes where expert weights live, never the computation.  So the reference for the
 *    layer output is a plain fully resident MoE layer:
 *      router  z = W_r x, scores and top-k by routing variant (Sec. 3.1: layer l selects k of N
 *              experts per token; the variants are the three workload definitions),
 *      expert  o_e(x) = W2 (silu(W1 x) * (W3 x)),  silu(a) = a / (1 + e^-a),
 *      combine y = sum_j g_j o_{e_j}(x)  (+ the shared expert's output for shared-expert models).
 *    Everything is fp64; stored weights and inputs are decoded exactly, with no other rounding.
 *  - The pager itself: an LRU simulator that executes Algorithm 1 (WispLayer.Step) step by step
 *    on a per-layer state pi, pi^-1, tau, c with C slots (Sec. 3.2, "Expert-map indirection" and
 *    "Per-step protocol"; the cap C of Sec. 3.1).
 *
 * Readings where the paper is silent (each one is listed with its reason in the design notes):
 *  - Top-k order is (score desc, expert id asc); gates follow that rank order.
 *  - LRU victims are ordered (tau asc, slot asc); empty slots carry tau = 0; faults take victims
 *    in ascending expert id.  All experts of one step share the tick c (Algorithm 1, tick update).
 *  - A step's reference set R is the union of every token's selection at that layer.  When
 *    |R| > C it is processed as consecutive chunks of C experts: resident ids ascending, then
 *    non-resident ids ascending, each chunk one Algorithm 1 step.  (The paper groups tokens
 *    instead and notes its decode runs never take this path.)
 *  - Shrinking the cap keeps the most recently used experts (largest tau, ties to the lower
 *    slot) and renumbers kept slots in their old slot order; growing appends empty slots.
 *
 * Blob format read here (a data format, implemented independently on each side):
 *   W1 [I,d] | W3 [I,d] | W2 [d,I], row-major; fp8 adds S1 [I/128,d/128] | S3 | S2 [d/128,I/128]
 *   as bf16 after the codes.  dtype 0 = fp32, 1 = bf16, 2 = fp8 E4M3FN with 128x128 bf16 scales.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------------------------------- */
/* Stored-value decoders, from the format definitions.                                       */
/* ---------------------------------------------------------------------------------------- */

/* bfloat16: sign, 8 exponent bits (bias 127), 7 fraction bits; the upper half of binary32. */
double oracle_bf16_value(uint16_t b) {
  int s = (b >> 15) & 1;
  int e = (b >> 7) & 0xFF;
  int f = b & 0x7F;
  double v;
  if (e == 0xFF) v = f ? NAN : INFINITY;
  else if (e == 0) v = ldexp((double)f, -126 - 7);
  else v = ldexp(1.0 + (double)f / 128.0, e - 127);
  return s ? -v : v;
}

/* OCP FP8 E4M3FN: sign, 4 exponent bits (bias 7), 3 mantissa bits; subnormals; no infinities;
 * exponent 1111 with mantissa 111 is NaN; the largest finite value is 448. */
double oracle_e4m3_value(uint8_t b) {
  int s = (b >> 7) & 1;
  int e = (b >> 3) & 0xF;
  int m = b & 0x7;
  double v;
  if (e == 0xF && m == 0x7) v = NAN;
  else if (e == 0) v = ldexp((double)m / 8.0, 1 - 7);
  else v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return s ? -v : v;
}

static double load_x(int x_dtype, const void* x, size_t i) {
  if (x_dtype == 0) return (double)((const float*)x)[i];
  return oracle_bf16_value(((const uint16_t*)x)[i]);
}

/* Weight (r, c) of matrix `which` (0 W1, 1 W3, 2 W2) of an expert blob. */
static double blob_weight(const void* blob, int dtype, int d, int I, int which, int r, int c) {
  size_t n = (size_t)d * I;
  int cols = which == 2 ? I : d;
  size_t idx = (size_t)which * n + (size_t)r * cols + c;
  if (dtype == 0) return (double)((const float*)blob)[idx];
  if (dtype == 1) return oracle_bf16_value(((const uint16_t*)blob)[idx]);
  /* fp8: code times the bf16 scale of its 128x128 block */
  const uint8_t* q = (const uint8_t*)blob;
  size_t sblk = (size_t)(d / 128) * (size_t)(I / 128);
  const uint16_t* sc = (const uint16_t*)(q + 3 * n) + (size_t)which * sblk;
  double s = oracle_bf16_value(sc[(size_t)(r / 128) * (cols / 128) + (c / 128)]);
  return oracle_e4m3_value(q[idx]) * s;
}

/* ---------------------------------------------------------------------------------------- */
/* Router                                                                                    */
/* ---------------------------------------------------------------------------------------- */
enum { ROUTE_SOFTMAX_RENORM = 0, ROUTE_TOPK_SOFTMAX = 1, ROUTE_SIGMOID_GROUP = 2 };

/* Is (sa, a) ranked before (sb, b)?  Score descending, then id ascending. */
static int ranks_before(double sa, int a, double sb, int b) {
  return sa > sb || (sa == sb && a < b);
}

/* Top-k of score[] over the ids with allowed[e] != 0, ranked (score desc, id asc), by k plain
 * argmax passes.  Returns the number selected. */
static int select_topk(const double* score, const int* allowed, int N, int k, int32_t* out) {
  int* taken = (int*)calloc((size_t)N, sizeof(int));
  int n = 0;
  for (int j = 0; j < k; ++j) {
    int best = -1;
    for (int e = 0; e < N; ++e) {
      if (taken[e] || (allowed && !allowed[e])) continue;
      if (best < 0 || ranks_before(score[e], e, score[best], best)) best = e;
    }
    if (best < 0) break;
    taken[best] = 1;
    out[n++] = best;
  }
  free(taken);
  return n;
}

/* z = W_r x in fp64 and the selection score of every expert: p = softmax(z) (variant 0), z
 * itself (variant 1) or s = sigmoid(z) (variant 2). */
static void route_scores(int variant, int N, int d, const float* Wr, int x_dtype, const void* x, double* z,
                         double* sc) {
  for (int e = 0; e < N; ++e) {
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += (double)Wr[(size_t)e * d + c] * load_x(x_dtype, x, (size_t)c);
    z[e] = acc;
  }
  if (variant == ROUTE_SOFTMAX_RENORM) {
    double m = z[0];
    for (int e = 1; e < N; ++e) m = z[e] > m ? z[e] : m;
    double den = 0.0;
    for (int e = 0; e < N; ++e) den += exp(z[e] - m);
    for (int e = 0; e < N; ++e) sc[e] = exp(z[e] - m) / den;
  } else if (variant == ROUTE_TOPK_SOFTMAX) {
    for (int e = 0; e < N; ++e) sc[e] = z[e];
  } else {
    for (int e = 0; e < N; ++e) sc[e] = 1.0 / (1.0 + exp(-z[e]));
  }
}

/* Gates of the routed set idx[k] (in its rank order): softmax of the set's logits (variant 1),
 * else the set's scores renormalised to sum 1 (p for variant 0, s for variant 2). */
static void gates_of_set(int variant, const double* z, const double* sc, const int32_t* idx, int k,
                         double* gates) {
  if (variant == ROUTE_TOPK_SOFTMAX) {
    double m = z[idx[0]];
    for (int j = 1; j < k; ++j) m = z[idx[j]] > m ? z[idx[j]] : m;
    double den = 0.0;
    for (int j = 0; j < k; ++j) den += exp(z[idx[j]] - m);
    for (int j = 0; j < k; ++j) gates[j] = exp(z[idx[j]] - m) / den;
  } else {
    double den = 0.0;
    for (int j = 0; j < k; ++j) den += sc[idx[j]];
    for (int j = 0; j < k; ++j) gates[j] = sc[idx[j]] / den;
  }
}

/*
 * Route one token.  z = W_r x in fp64 (W_r [N, d] fp32).
 *   variant 0, softmax then renormalise: p = softmax(z) over all N; R = top-k of p;
 *             g_j = p_{e_j} / sum_i p_{e_i}.
 *   variant 1, softmax over the top-k logits: R = top-k of z; g = softmax(z_R).
 *   variant 2, sigmoid, group-limited: s = sigmoid(z); experts split into n_groups groups of
 *             N / n_groups consecutive ids; a group's score is the sum of its two largest s;
 *             keep the topk_groups best groups (score desc, group asc); R = top-k of s among the
 *             kept ids; g_j = s_{e_j} / sum_i s_{e_i}.
 * Outputs: idx[k] in rank order, gates[k]; sel_score[N] = the selection score of every expert
 * (p, z or s); margin = score of the k-th minus the (k+1)-th candidate (over allowed ids);
 * group_margin = 4th-vs-5th kept-group score gap for variant 2 (else +inf).
 */
void oracle_route(int variant, int N, int d, int k, int n_groups, int topk_groups, const float* Wr,
                  int x_dtype, const void* x, int32_t* idx, double* gates, double* sel_score,
                  double* margin, double* group_margin) {
  double* z = (double*)malloc(sizeof(double) * (size_t)N);
  double* sc = (double*)malloc(sizeof(double) * (size_t)N);
  route_scores(variant, N, d, Wr, x_dtype, x, z, sc);
  int* allowed = NULL;
  double gm = INFINITY;
  if (variant == ROUTE_SIGMOID_GROUP) {
    int gsize = N / n_groups;
    double* gscore = (double*)malloc(sizeof(double) * (size_t)n_groups);
    for (int g = 0; g < n_groups; ++g) {
      int32_t top2[2];
      int* in_g = (int*)calloc((size_t)N, sizeof(int));
      for (int e = g * gsize; e < (g + 1) * gsize; ++e) in_g[e] = 1;
      int n2 = select_topk(sc, in_g, N, 2, top2);
      gscore[g] = 0.0;
      for (int i = 0; i < n2; ++i) gscore[g] += sc[top2[i]];
      free(in_g);
    }
    int32_t* kept = (int32_t*)malloc(sizeof(int32_t) * (size_t)(topk_groups + 1));
    int nk = select_topk(gscore, NULL, n_groups, topk_groups + 1 <= n_groups ? topk_groups + 1 : topk_groups, kept);
    if (nk > topk_groups) gm = gscore[kept[topk_groups - 1]] - gscore[kept[topk_groups]];
    allowed = (int*)calloc((size_t)N, sizeof(int));
    for (int i = 0; i < topk_groups && i < nk; ++i)
      for (int e = kept[i] * gsize; e < (kept[i] + 1) * gsize; ++e) allowed[e] = 1;
    free(kept);
    free(gscore);
  }
  int32_t* sel = (int32_t*)malloc(sizeof(int32_t) * (size_t)(k + 1));
  int ns = select_topk(sc, allowed, N, k + 1, sel);
  for (int j = 0; j < k; ++j) idx[j] = sel[j];
  if (margin) *margin = ns > k ? sc[sel[k - 1]] - sc[sel[k]] : INFINITY;
  if (group_margin) *group_margin = gm;
  gates_of_set(variant, z, sc, idx, k, gates);
  if (sel_score) memcpy(sel_score, sc, sizeof(double) * (size_t)N);
  free(sel);
  free(allowed);
  free(sc);
  free(z);
}

/* ---------------------------------------------------------------------------------------- */
/* Expert FFN and layer                                                                      */
/* ---------------------------------------------------------------------------------------- */

/* o = W2 (silu(W1 x) * (W3 x)) in fp64 for one token.  h_out (optional, length I) gets h. */
void oracle_expert(const void* blob, int dtype, int d, int I, int x_dtype, const void* x, double* o,
                   double* h_out) {
  double* xv = (double*)malloc(sizeof(double) * (size_t)d);
  double* h = (double*)malloc(sizeof(double) * (size_t)I);
  for (int c = 0; c < d; ++c) xv[c] = load_x(x_dtype, x, (size_t)c);
#pragma omp parallel for schedule(static)
  for (int i = 0; i < I; ++i) {
    double a = 0.0, b = 0.0;
    for (int c = 0; c < d; ++c) {
      a += blob_weight(blob, dtype, d, I, 0, i, c) * xv[c];
      b += blob_weight(blob, dtype, d, I, 1, i, c) * xv[c];
    }
    h[i] = a / (1.0 + exp(-a)) * b;
  }
#pragma omp parallel for schedule(static)
  for (int r = 0; r < d; ++r) {
    double acc = 0.0;
    for (int i = 0; i < I; ++i) acc += blob_weight(blob, dtype, d, I, 2, r, i) * h[i];
    o[r] = acc;
  }
  if (h_out) memcpy(h_out, h, sizeof(double) * (size_t)I);
  free(h);
  free(xv);
}

/*
 * One fully resident MoE layer for T tokens: route each token, run its k chosen experts, combine
 * in rank order, then add the shared expert (weight 1) when shared_blob != NULL.
 * blobs[e] points at expert e's blob.  x is [T, d] (fp32 or bf16 bits).  Outputs idx, gates
 * [T, k]; y [T, d] fp64; margins [T] (may be NULL).
 */
void oracle_moe_layer(int variant, int N, int d, int I, int k, int n_groups, int topk_groups, int w_dtype,
                      const void* const* blobs, const void* shared_blob, const float* Wr, int x_dtype,
                      const void* x, int T, int32_t* idx, double* gates, double* y, double* margins,
                      double* group_margins) {
  size_t xs = x_dtype == 0 ? 4 : 2;
  double* o = (double*)malloc(sizeof(double) * (size_t)d);
  for (int t = 0; t < T; ++t) {
    const void* xt = (const char*)x + (size_t)t * d * xs;
    oracle_route(variant, N, d, k, n_groups, topk_groups, Wr, x_dtype, xt, idx + (size_t)t * k,
                 gates + (size_t)t * k, NULL, margins ? margins + t : NULL,
                 group_margins ? group_margins + t : NULL);
    double* yt = y + (size_t)t * d;
    for (int r = 0; r < d; ++r) yt[r] = 0.0;
    for (int j = 0; j < k; ++j) {
      oracle_expert(blobs[idx[(size_t)t * k + j]], w_dtype, d, I, x_dtype, xt, o, NULL);
      for (int r = 0; r < d; ++r) yt[r] += gates[(size_t)t * k + j] * o[r];
    }
    if (shared_blob) {
      oracle_expert(shared_blob, w_dtype, d, I, x_dtype, xt, o, NULL);
      for (int r = 0; r < d; ++r) yt[r] += o[r];
    }
  }
  free(o);
}

/* Gates of a given routed set idx[k] of one token (the rule of oracle_moe_layer_routed), without
 * the expert outputs. */
void oracle_route_gates(int variant, int N, int d, const float* Wr, int x_dtype, const void* x, int k,
                        const int32_t* idx, double* gates) {
  double* z = (double*)malloc(sizeof(double) * (size_t)N);
  double* sc = (double*)malloc(sizeof(double) * (size_t)N);
  route_scores(variant, N, d, Wr, x_dtype, x, z, sc);
  gates_of_set(variant, z, sc, idx, k, gates);
  free(sc);
  free(z);
}

/*
 * The same layer for a routed set given by the caller instead of the oracle's own selection:
 * idx [T, k] in rank order.  The gates follow the routing variant's rule applied to that set
 * (softmax of its logits for variant 1, its renormalised p or s otherwise), the combine runs in
 * the given rank order, and the shared expert is added as in oracle_moe_layer.  Used where two
 * selections are both correct (a near-tie at the k-th score): the output of the set a kernel chose
 * is then compared with this definition evaluated on that set.  Outputs gates [T, k], y [T, d].
 */
void oracle_moe_layer_routed(int variant, int N, int d, int I, int k, int w_dtype, const void* const* blobs,
                             const void* shared_blob, const float* Wr, int x_dtype, const void* x, int T,
                             const int32_t* idx, double* gates, double* y) {
  size_t xs = x_dtype == 0 ? 4 : 2;
  double* o = (double*)malloc(sizeof(double) * (size_t)d);
  double* z = (double*)malloc(sizeof(double) * (size_t)N);
  double* sc = (double*)malloc(sizeof(double) * (size_t)N);
  for (int t = 0; t < T; ++t) {
    const void* xt = (const char*)x + (size_t)t * d * xs;
    const int32_t* it = idx + (size_t)t * k;
    double* gt = gates + (size_t)t * k;
    route_scores(variant, N, d, Wr, x_dtype, xt, z, sc);
    gates_of_set(variant, z, sc, it, k, gt);
    double* yt = y + (size_t)t * d;
    for (int r = 0; r < d; ++r) yt[r] = 0.0;
    for (int j = 0; j < k; ++j) {
      oracle_expert(blobs[it[j]], w_dtype, d, I, x_dtype, xt, o, NULL);
      for (int r = 0; r < d; ++r) yt[r] += gt[j] * o[r];
    }
    if (shared_blob) {
      oracle_expert(shared_blob, w_dtype, d, I, x_dtype, xt, o, NULL);
      for (int r = 0; r < d; ++r) yt[r] += o[r];
    }
  }
  free(sc);
  free(z);
  free(o);
}

/* Output of one (token, expert) pair, for sampled checks at full size: y-contribution before
 * gating, i.e. o_e(x). */
void oracle_expert_output(const void* blob, int dtype, int d, int I, int x_dtype, const void* x, double* o) {
  oracle_expert(blob, dtype, d, I, x_dtype, x, o, NULL);
}

/* ---------------------------------------------------------------------------------------- */
/* LRU simulator: Algorithm 1 per layer                                                       */
/* ---------------------------------------------------------------------------------------- */
typedef struct {
  int N, C;
  int32_t* pi;     /* expert -> slot, -1 = not resident */
  int32_t* pinv;   /* slot -> expert, -1 = empty */
  uint64_t* tau;   /* slot -> tick of last use */
  uint64_t c;      /* clock */
} oracle_lru;

oracle_lru* oracle_lru_new(int N, int C) {
  if (N <= 0 || C <= 0 || C > N) return NULL;
  oracle_lru* s = (oracle_lru*)calloc(1, sizeof(oracle_lru));
  s->N = N; s->C = C;
  s->pi = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
  s->pinv = (int32_t*)malloc(sizeof(int32_t) * (size_t)C);
  s->tau = (uint64_t*)calloc((size_t)C, sizeof(uint64_t));
  for (int e = 0; e < N; ++e) s->pi[e] = -1;
  for (int i = 0; i < C; ++i) s->pinv[i] = -1;
  return s;
}

void oracle_lru_free(oracle_lru* s) {
  if (!s) return;
  free(s->pi); free(s->pinv); free(s->tau); free(s);
}

int oracle_lru_slot(const oracle_lru* s, int e) { return s->pi[e]; }
int oracle_lru_expert_in(const oracle_lru* s, int slot) { return s->pinv[slot]; }
uint64_t oracle_lru_tick(const oracle_lru* s, int slot) { return s->tau[slot]; }
uint64_t oracle_lru_clock(const oracle_lru* s) { return s->c; }
int oracle_lru_cap(const oracle_lru* s) { return s->C; }

static int cmp_int(const void* a, const void* b) {
  int x = *(const int*)a, y = *(const int*)b;
  return (x > y) - (x < y);
}

/* One Algorithm 1 step on the distinct ids G[0..g) (|G| <= C).  Appends each fault and its slot
 * to miss_ids / miss_slots (in assignment order) and returns the number of faults. */
static int alg1_step(oracle_lru* s, const int* G, int g, int32_t* miss_ids, int32_t* miss_slots) {
  /* faults M, ascending */
  int* M = (int*)malloc(sizeof(int) * (size_t)(g ? g : 1));
  int nm = 0;
  for (int i = 0; i < g; ++i) if (s->pi[G[i]] < 0) M[nm++] = G[i];
  qsort(M, (size_t)nm, sizeof(int), cmp_int);
  /* victims U: slots whose occupant is not in G (empty slots included), by (tau asc, slot asc);
   * selection by repeated minimum keeps this obviously ordered */
  int* inG = (int*)calloc((size_t)s->N, sizeof(int));
  for (int i = 0; i < g; ++i) inG[G[i]] = 1;
  int* used = (int*)calloc((size_t)s->C, sizeof(int));
  for (int i = 0; i < nm; ++i) {
    int best = -1;
    for (int sl = 0; sl < s->C; ++sl) {
      if (used[sl]) continue;
      if (s->pinv[sl] >= 0 && inG[s->pinv[sl]]) continue;
      if (best < 0 || s->tau[sl] < s->tau[best]) best = sl;
    }
    /* |G| <= C guarantees a victim exists */
    used[best] = 1;
    int old = s->pinv[best];
    if (old >= 0) s->pi[old] = -1;
    s->pi[M[i]] = best;
    s->pinv[best] = M[i];
    if (miss_ids) miss_ids[i] = M[i];
    if (miss_slots) miss_slots[i] = best;
  }
  /* clock and ticks */
  s->c += 1;
  for (int i = 0; i < g; ++i) s->tau[s->pi[G[i]]] = s->c;
  free(used);
  free(inG);
  free(M);
  return nm;
}

/*
 * One layer-step: R = the distinct ids among ids[0..n).  If |R| <= C this is one Algorithm 1
 * step; otherwise R is ordered (resident ascending, then non-resident ascending) and cut into
 * chunks of C, each one step.  Residency is judged once, at the start of the layer-step.
 * Outputs: hits, misses, chunks; miss_ids / miss_slots (capacity n) in assignment order.
 * Returns -1 on an id out of range.
 */
int oracle_lru_step(oracle_lru* s, const int32_t* ids, int n, int32_t* hits, int32_t* misses,
                    int32_t* chunks, int32_t* miss_ids, int32_t* miss_slots) {
  int* seen = (int*)calloc((size_t)s->N, sizeof(int));
  int* R = (int*)malloc(sizeof(int) * (size_t)(n ? n : 1));
  int nr = 0;
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= s->N) { free(seen); free(R); return -1; }
    if (!seen[ids[i]]) { seen[ids[i]] = 1; R[nr++] = ids[i]; }
  }
  int total_miss = 0, nchunks = 0;
  if (nr <= s->C) {
    total_miss = alg1_step(s, R, nr, miss_ids, miss_slots);
    nchunks = nr > 0 ? 1 : 0;
  } else {
    int* ord = (int*)malloc(sizeof(int) * (size_t)nr);
    int* res = (int*)malloc(sizeof(int) * (size_t)nr);
    int* non = (int*)malloc(sizeof(int) * (size_t)nr);
    int a = 0, b = 0;
    for (int i = 0; i < nr; ++i) {
      if (s->pi[R[i]] >= 0) res[a++] = R[i];
      else non[b++] = R[i];
    }
    qsort(res, (size_t)a, sizeof(int), cmp_int);
    qsort(non, (size_t)b, sizeof(int), cmp_int);
    memcpy(ord, res, sizeof(int) * (size_t)a);
    memcpy(ord + a, non, sizeof(int) * (size_t)b);
    for (int off = 0; off < nr; off += s->C) {
      int g = nr - off < s->C ? nr - off : s->C;
      total_miss += alg1_step(s, ord + off, g, miss_ids ? miss_ids + total_miss : NULL,
                              miss_slots ? miss_slots + total_miss : NULL);
      nchunks++;
    }
    free(ord); free(res); free(non);
  }
  *hits = nr - total_miss;
  *misses = total_miss;
  if (chunks) *chunks = nchunks;
  free(seen);
  free(R);
  return 0;
}

/*
 * Speculative prefetch (Sec. 4; the victim rule is this layer's Algorithm 1 rule, a reading: the
 * paper states only that speculative copies take slots and may evict experts still needed).
 * P = the distinct ids of ids[0..n) in the order given, keeping the first C.  Every id of P that is
 * not resident takes, in P's order, the not-yet-taken slot of smallest (tau, slot) among the slots
 * whose occupant is not in P (empty slots have tau = 0), evicting that occupant; its tick becomes
 * the current clock c.  No step is counted and c does not move.  fill_ids / fill_slots get the
 * copies in order.  Returns their count, or -1 on an id out of range (nothing changed).
 */
int oracle_lru_prefetch(oracle_lru* s, const int32_t* ids, int n, int32_t* fill_ids, int32_t* fill_slots) {
  if (n < 0) return -1;
  for (int i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= s->N) return -1;
  int* inP = (int*)calloc((size_t)s->N, sizeof(int));
  int* P = (int*)malloc(sizeof(int) * (size_t)(n ? n : 1));
  int np_ = 0;
  for (int i = 0; i < n && np_ < s->C; ++i)
    if (!inP[ids[i]]) { inP[ids[i]] = 1; P[np_++] = ids[i]; }
  int* taken = (int*)calloc((size_t)s->C, sizeof(int));
  int nf = 0;
  for (int i = 0; i < np_; ++i) {
    int e = P[i];
    if (s->pi[e] >= 0) continue;
    int best = -1;
    for (int sl = 0; sl < s->C; ++sl) {
      if (taken[sl]) continue;
      if (s->pinv[sl] >= 0 && inP[s->pinv[sl]]) continue;
      if (best < 0 || s->tau[sl] < s->tau[best]) best = sl;
    }
    /* |P| <= C: at least as many such slots as absent members of P */
    taken[best] = 1;
    if (s->pinv[best] >= 0) s->pi[s->pinv[best]] = -1;
    s->pi[e] = best;
    s->pinv[best] = e;
    s->tau[best] = s->c;
    if (fill_ids) fill_ids[nf] = e;
    if (fill_slots) fill_slots[nf] = best;
    nf++;
  }
  free(taken);
  free(P);
  free(inP);
  return nf;
}

/*
 * Change the cap to newC (1 <= newC <= N).  Shrink: keep the newC resident experts with the
 * largest tau (ties: lower slot first), renumber them 0.. in their old slot order, drop the rest.
 * Grow: keep every slot and append empty ones.  Ticks and the clock are kept.
 */
int oracle_lru_resize(oracle_lru* s, int newC) {
  if (newC <= 0 || newC > s->N) return -1;
  int32_t* pinv = (int32_t*)malloc(sizeof(int32_t) * (size_t)newC);
  uint64_t* tau = (uint64_t*)calloc((size_t)newC, sizeof(uint64_t));
  for (int i = 0; i < newC; ++i) pinv[i] = -1;
  if (newC >= s->C) {
    for (int i = 0; i < s->C; ++i) { pinv[i] = s->pinv[i]; tau[i] = s->tau[i]; }
  } else {
    int* keep = (int*)calloc((size_t)s->C, sizeof(int));
    for (int j = 0; j < newC; ++j) {
      int best = -1;
      for (int sl = 0; sl < s->C; ++sl) {
        if (keep[sl] || s->pinv[sl] < 0) continue;
        if (best < 0 || s->tau[sl] > s->tau[best]) best = sl;
      }
      if (best < 0) break;
      keep[best] = 1;
    }
    int n = 0;
    for (int sl = 0; sl < s->C; ++sl) {
      if (keep[sl]) { pinv[n] = s->pinv[sl]; tau[n] = s->tau[sl]; n++; }
    }
    free(keep);
  }
  for (int e = 0; e < s->N; ++e) s->pi[e] = -1;
  for (int i = 0; i < newC; ++i) if (pinv[i] >= 0) s->pi[pinv[i]] = i;
  free(s->pinv); free(s->tau);
  s->pinv = pinv; s->tau = tau; s->C = newC;
  return 0;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
