/*
 * lethe_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, sequential CPU reference for the Lethe decode/prune hot path
 * (Lethe: Layer- and Time-Adaptive KV Cache Pruning, arXiv 2511.06029).
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this file's library.  The product path never calls it and shares
 * no code, header, table or constant with it.
 *
 * Precision: inputs arrive as fp32 arrays (bf16 data widened exactly by the
 * caller); every arithmetic step here runs in fp64, except the one place where
 * the method turns a float into an integer (the budget weights), which is done
 * in fp32 exactly as specified below so both sides take that decision in the
 * same precision.  Build with -O2 -ffp-contract=off and without -ffast-math.
 *
 * Loops run in a fixed, documented order; nothing is blocked, fused or
 * reordered beyond the definitions cited at each function.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Decode attention with importance accumulation for one segment.
 *
 * One (layer, sequence, KV head) segment of n cached rows; G query heads share
 * this KV head (grouped-query attention: query head i reads KV head
 * floor(i / G), which is what the repeat-interleave of keys in Eq. 3 of
 * "Spatial KV Cache Pruning via Layerwise Sparsity Estimation" expresses).
 *
 * For each query head g (ascending), as plain softmax attention over the
 * cache (the decode step the paper's System Overview describes):
 *   x_j  = scale * sum_d q[g][d] * K[j][d]          (d ascending)
 *   m    = max_j x_j
 *   l    = sum_j exp(x_j - m)                         (j ascending)
 *   p_j  = exp(x_j - m) / l
 *   out[g][d] = sum_j p_j * V[j][d]                   (j ascending)
 * Importance update, Eq. 5 of the RASR section read per token j and summed over
 * the G query heads of this KV group:
 *   s_out[j] = gamma * s_in[j] + sum_g p_gj            (g ascending)
 *
 * q: [G][D], K and V: [n][D] (row-major), s_in: [n] or NULL (all zero),
 * s_out: [n], out: [G][D].  n == 0 gives out = 0 and touches nothing else.
 * Returns 0, or -1 if scratch memory could not be allocated.
 */
int lethe_oracle_attend(int64_t n, int D, int G, const float* q, const float* K,
                        const float* V, double scale, double gamma,
                        const double* s_in, double* s_out, double* out) {
  for (int g = 0; g < G; ++g)
    for (int d = 0; d < D; ++d) out[(int64_t)g * D + d] = 0.0;
  if (n <= 0) return 0;
  double* x = (double*)malloc(sizeof(double) * (size_t)n);
  if (!x) return -1;
  for (int64_t j = 0; j < n; ++j) s_out[j] = gamma * (s_in ? s_in[j] : 0.0);
  for (int g = 0; g < G; ++g) {
    const float* qg = q + (int64_t)g * D;
    for (int64_t j = 0; j < n; ++j) {
      double acc = 0.0;
      for (int d = 0; d < D; ++d) acc += (double)qg[d] * (double)K[j * D + d];
      x[j] = scale * acc;
    }
    double m = x[0];
    for (int64_t j = 1; j < n; ++j)
      if (x[j] > m || isnan(x[j])) m = x[j];
    double l = 0.0;
    for (int64_t j = 0; j < n; ++j) l += exp(x[j] - m);
    double* og = out + (int64_t)g * D;
    for (int64_t j = 0; j < n; ++j) {
      double p = exp(x[j] - m) / l;
      for (int d = 0; d < D; ++d) og[d] += p * (double)V[j * D + d];
      s_out[j] += p;
    }
  }
  free(x);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Hoyer sparsity, Eq. 1 of "Attention Sparsity as a Basis for Fine-Grained
 * Cache Management":
 *   S(a) = (sqrt(n) - ||a||_1 / ||a||_2) / (sqrt(n) - 1)
 * for a non-negative vector a of length n.  Degenerate cases, which the
 * equation leaves undefined: n <= 1 or ||a||_2 == 0 give 0.  The result is
 * clamped to [0, 1] with fmin/fmax, so a NaN result also becomes 0.
 */
double lethe_oracle_hoyer(int64_t n, const double* a) {
  if (n <= 1) return 0.0;
  double l1 = 0.0, l2sq = 0.0;
  for (int64_t j = 0; j < n; ++j) {
    l1 += fabs(a[j]);
    l2sq += a[j] * a[j];
  }
  if (!(l2sq > 0.0)) return 0.0;
  double rn = sqrt((double)n);
  double S = (rn - l1 / sqrt(l2sq)) / (rn - 1.0);
  return fmin(fmax(S, 0.0), 1.0);
}

/* Layer sparsity of one (layer, sequence): the per-token importance is the
 * head-summed score a_j = sum_h s[h][j] (Eq. 2 collapses attention over heads;
 * here over the H KV-head score vectors of the sequence, h ascending), and its
 * Hoyer sparsity (Eq. 1) is the layer's redundancy estimate.
 * s: [H][n] (head-major, each row the score vector of one KV head).
 */
double lethe_oracle_layer_sparsity(int64_t n, int H, const double* s) {
  if (n <= 1) return 0.0;
  double* a = (double*)malloc(sizeof(double) * (size_t)n);
  if (!a) return NAN;
  for (int64_t j = 0; j < n; ++j) {
    double acc = 0.0;
    for (int h = 0; h < H; ++h) acc += s[(int64_t)h * n + j];
    a[j] = acc;
  }
  double S = lethe_oracle_hoyer(n, a);
  free(a);
  return S;
}

/* ------------------------------------------------------------------------- */
/* Layerwise budget split for one sequence.  The paper assigns each layer a
 * token budget from its estimated attention redundancy (Abstract; "Spatial KV
 * Cache Pruning via Layerwise Sparsity Estimation") but prints no formula; this
 * is the reading used throughout this code base:
 *
 *   floors f_l = min(n_l, recent + sink), caps c_l = n_l.
 *   If sum n_l <= G_b: b_l = n_l (nothing to prune).
 *   Else if sum f_l > G_b: infeasible -> b_l = n_l and return 1.
 *   Else weights (density, higher for denser layers), computed in fp32:
 *       Sc  = S_l clamped to [0, 1] (NaN -> 0)
 *       w_l = 1 + (uint32) floorf((1.0f - Sc) * 16777216.0f)
 *     R = G_b - sum f_l over the active set A = { l : c_l > f_l }; b_l = f_l
 *     outside A.  Repeat:
 *       W = sum_{l in A} w_l;  q_l = floor(R * w_l / W)   (exact integers)
 *       if some l in A has f_l + q_l >= c_l: every such l gets b_l = c_l,
 *         R -= (c_l - f_l), l leaves A, and the loop repeats;
 *       else b_l = f_l + q_l for l in A, and the R - sum q_l leftover tokens
 *         go one each to the layers of A with the largest remainder
 *         (R * w_l mod W), ties to the lower layer index; stop.
 *   Result: sum b_l = G_b exactly and f_l <= b_l <= n_l.
 *
 * n, S, budget: [L].  Returns 0, or 1 when infeasible.
 */
int lethe_oracle_budget(int L, const int32_t* n, const float* S, int32_t recent,
                        int32_t sink, int64_t G_b, int32_t* budget) {
  int64_t sum_n = 0, sum_f = 0;
  int64_t f[256], c[256];
  uint64_t w[256];
  int active[256];
  if (L > 256) return -1;
  for (int l = 0; l < L; ++l) {
    int64_t nl = n[l] > 0 ? n[l] : 0;
    int64_t fl = (int64_t)recent + (int64_t)sink;
    if (fl > nl) fl = nl;
    f[l] = fl;
    c[l] = nl;
    sum_n += nl;
    sum_f += fl;
    float Sc = S[l];
    if (!(Sc >= 0.0f)) Sc = 0.0f;
    if (Sc > 1.0f) Sc = 1.0f;
    float scaled = (1.0f - Sc) * 16777216.0f;
    w[l] = 1u + (uint64_t)(uint32_t)floorf(scaled);
  }
  if (sum_n <= G_b) {
    for (int l = 0; l < L; ++l) budget[l] = (int32_t)c[l];
    return 0;
  }
  if (sum_f > G_b) {
    for (int l = 0; l < L; ++l) budget[l] = (int32_t)c[l];
    return 1;
  }
  uint64_t R = (uint64_t)(G_b - sum_f);
  for (int l = 0; l < L; ++l) {
    active[l] = c[l] > f[l];
    budget[l] = (int32_t)f[l];
  }
  for (;;) {
    uint64_t W = 0;
    for (int l = 0; l < L; ++l)
      if (active[l]) W += w[l];
    /* Every layer that reaches its cap in this pass is fixed at once; all
       quotas of the pass are taken against the same R and W. */
    int capped[256];
    int capped_any = 0;
    for (int l = 0; l < L; ++l) {
      capped[l] = 0;
      if (!active[l]) continue;
      uint64_t ql = (R * w[l]) / W;
      if ((uint64_t)f[l] + ql >= (uint64_t)c[l]) capped[l] = capped_any = 1;
    }
    if (capped_any) {
      uint64_t taken = 0;
      for (int l = 0; l < L; ++l) {
        if (!capped[l]) continue;
        budget[l] = (int32_t)c[l];
        taken += (uint64_t)(c[l] - f[l]);
        active[l] = 0;
      }
      R -= taken;
      continue;
    }
    uint64_t given = 0;
    uint64_t rem[256];
    for (int l = 0; l < L; ++l) {
      if (!active[l]) continue;
      uint64_t ql = (R * w[l]) / W;
      rem[l] = (R * w[l]) % W;
      budget[l] = (int32_t)(f[l] + (int64_t)ql);
      given += ql;
    }
    uint64_t left = R - given;
    /* Largest remainder first, ties to the lower layer index: repeatedly pick
       the best not-yet-chosen active layer. */
    int chosen[256];
    for (int l = 0; l < L; ++l) chosen[l] = 0;
    for (uint64_t t = 0; t < left; ++t) {
      int best = -1;
      for (int l = 0; l < L; ++l) {
        if (!active[l] || chosen[l]) continue;
        if (best < 0 || rem[l] > rem[best]) best = l;
      }
      chosen[best] = 1;
      budget[best] += 1;
    }
    break;
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* RASR retention for one segment (RASR section: tokens are ranked by their
 * accumulated score, the recent window and the boundary/sink tokens are always
 * kept, the rest compete for what is left of the layer's budget; the sink and
 * recent index sets follow Algorithm 1's sink_indices and recent_indices).
 *
 *   k' = max(k, 0).  If k' >= n: keep everything.
 *   r' = min(recent, k'), s' = min(sink, k' - r'), m = k' - r' - s'.
 *   Keep [0, s') and [n - r', n); among the candidates [s', n - r') keep the
 *   first m in the order (score descending, index ascending), where +0 and -0
 *   compare equal and NaN ranks after every number.
 *
 * s: [n] fp32 scores, keep: [n] output (1 keep, 0 evict).
 */
typedef struct {
  float v;
  int64_t j;
} cand_t;

static int cand_cmp(const void* pa, const void* pb) {
  const cand_t* a = (const cand_t*)pa;
  const cand_t* b = (const cand_t*)pb;
  int na = isnan(a->v), nb = isnan(b->v);
  if (na != nb) return na ? 1 : -1;
  if (!na) {
    if (a->v > b->v) return -1;
    if (a->v < b->v) return 1;
  }
  return (a->j < b->j) ? -1 : (a->j > b->j ? 1 : 0);
}

int lethe_oracle_select(int64_t n, const float* s, int64_t k, int32_t recent,
                        int32_t sink, uint8_t* keep) {
  if (k < 0) k = 0;
  if (k >= n) {
    for (int64_t j = 0; j < n; ++j) keep[j] = 1;
    return 0;
  }
  int64_t r = recent < k ? recent : k;
  int64_t sk = sink < (k - r) ? sink : (k - r);
  int64_t m = k - r - sk;
  for (int64_t j = 0; j < n; ++j) keep[j] = (j < sk || j >= n - r) ? 1 : 0;
  int64_t nc = (n - r) - sk;
  if (nc <= 0 || m <= 0) return 0;
  cand_t* cs = (cand_t*)malloc(sizeof(cand_t) * (size_t)nc);
  if (!cs) return -1;
  for (int64_t i = 0; i < nc; ++i) {
    cs[i].v = s[sk + i];
    cs[i].j = sk + i;
  }
  qsort(cs, (size_t)nc, sizeof(cand_t), cand_cmp);
  for (int64_t i = 0; i < m; ++i) keep[cs[i].j] = 1;
  free(cs);
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Selection score of the kept set that all KV heads of one (layer, sequence)
 * share.  Eq. 2 collapses attention over every head into one importance
 * vector per layer, and the GQA note after it (Eq. 3) makes that vector the
 * same for every KV head; here the per-head accumulated scores stand in for
 * the attention and are summed over heads:
 *   a_j = (...((s[0][j] + s[1][j]) + s[2][j]) + ...) + s[H-1][j]
 * in fp32, h ascending, rounded after every addition.  Ranking is a decision
 * on floats, so it is taken on exactly the fp32 values a device forms.
 * s: [H][n] fp32 (head-major), a: [n].
 */
void lethe_oracle_head_sum_f32(int64_t n, int H, const float* s, float* a) {
  for (int64_t j = 0; j < n; ++j) {
    float acc = s[j];
    for (int h = 1; h < H; ++h) acc = acc + s[(int64_t)h * n + j];
    a[j] = acc;
  }
}

/* ------------------------------------------------------------------------- */
/* Algorithm 1, Segmented Attention-Based Token Shrinking, for one score
 * vector of n tokens, together with the size trigger of the System Overview
 * (pruning starts once the cache holds more than L_evict tokens).
 *
 *   0. If n <= L_evict (negative L_evict counts as 0): nothing happens, every
 *      token is kept, L_evict is unchanged; returns -2.
 *   1. Rank all n tokens: top_values / top_indices in the order (value
 *      descending, index ascending), +0 and -0 equal, NaN after every number.
 *   2. Cut points c_d = floor(n * d / D) for d = 1, ..., D - 1, in that order.
 *   3. The breakpoint is the first cut point whose head-to-cut ratio
 *      top_values[0] / top_values[c] reaches tau.  The algorithm's test is
 *      printed as "<= tau" but the prose asks for the point where attention
 *      drops sharply, and with "<=" only the first cut could ever match (the
 *      ratio never decreases along the ranking); the reading here is ">=".
 *      The ratio is compared without rounding, as tau * v_cut <= v_head with
 *      both sides widened to fp64 (a product of two fp32 values is exact
 *      there).  An undefined ratio is not a breakpoint: a head that is not
 *      positive (0, negative, NaN) or a NaN cut value.
 *   4. Sink indices [0, sink) and recent indices [n - recent, n), clipped to
 *      [0, n).
 *   5. With a breakpoint c: the kept set is sink U top_indices[0 .. c) U
 *      recent, and L_evict <- max(L_evict, c + recent).  Without one the
 *      algorithm leaves the retained set unassigned and the prose says
 *      pruning is delayed: every token is kept and L_evict <- 2 * L_evict.
 *      L_evict saturates at 2^31 - 1.
 *
 * a: [n] fp32 scores, keep: [n] output (1 keep, 0 evict), L_evict: in/out.
 * Returns the breakpoint (>= 0), -1 (no breakpoint), -2 (not triggered), or
 * -3 if scratch memory could not be allocated.
 */
int64_t lethe_oracle_shrink(int64_t n, const float* a, int32_t D, float tau, int32_t recent,
                            int32_t sink, int32_t* L_evict, uint8_t* keep) {
  int64_t Lev = *L_evict > 0 ? *L_evict : 0;
  if (n <= Lev) {
    for (int64_t j = 0; j < n; ++j) keep[j] = 1;
    *L_evict = (int32_t)Lev;
    return -2;
  }
  cand_t* top = (cand_t*)malloc(sizeof(cand_t) * (size_t)n);
  if (!top) return -3;
  for (int64_t j = 0; j < n; ++j) {
    top[j].v = a[j];
    top[j].j = j;
  }
  qsort(top, (size_t)n, sizeof(cand_t), cand_cmp);
  int64_t breakpoint = -1;
  for (int64_t d = 1; d <= (int64_t)D - 1; ++d) {
    int64_t c = (n * d) / D;
    double v_head = (double)top[0].v;
    double v_cut = (double)top[c].v;
    int defined = v_head > 0.0 && !isnan(v_cut);
    if (defined && (double)tau * v_cut <= v_head) {
      breakpoint = c;
      break;
    }
  }
  int64_t r = recent < n ? recent : n;
  int64_t sk = sink < n ? sink : n;
  if (breakpoint >= 0) {
    for (int64_t j = 0; j < n; ++j) keep[j] = (j < sk || j >= n - r) ? 1 : 0;
    for (int64_t i = 0; i < breakpoint; ++i) keep[top[i].j] = 1;
    int64_t next = breakpoint + (int64_t)recent;
    if (next > Lev) Lev = next;
  } else {
    for (int64_t j = 0; j < n; ++j) keep[j] = 1;
    Lev = 2 * Lev;
  }
  if (Lev > 2147483647) Lev = 2147483647;
  *L_evict = (int32_t)Lev;
  free(top);
  return breakpoint;
}

/* ------------------------------------------------------------------------- */
/* Prefill attention with score seeding for one segment: the qlen newest of
 * the segment's n cached rows come with queries (a prompt, or one chunk of
 * it).  Query i sits at position p = n - qlen + i and attends, causally, to
 * rows 0 .. p.  For each query head g of the KV group (ascending) and each
 * query i (ascending), as plain softmax attention:
 *   x_j  = scale * sum_d q[i][g][d] * K[j][d]          (d ascending), j <= p
 *   m    = max_j x_j,  l = sum_j exp(x_j - m),  p_j = exp(x_j - m) / l
 *   out[i][g][d] = sum_j p_j * V[j][d]                  (j ascending)
 * and the importance of Eq. 2 (attention summed over query heads and query
 * positions, here over the G heads of the group and the qlen queries):
 *   s_out[j] = s_in[j] + sum_g sum_i p_{g,i,j}          (g, then i ascending)
 * No decay between the queries of one call: they are one observation.
 *
 * q: [qlen][G][D], K and V: [n][D], s_in: [n] or NULL (zero), s_out: [n],
 * out: [qlen][G][D].  Requires 0 <= qlen <= n.  Returns 0, -1 on bad sizes,
 * -2 if scratch memory could not be allocated.
 */
int lethe_oracle_prefill(int64_t n, int64_t qlen, int D, int G, const float* q, const float* K,
                         const float* V, double scale, const double* s_in, double* s_out,
                         double* out) {
  if (qlen < 0 || qlen > n) return -1;
  for (int64_t j = 0; j < n; ++j) s_out[j] = s_in ? s_in[j] : 0.0;
  for (int64_t e = 0; e < qlen * G * D; ++e) out[e] = 0.0;
  if (qlen == 0) return 0;
  double* x = (double*)malloc(sizeof(double) * (size_t)n);
  if (!x) return -2;
  for (int g = 0; g < G; ++g) {
    for (int64_t i = 0; i < qlen; ++i) {
      const int64_t p = n - qlen + i;
      const float* qi = q + (i * G + g) * D;
      for (int64_t j = 0; j <= p; ++j) {
        double acc = 0.0;
        for (int d = 0; d < D; ++d) acc += (double)qi[d] * (double)K[j * D + d];
        x[j] = scale * acc;
      }
      double m = x[0];
      for (int64_t j = 1; j <= p; ++j)
        if (x[j] > m || isnan(x[j])) m = x[j];
      double l = 0.0;
      for (int64_t j = 0; j <= p; ++j) l += exp(x[j] - m);
      double* oi = out + (i * G + g) * D;
      for (int64_t j = 0; j <= p; ++j) {
        double pj = exp(x[j] - m) / l;
        for (int d = 0; d < D; ++d) oi[d] += pj * (double)V[j * D + d];
        s_out[j] += pj;
      }
    }
  }
  free(x);
  return 0;
}
