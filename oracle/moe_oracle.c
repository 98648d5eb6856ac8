/*
 * moe_oracle.c -- plain, slow CPU oracle of one split-expert MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or constant with the GPU library and must never be used as
 * a fallback for it.
 *
 * What it computes (arXiv 2509.08342, "MoEpic"):
 *   - the MoE module of Sec. 2.1, Eq. (2): router scores s = softmax(R(h)),
 *     the K experts with the highest scores, and the score-weighted sum of
 *     their outputs divided by the sum of the selected scores;
 *   - the speculative next-layer prediction of Sec. 3.2, Eq. (3): the next
 *     layer's router applied to the current layer's intermediate activation,
 *     experts ranked by descending predicted score;
 *   - the expert split of Sec. 2.3 / Sec. 3.1: an expert is cut into a top and a
 *     bottom segment whose results are combined ("concatenated") at compute
 *     time.  The cut runs along the FFN intermediate axis, so an expert's
 *     output is the sum of per-range outputs E^[lo,hi)(h).
 *
 * Precision.  Everything that produces a real-valued output is accumulated in
 * double precision.  The one floating-point quantity that decides an integer
 * (which experts are selected) is the router logit; it is computed in single
 * precision in a fixed, canonical summation order so that any other
 * implementation that follows the same order reaches the identical selection:
 *   partial[l] = fused-multiply-add accumulation, starting at +0, over
 *                j = l, l+64, l+128, ... (ascending), for l = 0..63;
 *   then for s = 32, 16, 8, 4, 2, 1: partial[l] = partial[l] + partial[l+s]
 *   for l < s; the logit is partial[0] (+ bias, added once afterwards).
 * This needs d to be a multiple of 64.  Selection takes the K largest logits;
 * equal logits go to the lower expert index.
 *
 * Layouts (all row-major, single precision; bf16 data is passed upcast, which
 * is exact):
 *   h      [T][d]         token activations
 *   w_r    [d][E]         router weight, logits = h . w_r
 *   w_gate [d][F], w_up [d][F], w_down [F][d]   one expert's SwiGLU FFN:
 *          E(h)[c] = sum_f silu(h.w_gate[:,f]) * (h.w_up[:,f]) * w_down[f][c]
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- router -- */

/* One router logit in the canonical single-precision order (see header).
 * The column e of w_r is read with stride E. */
static float canonical_logit(const float *h, const float *w_r, int d, int E,
                             int e) {
  float partial[64];
  for (int l = 0; l < 64; ++l) {
    float acc = 0.0f;
    for (int j = l; j < d; j += 64)
      acc = fmaf(h[j], w_r[(size_t)j * E + e], acc);
    partial[l] = acc;
  }
  for (int s = 32; s >= 1; s >>= 1)
    for (int l = 0; l < s; ++l)
      partial[l] = partial[l] + partial[l + s];
  return partial[0];
}

/* Router logits R(h) for T tokens (Sec. 2.1): logits[t][e] = h_t . w_r[:,e]
 * (+ bias[e] if bias is non-NULL).  Returns -1 if d is not a multiple of 64. */
int orc_router_logits(const float *h, const float *w_r, const float *bias,
                      int T, int d, int E, float *logits) {
  if (d % 64 != 0) return -1;
  for (int t = 0; t < T; ++t)
    for (int e = 0; e < E; ++e) {
      float v = canonical_logit(h + (size_t)t * d, w_r, d, E, e);
      if (bias) v = v + bias[e];
      logits[(size_t)t * E + e] = v;
    }
  return 0;
}

/* The value a logit is ranked and exponentiated by.  The paper never meets a
 * non-number; this implementation reads a NaN logit as minus infinity: the
 * expert ranks with the lowest logits (equal to -inf, so the lower index
 * first among them) and its softmax score is 0. */
static float rank_value(float v) { return isnan(v) ? -INFINITY : v; }

/* Top-K selection (Sec. 2.1: the K experts with the highest scores).  Since
 * softmax is monotone, ranking by logit ranks by score; ranking by logit also
 * keeps apart logits that exp() would round to equal scores.  K passes of
 * argmax, each taking the largest remaining logit, lowest index on ties.
 * idx[t][k] lists the selected experts in selection order. */
void orc_topk(const float *logits, int T, int E, int K, int32_t *idx) {
  unsigned char *taken = (unsigned char *)malloc((size_t)E);
  for (int t = 0; t < T; ++t) {
    const float *l = logits + (size_t)t * E;
    memset(taken, 0, (size_t)E);
    for (int k = 0; k < K; ++k) {
      int best = -1;
      for (int e = 0; e < E; ++e) {
        if (taken[e]) continue;
        if (best < 0 || rank_value(l[e]) > rank_value(l[best])) best = e;
      }
      taken[best] = 1;
      idx[(size_t)t * K + k] = best;
    }
  }
  free(taken);
}

/* softmax over E logits of one token, in double precision with the maximum
 * subtracted first (Sec. 2.1, s = softmax[R(h)]); NaN logits read as -inf. */
static void softmax_row(const float *l, int E, double *p) {
  double m = rank_value(l[0]);
  for (int e = 1; e < E; ++e)
    if (rank_value(l[e]) > m) m = rank_value(l[e]);
  double z = 0.0;
  for (int e = 0; e < E; ++e) {
    p[e] = exp((double)rank_value(l[e]) - m);
    z += p[e];
  }
  for (int e = 0; e < E; ++e) p[e] /= z;
}

/* Gate weights of Eq. (2): w[t][k] = s_{idx[t][k]} / sum_k' s_{idx[t][k']}.
 * With renormalize = 0 the plain score s_{idx[t][k]} is returned instead. */
void orc_gate_weights(const float *logits, const int32_t *idx, int T, int E,
                      int K, int renormalize, double *w) {
  double *p = (double *)malloc(sizeof(double) * (size_t)E);
  for (int t = 0; t < T; ++t) {
    softmax_row(logits + (size_t)t * E, E, p);
    double sel = 0.0;
    for (int k = 0; k < K; ++k) sel += p[idx[(size_t)t * K + k]];
    for (int k = 0; k < K; ++k) {
      double s = p[idx[(size_t)t * K + k]];
      w[(size_t)t * K + k] = renormalize ? s / sel : s;
    }
  }
  free(p);
}

/* ---------------------------------------------------------------- expert -- */

static double silu(double x) { return x / (1.0 + exp(-x)); }

/* Gate and up dot products of one token for units f in [lo,hi):
 * g[f-lo] = sum_j h[j] w_gate[j][f], u[f-lo] = sum_j h[j] w_up[j][f], each
 * summed over j in ascending order (rows of the weights are walked in
 * storage order, which does not change any sum). */
static void gate_up(const float *h, const float *w_gate, const float *w_up,
                    int d, int F, int lo, int hi, double *g, double *u) {
  int n = hi - lo;
  for (int i = 0; i < n; ++i) g[i] = u[i] = 0.0;
  for (int j = 0; j < d; ++j) {
    double hj = (double)h[j];
    const float *gr = w_gate + (size_t)j * F + lo;
    const float *ur = w_up + (size_t)j * F + lo;
    for (int i = 0; i < n; ++i) {
      g[i] += hj * (double)gr[i];
      u[i] += hj * (double)ur[i];
    }
  }
}

/* Range form of one expert for one token: acc[c] += sum_{f in [lo,hi)}
 * silu(h.G_f) * (h.U_f) * w_down[f][c], units f in ascending order.  Calling
 * it on [0,F) gives E(h); calling it on [0,F_top) and then on [F_top,F) with
 * the same accumulator reproduces E(h) exactly (the top segment's result
 * continued by the bottom's), which is how the split of Sec. 3.1 leaves the
 * output unchanged. */
void orc_expert_range(const float *h, const float *w_gate, const float *w_up,
                      const float *w_down, int d, int F, int lo, int hi,
                      double *acc) {
  if (hi <= lo) return;
  double *g = (double *)malloc(sizeof(double) * (size_t)(hi - lo));
  double *u = (double *)malloc(sizeof(double) * (size_t)(hi - lo));
  gate_up(h, w_gate, w_up, d, F, lo, hi, g, u);
  for (int f = lo; f < hi; ++f) {
    double a = silu(g[f - lo]) * u[f - lo];
    const float *dr = w_down + (size_t)f * d;
    for (int c = 0; c < d; ++c) acc[c] += a * (double)dr[c];
  }
  free(g);
  free(u);
}

/* The SwiGLU intermediate activations a_f = silu(h.G_f) * (h.U_f) of one
 * token for f in [lo,hi), written to a[f-lo]. */
void orc_expert_act(const float *h, const float *w_gate, const float *w_up,
                    int d, int F, int lo, int hi, double *a) {
  if (hi <= lo) return;
  double *g = (double *)malloc(sizeof(double) * (size_t)(hi - lo));
  double *u = (double *)malloc(sizeof(double) * (size_t)(hi - lo));
  gate_up(h, w_gate, w_up, d, F, lo, hi, g, u);
  for (int f = lo; f < hi; ++f) a[f - lo] = silu(g[f - lo]) * u[f - lo];
  free(g);
  free(u);
}

/* ----------------------------------------------------------------- layer -- */

/* The MoE module of Eq. (2) without the residual and the Norm: for each of
 * the T tokens, y_t = sum_k w[t][k] * E_{idx[t][k]}(h_t), k in selection
 * order, plus the n_shared always-active experts with weight 1 (an extension
 * for models that have them; n_shared = 0 is the paper's module).
 *
 * experts_gate/up/down are arrays of E pointers to each routed expert's
 * weights, shared_gate/up/down arrays of n_shared pointers (F_shared
 * intermediate units each).  y is [T][d] double. */
void orc_moe_combine(const float *h, int T, int d, int F, int K,
                     const int32_t *idx, const double *w,
                     const float *const *experts_gate,
                     const float *const *experts_up,
                     const float *const *experts_down, int n_shared,
                     int F_shared, const float *const *shared_gate,
                     const float *const *shared_up,
                     const float *const *shared_down, double *y) {
  double *tmp = (double *)malloc(sizeof(double) * (size_t)d);
  for (int t = 0; t < T; ++t) {
    const float *ht = h + (size_t)t * d;
    double *yt = y + (size_t)t * d;
    for (int c = 0; c < d; ++c) yt[c] = 0.0;
    for (int k = 0; k < K; ++k) {
      int e = idx[(size_t)t * K + k];
      for (int c = 0; c < d; ++c) tmp[c] = 0.0;
      orc_expert_range(ht, experts_gate[e], experts_up[e], experts_down[e], d,
                       F, 0, F, tmp);
      double wk = w[(size_t)t * K + k];
      for (int c = 0; c < d; ++c) yt[c] += wk * tmp[c];
    }
    for (int s = 0; s < n_shared; ++s) {
      for (int c = 0; c < d; ++c) tmp[c] = 0.0;
      orc_expert_range(ht, shared_gate[s], shared_up[s], shared_down[s], d,
                       F_shared, 0, F_shared, tmp);
      for (int c = 0; c < d; ++c) yt[c] += tmp[c];
    }
  }
  free(tmp);
}

/* ------------------------------------------------------------ prediction -- */

/* Speculative prediction of Eq. (3): scores of the next layer's experts from
 * the next layer's router applied to this layer's activation h.  For T > 1
 * tokens the per-token probabilities are summed (one ranking per layer pass).
 * score[e] (double) and order[E]: experts by descending score, lower index
 * first on equal scores.  logits_next [T][E] come from orc_router_logits with
 * the next layer's router weight. */
void orc_predict(const float *logits_next, int T, int E, double *score,
                 int32_t *order) {
  double *p = (double *)malloc(sizeof(double) * (size_t)E);
  for (int e = 0; e < E; ++e) score[e] = 0.0;
  for (int t = 0; t < T; ++t) {
    softmax_row(logits_next + (size_t)t * E, E, p);
    for (int e = 0; e < E; ++e) score[e] += p[e];
  }
  /* insertion sort on (-score, e): stable, so equal scores keep index order */
  for (int e = 0; e < E; ++e) order[e] = e;
  for (int i = 1; i < E; ++i) {
    int32_t v = order[i];
    int j = i - 1;
    while (j >= 0 && score[order[j]] < score[v]) {
      order[j + 1] = order[j];
      --j;
    }
    order[j + 1] = v;
  }
  free(p);
}

/* -------------------------------------------------------------- grouping -- */

/* Token-to-expert grouping: the T*K (token, k) slots, slot = t*K + k, sorted
 * stably by expert.  offsets[E+1] is the exclusive prefix sum of the per-
 * expert counts; perm[offsets[e] .. offsets[e+1]) lists the slots routed to
 * expert e in ascending slot order. */
void orc_group(const int32_t *idx, int T, int K, int E, int32_t *offsets,
               int32_t *perm) {
  for (int e = 0; e <= E; ++e) offsets[e] = 0;
  for (int s = 0; s < T * K; ++s) offsets[idx[s] + 1] += 1;
  for (int e = 0; e < E; ++e) offsets[e + 1] += offsets[e];
  int32_t *fill = (int32_t *)malloc(sizeof(int32_t) * (size_t)(E > 0 ? E : 1));
  for (int e = 0; e < E; ++e) fill[e] = offsets[e];
  for (int s = 0; s < T * K; ++s) perm[fill[idx[s]]++] = s;
  free(fill);
}

/* ------------------------------------------------------------------ glue -- */

/* Stack glue between two experts-only layers (Eqs. (1)-(2) with the attention
 * term taken as zero and a weightless RMS norm standing in for Norm):
 * out_t = x_t / sqrt(mean_c(x_t[c]^2) + eps) with x = h + y. */
void orc_residual_rmsnorm(const double *h, const double *y, int T, int d,
                          double eps, double *out) {
  for (int t = 0; t < T; ++t) {
    double ss = 0.0;
    for (int c = 0; c < d; ++c) {
      double x = h[(size_t)t * d + c] + y[(size_t)t * d + c];
      ss += x * x;
    }
    double inv = 1.0 / sqrt(ss / d + eps);
    for (int c = 0; c < d; ++c)
      out[(size_t)t * d + c] = (h[(size_t)t * d + c] + y[(size_t)t * d + c]) * inv;
  }
}

/* ------------------------------------------------------------ split size -- */

/* Number of intermediate units in the top segment for split ratio r, rounded
 * to whole chunks of g units: g * floor(r*F/g + 1/2).  The paper defines the
 * split ratio as the top segment's share of the expert (Sec. 2.3); it gives
 * no rounding rule, this is the chosen one. */
int orc_top_units(double r, int F, int g) {
  int u = g * (int)floor(r * (double)F / (double)g + 0.5);
  if (u < 0) u = 0;
  if (u > F) u = F;
  return u;
}
