/*
 * slimwise_oracle.c -- CPU oracle of the SlimWise batched-decode MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY: a plain, slow, single-threaded definition of
 * the layer, used by the tests, the smoke check and the benchmark's CPU
 * baseline to check the HIP library.  It shares no code with that library.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -shared -fPIC
 * (no FMA contraction: every product and every sum rounds to fp32 on its
 * own, in the order written here).
 *
 * Readings where the paper leaves a detail open (each is restated where it
 * is used):
 *   - tau in Eq. 2 is taken as -inf: a masked expert is never selected and
 *     adds nothing to the renormalised gates.  This equals any finite tau
 *     whenever at least k experts are kept.
 *   - the gate of a selected expert is the softmax of its logit over the k
 *     selected logits (identical to softmax over all m, then top-k, then
 *     renormalising over the k).
 *   - top-k and importance ties go to the smaller expert id.
 *   - the expert FFN is SwiGLU, gate rows first in W13.
 */
#include "swo.h"

#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

/* A bf16 value is the top 16 bits of an IEEE fp32 value: widening is exact. */
static float widen_bf16(uint16_t bits) {
  uint32_t u = ((uint32_t)bits) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* Section 3.1 (SlimWise Serving Framework): K'_l is built by ranking the
 * layer's experts by an importance criterion and retaining the top m'.  The
 * importance scores themselves come from calibration statistics (Appendix,
 * "Pruning"); here they are an input.  The compacted arrays are the pruned
 * checkpoint that holds only the retained experts and their router entries. */
int swo_prune_compact(int hidden, int inter, int n_experts, int top_k,
                      const float* importance, int n_keep,
                      const uint16_t* w13, const uint16_t* w2,
                      const float* wr, const float* bias,
                      int32_t* kept, int32_t* remap, uint8_t* keep_mask,
                      uint16_t* w13_c, uint16_t* w2_c, float* wr_c,
                      float* bias_c) {
  if (hidden <= 0 || inter <= 0 || n_experts <= 0 || top_k <= 0) return -1;
  if (n_keep < top_k || n_keep > n_experts) return -1;
  if (!importance || !kept || !remap || !keep_mask) return -1;
  if (w13_c && !w13) return -1;
  if (w2_c && !w2) return -1;
  if (wr_c && !wr) return -1;
  if (bias_c && !bias) return -1;

  /* order[] = expert ids sorted by (importance desc, id asc): insertion
   * sort, where an element moves left only past strictly lower-ranked ones,
   * so equal scores keep ascending id order. */
  int32_t order[n_experts];
  for (int e = 0; e < n_experts; ++e) order[e] = e;
  for (int i = 1; i < n_experts; ++i) {
    int32_t cur = order[i];
    int j = i - 1;
    while (j >= 0 && importance[order[j]] < importance[cur]) {
      order[j + 1] = order[j];
      --j;
    }
    order[j + 1] = cur;
  }

  for (int e = 0; e < n_experts; ++e) keep_mask[e] = 0;
  for (int r = 0; r < n_keep; ++r) keep_mask[order[r]] = 1;

  /* kept ids ascending, and the original -> compact index map */
  int c = 0;
  for (int e = 0; e < n_experts; ++e) {
    if (keep_mask[e]) {
      kept[c] = e;
      remap[e] = c;
      ++c;
    } else {
      remap[e] = -1;
    }
  }

  const size_t h = (size_t)hidden, in = (size_t)inter;
  for (int ci = 0; ci < n_keep; ++ci) {
    const size_t e = (size_t)kept[ci];
    if (w13_c) memcpy(w13_c + ci * 2 * in * h, w13 + e * 2 * in * h, 2 * in * h * sizeof(uint16_t));
    if (w2_c) memcpy(w2_c + ci * h * in, w2 + e * h * in, h * in * sizeof(uint16_t));
    if (wr_c) memcpy(wr_c + ci * h, wr + e * h, h * sizeof(float));
    if (bias_c) bias_c[ci] = bias[e];
  }
  return 0;
}

/* Section 3.1, Eq. 2: masked logits z~_i = z_i for kept experts and tau
 * otherwise; the masked router picks the top k inside K'_l, and the gates
 * are renormalised over the k selected experts only, so a surviving
 * expert's gate does not depend on the removed experts. */
int swo_route(int hidden, int n_experts, int top_k, const uint16_t* x,
              int n_tokens, const float* wr, const float* bias,
              const uint8_t* keep_mask, int32_t* topk_ids, float* topk_w,
              float* gap, float* logits) {
  if (hidden <= 0 || n_experts <= 0 || top_k <= 0 || n_tokens < 0) return -1;
  if (n_tokens > 0 && (!x || !wr || !topk_ids || !topk_w)) return -1;
  int n_eligible = 0;
  for (int e = 0; e < n_experts; ++e)
    if (!keep_mask || keep_mask[e]) ++n_eligible;
  if (top_k > n_eligible) return -1;

  float z[n_experts];
  unsigned char taken[n_experts];
  for (int t = 0; t < n_tokens; ++t) {
    const uint16_t* xt = x + (size_t)t * hidden;
    /* router logits, one fp32 term at a time in ascending h */
    for (int e = 0; e < n_experts; ++e) {
      const float* we = wr + (size_t)e * hidden;
      float acc = 0.0f;
      for (int hh = 0; hh < hidden; ++hh) acc += widen_bf16(xt[hh]) * we[hh];
      if (bias) acc += bias[e];
      z[e] = acc;
      if (logits) logits[(size_t)t * n_experts + e] = acc;
    }
    /* top-k over the eligible experts: k passes, each taking the largest
     * remaining logit; scanning ids upward with a strict '>' keeps the
     * smaller id on equal logits. */
    for (int e = 0; e < n_experts; ++e) taken[e] = (keep_mask && !keep_mask[e]) ? 1 : 0;
    int32_t* ids = topk_ids + (size_t)t * top_k;
    for (int j = 0; j < top_k; ++j) {
      int best = -1;
      for (int e = 0; e < n_experts; ++e) {
        if (taken[e]) continue;
        if (best < 0 || z[e] > z[best]) best = e;
      }
      ids[j] = best;
      taken[best] = 1;
    }
    if (gap) {
      int next = -1;
      for (int e = 0; e < n_experts; ++e) {
        if (taken[e]) continue;
        if (next < 0 || z[e] > z[next]) next = e;
      }
      gap[t] = next < 0 ? INFINITY : z[ids[top_k - 1]] - z[next];
    }
    /* gates: softmax over the k selected logits, shifted by the largest */
    float* w = topk_w + (size_t)t * top_k;
    const float zmax = z[ids[0]];
    float denom = 0.0f;
    for (int j = 0; j < top_k; ++j) {
      w[j] = expf(z[ids[j]] - zmax);
      denom += w[j];
    }
    for (int j = 0; j < top_k; ++j) w[j] = w[j] / denom;
  }
  return 0;
}

/* Section 2.1: a decode step reads every distinct expert selected across the
 * batch; active[] is that set and n_active its size (Eq. 1 gives its
 * expectation under uniform routing).  The grouping is written as the
 * direct double loop: for each expert in turn, every pair routed to it in
 * ascending pair order. */
int swo_dispatch(int n_experts, int top_k, const int32_t* topk_ids,
                 int n_tokens, int32_t* counts, int32_t* offsets,
                 int32_t* perm, int32_t* active, int32_t* n_active) {
  if (n_experts <= 0 || top_k <= 0 || n_tokens < 0) return -1;
  if (!counts || !offsets || !active || !n_active) return -1;
  if (n_tokens > 0 && (!topk_ids || !perm)) return -1;
  const int n_pairs = n_tokens * top_k;
  for (int p = 0; p < n_pairs; ++p)
    if (topk_ids[p] < 0 || topk_ids[p] >= n_experts) return -1;

  int pos = 0, na = 0;
  for (int e = 0; e < n_experts; ++e) {
    offsets[e] = pos;
    int c = 0;
    for (int p = 0; p < n_pairs; ++p) {
      if (topk_ids[p] == e) {
        perm[pos++] = p;
        ++c;
      }
    }
    counts[e] = c;
    if (c > 0) active[na++] = e;
  }
  offsets[n_experts] = pos;
  *n_active = na;
  return 0;
}

/* SwiGLU activation of the gate, times the up projection. */
static float swiglu_f32(float g, float u) { return (g / (1.0f + expf(-g))) * u; }
static double swiglu_f64(double g, double u) { return (g / (1.0 + exp(-g))) * u; }

/* Section 2.1 / Section 3.1: each token is processed by its k selected
 * experts and their outputs are combined with the renormalised gates.  The
 * expert is a gated FFN whose last matrix is the down projection (Section
 * 3.3 names it); the gate/up pair with SiLU is the SwiGLU form. */
int swo_forward(int hidden, int inter, int n_experts, int top_k,
                const uint16_t* x, int n_tokens, const uint16_t* w13,
                const uint16_t* w2, const int32_t* topk_ids,
                const float* topk_w, float* out) {
  if (hidden <= 0 || inter <= 0 || n_experts <= 0 || top_k <= 0 || n_tokens < 0) return -1;
  if (n_tokens > 0 && (!x || !w13 || !w2 || !topk_ids || !topk_w || !out)) return -1;
  for (int p = 0; p < n_tokens * top_k; ++p)
    if (topk_ids[p] < 0 || topk_ids[p] >= n_experts) return -1;

  const size_t H = (size_t)hidden, I = (size_t)inter;
  float a[inter];
  for (int t = 0; t < n_tokens; ++t) {
    const uint16_t* xt = x + (size_t)t * H;
    float* ot = out + (size_t)t * H;
    for (size_t o = 0; o < H; ++o) ot[o] = 0.0f;
    for (int j = 0; j < top_k; ++j) {
      const size_t e = (size_t)topk_ids[(size_t)t * top_k + j];
      const float wj = topk_w[(size_t)t * top_k + j];
      const uint16_t* gate = w13 + e * 2 * I * H;
      const uint16_t* up = gate + I * H;
      const uint16_t* down = w2 + e * H * I;
      for (size_t i = 0; i < I; ++i) {
        float g = 0.0f, u = 0.0f;
        for (size_t h = 0; h < H; ++h) {
          const float xv = widen_bf16(xt[h]);
          g += widen_bf16(gate[i * H + h]) * xv;
          u += widen_bf16(up[i * H + h]) * xv;
        }
        a[i] = swiglu_f32(g, u);
      }
      for (size_t o = 0; o < H; ++o) {
        float y = 0.0f;
        for (size_t i = 0; i < I; ++i) y += widen_bf16(down[o * I + i]) * a[i];
        ot[o] += wj * y;
      }
    }
  }
  return 0;
}

int swo_forward_f64(int hidden, int inter, int n_experts, int top_k,
                    const uint16_t* x, int n_tokens, const uint16_t* w13,
                    const uint16_t* w2, const int32_t* topk_ids,
                    const float* topk_w, double* out) {
  if (hidden <= 0 || inter <= 0 || n_experts <= 0 || top_k <= 0 || n_tokens < 0) return -1;
  if (n_tokens > 0 && (!x || !w13 || !w2 || !topk_ids || !topk_w || !out)) return -1;
  for (int p = 0; p < n_tokens * top_k; ++p)
    if (topk_ids[p] < 0 || topk_ids[p] >= n_experts) return -1;

  const size_t H = (size_t)hidden, I = (size_t)inter;
  double a[inter];
  for (int t = 0; t < n_tokens; ++t) {
    const uint16_t* xt = x + (size_t)t * H;
    double* ot = out + (size_t)t * H;
    for (size_t o = 0; o < H; ++o) ot[o] = 0.0;
    for (int j = 0; j < top_k; ++j) {
      const size_t e = (size_t)topk_ids[(size_t)t * top_k + j];
      const double wj = (double)topk_w[(size_t)t * top_k + j];
      const uint16_t* gate = w13 + e * 2 * I * H;
      const uint16_t* up = gate + I * H;
      const uint16_t* down = w2 + e * H * I;
      for (size_t i = 0; i < I; ++i) {
        double g = 0.0, u = 0.0;
        for (size_t h = 0; h < H; ++h) {
          const double xv = (double)widen_bf16(xt[h]);
          g += (double)widen_bf16(gate[i * H + h]) * xv;
          u += (double)widen_bf16(up[i * H + h]) * xv;
        }
        a[i] = swiglu_f64(g, u);
      }
      for (size_t o = 0; o < H; ++o) {
        double y = 0.0;
        for (size_t i = 0; i < I; ++i) y += (double)widen_bf16(down[o * I + i]) * a[i];
        ot[o] += wj * y;
      }
    }
  }
  return 0;
}

/* Section 3.3 (the distilled pruned decoder keeps an always-on shared expert
 * behind a sigmoid gate; the frozen expert SE1 and the added SE2, whose down
 * projection starts at zero, share that gate, so their concatenation is one
 * expert of twice the intermediate width).  For every token,
 *   out[t] += sigmoid(gate_w . x[t]) * W2s (silu(W1s x[t]) * W3s x[t]),
 * with W13s = [W1s; W3s] ([2I, H], gate rows first) and W2s = [H, I].  The
 * gate's dot product and every contraction accumulate in ascending index
 * order in fp32; the shared term is added to out after the routed sum. */
int swo_shared_expert(int hidden, int inter, const uint16_t* x, int n_tokens,
                      const uint16_t* w13, const uint16_t* w2, const float* gate_w,
                      float* out) {
  if (hidden <= 0 || inter <= 0 || n_tokens < 0) return -1;
  if (n_tokens > 0 && (!x || !w13 || !w2 || !gate_w || !out)) return -1;
  const size_t H = (size_t)hidden, I = (size_t)inter;
  const uint16_t* gate = w13;
  const uint16_t* up = w13 + I * H;
  float a[inter];
  for (int t = 0; t < n_tokens; ++t) {
    const uint16_t* xt = x + (size_t)t * H;
    float* ot = out + (size_t)t * H;
    float z = 0.0f;
    for (size_t h = 0; h < H; ++h) z += gate_w[h] * widen_bf16(xt[h]);
    const float s = 1.0f / (1.0f + expf(-z));
    for (size_t i = 0; i < I; ++i) {
      float g = 0.0f, u = 0.0f;
      for (size_t h = 0; h < H; ++h) {
        const float xv = widen_bf16(xt[h]);
        g += widen_bf16(gate[i * H + h]) * xv;
        u += widen_bf16(up[i * H + h]) * xv;
      }
      a[i] = swiglu_f32(g, u);
    }
    for (size_t o = 0; o < H; ++o) {
      float y = 0.0f;
      for (size_t i = 0; i < I; ++i) y += widen_bf16(w2[o * I + i]) * a[i];
      ot[o] += s * y;
    }
  }
  return 0;
}

/* Section 2.3 (importance criteria computed from calibration tokens; the
 * routing-mass criterion aggregates the router's gate probabilities).  Two
 * aggregates are accumulated into the caller's arrays, token by token in
 * ascending order:
 *   mass_softmax[e] += softmax(z_t)[e], the softmax over the eligible
 *                      experts' logits (masked experts receive nothing);
 *   mass_topk[e]    += the renormalised gate expert e receives among the
 *                      token's top-k (slot order), as routed by swo_route.
 * Either may be NULL. */
int swo_routing_mass(int hidden, int n_experts, int top_k, const uint16_t* x, int n_tokens,
                     const float* wr, const float* bias, const uint8_t* keep_mask,
                     float* mass_softmax, float* mass_topk) {
  if (hidden <= 0 || n_experts <= 0 || top_k <= 0 || n_tokens < 0) return -1;
  if (n_tokens == 0) return 0;
  const size_t T = (size_t)n_tokens, m = (size_t)n_experts, k = (size_t)top_k;
  float* z = (float*)malloc(T * m * sizeof(float));
  int32_t* ids = (int32_t*)malloc(T * k * sizeof(int32_t));
  float* w = (float*)malloc(T * k * sizeof(float));
  int rc = (z && ids && w) ? 0 : -1;
  if (rc == 0)
    rc = swo_route(hidden, n_experts, top_k, x, n_tokens, wr, bias, keep_mask, ids, w, NULL, z);
  if (rc == 0) {
    for (size_t t = 0; t < T; ++t) {
      const float* zt = z + t * m;
      if (mass_softmax) {
        float zmax = -INFINITY;
        for (size_t e = 0; e < m; ++e)
          if ((!keep_mask || keep_mask[e]) && zt[e] > zmax) zmax = zt[e];
        float denom = 0.0f;
        for (size_t e = 0; e < m; ++e)
          if (!keep_mask || keep_mask[e]) denom += expf(zt[e] - zmax);
        for (size_t e = 0; e < m; ++e)
          if (!keep_mask || keep_mask[e]) mass_softmax[e] += expf(zt[e] - zmax) / denom;
      }
      if (mass_topk)
        for (size_t j = 0; j < k; ++j) mass_topk[ids[t * k + j]] += w[t * k + j];
    }
  }
  free(z);
  free(ids);
  free(w);
  return rc;
}

