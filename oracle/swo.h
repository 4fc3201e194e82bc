/*
 * swo.h -- CPU oracle of the SlimWise batched-decode MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, single-threaded
 * definition of what the layer computes, used to check the HIP library.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load it.  It shares no code, header, table or helper with the HIP
 * path, and the HIP path never calls it.
 *
 * Paper: "SlimWise: Decoupling Expert Pruning Across Prefill and Decode for
 * Efficient MoE Serving" (arXiv 2609.34117).
 *
 * Conventions (all host pointers, row-major, no padding):
 *   x        bf16 bits  [T, H]          token activations
 *   wr       fp32       [m, H]          router gate weight, row e = expert e
 *   bias     fp32       [m] or NULL     per-expert router logit bias
 *   w13      bf16 bits  [m, 2I, H]      rows 0..I-1 gate proj, I..2I-1 up proj
 *   w2       bf16 bits  [m, H, I]       down projection, row o = output o
 *   topk_ids int32      [T, k]          pool-space expert ids, (z desc, id asc)
 *   topk_w   fp32       [T, k]          gates, renormalised over the k
 * Every function returns 0 on success and -1 on a bad argument.
 */
#ifndef SWO_H
#define SWO_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Section 3.1: rank experts by importance, keep the top n_keep (k <= n_keep
 * <= m).  Ties in importance go to the smaller expert id.  kept[] lists the
 * kept original ids ascending; remap[e] is the compact index or -1;
 * keep_mask[e] is 1 for kept experts.  The compacted arrays (each may be
 * NULL) are row copies in kept[] order: this is the "separate pruned
 * checkpoint" form of the pruned decoder. */
int swo_prune_compact(int hidden, int inter, int n_experts, int top_k,
                      const float* importance, int n_keep,
                      const uint16_t* w13, const uint16_t* w2,
                      const float* wr, const float* bias,
                      int32_t* kept, int32_t* remap, uint8_t* keep_mask,
                      uint16_t* w13_c, uint16_t* w2_c, float* wr_c,
                      float* bias_c);

/* Section 3.1, Eq. 2 and the renormalisation that follows it.  Router
 * logits z = wr . x (+ bias), masked experts excluded from selection
 * (tau = -inf), top-k by (z desc, id asc), gates = softmax over the k
 * selected logits.  gap[t] (nullable) = z_(k) - z_(k+1) over the eligible
 * experts, +inf when exactly k are eligible.  logits (nullable) receives the
 * unmasked z [T, m]. */
int swo_route(int hidden, int n_experts, int top_k, const uint16_t* x,
              int n_tokens, const float* wr, const float* bias,
              const uint8_t* keep_mask, int32_t* topk_ids, float* topk_w,
              float* gap, float* logits);

/* Section 2.1: the union of experts a decode step touches.  counts[e] =
 * number of (token, slot) pairs routed to e; offsets = exclusive prefix sum
 * (offsets[m] = T*k); perm = flat pair ids p = t*k+j grouped by expert
 * (ascending expert), ascending p inside an expert; active = experts with a
 * nonzero count, ascending; n_active = their number. */
int swo_dispatch(int n_experts, int top_k, const int32_t* topk_ids,
                 int n_tokens, int32_t* counts, int32_t* offsets,
                 int32_t* perm, int32_t* active, int32_t* n_active);

/* The MoE layer output, fp32 accumulation: for every token t and slot j
 * with e = topk_ids[t,j], the SwiGLU expert FFN
 *   g = W13[e,0:I] x_t, u = W13[e,I:2I] x_t, a = silu(g) * u,
 *   y = W2[e] a,
 * and out[t] = sum_j topk_w[t,j] * y, summed in slot order.  Dot products
 * accumulate one term at a time in ascending index order. */
int swo_forward(int hidden, int inter, int n_experts, int top_k,
                const uint16_t* x, int n_tokens, const uint16_t* w13,
                const uint16_t* w2, const int32_t* topk_ids,
                const float* topk_w, float* out);

/* The same computation in fp64 (the shadow that bounds the fp32 oracle's
 * own rounding error). */
int swo_forward_f64(int hidden, int inter, int n_experts, int top_k,
                    const uint16_t* x, int n_tokens, const uint16_t* w13,
                    const uint16_t* w2, const int32_t* topk_ids,
                    const float* topk_w, double* out);

/* Section 3.3: the always-on shared expert behind a sigmoid gate, added to
 * the layer output: for every token,
 *   out[t] += sigmoid(gate_w . x_t) * W2s (silu(W1s x_t) * W3s x_t),
 * W13s = [2I, H] (gate rows first), W2s = [H, I], gate_w fp32 [H]. */
int swo_shared_expert(int hidden, int inter, const uint16_t* x, int n_tokens,
                      const uint16_t* w13, const uint16_t* w2, const float* gate_w,
                      float* out);

/* Section 2.3: the routing-mass statistics of a batch of calibration
 * tokens, accumulated into mass_softmax[m] (softmax over the eligible
 * experts' logits) and mass_topk[m] (renormalised top-k gates); either may
 * be NULL. */
int swo_routing_mass(int hidden, int n_experts, int top_k, const uint16_t* x, int n_tokens,
                     const float* wr, const float* bias, const uint8_t* keep_mask,
                     float* mass_softmax, float* mass_topk);

#ifdef __cplusplus
}
#endif
#endif
