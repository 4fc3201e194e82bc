/*
 * slimwise.h -- C ABI of the SlimWise batched-decode MoE layer on MI355X.
 *
 * The layer is the hot path of decode-only expert pruning in "SlimWise:
 * Decoupling Expert Pruning Across Prefill and Decode for Efficient MoE
 * Serving" (arXiv 2609.34117): each decode step reads the weights of every
 * distinct expert chosen across the batch (Section 2.1, Eq. 1), and a pruned
 * decoder -- a compacted checkpoint, or the full pool behind a router mask
 * (Section 3.1, Eq. 2) -- shrinks that set.
 *
 * Conventions shared by every call:
 *   - Every array pointer is a DEVICE pointer on the current HIP device;
 *     the caller allocates and owns all memory.  The library never
 *     allocates, never synchronises and is re-entrant; calls are ordered on
 *     `stream` (a hipStream_t; NULL = the default stream).  It keeps no
 *     mutable global state, except the static per-device scratch of
 *     sw_moe_forward_no_alloc (see there).  Calls on one stream that share output or workspace
 *     buffers must not overlap with calls on other streams.
 *   - bf16 tensors are passed as their raw 16-bit patterns (uint16_t).
 *   - Layouts are dense row-major:
 *       x     bf16 [T, H]         token activations
 *       w13   bf16 [m, 2I, H]     per expert: rows 0..I-1 the gate projection,
 *                                 rows I..2I-1 the up projection
 *       w2    bf16 [m, H, I]      per expert: the down projection
 *       wr    fp32 [m, H]         router gate weight, row e = expert e
 *       bias  fp32 [m]            optional per-expert router logit bias
 *     where m is the number of experts in the pool handed to the call
 *     (`n_experts`): the full pool m, or the compacted pool m' whose ids are
 *     compact indices (map back through `kept`).
 *   - Alignment: x, w13, w2, wr, out and workspace must be 16-byte aligned;
 *     H and I must be multiples of 8.
 *   - Arguments are validated before anything is launched; a non-SW_OK
 *     status means nothing was enqueued (SW_ERR_DEVICE: a launch failed).
 *   - Data-dependent errors that the host cannot see without a sync are
 *     reported in-band on the device, as documented per call.
 *   - Limits: 1 <= top_k <= 32, top_k <= n_experts <= 1024, 0 <= T,
 *     T * top_k < 2^31, and (in bytes) 4*I*H, 4*m*H, 2*T*H and 2*T*k*I below 2^31
 *     (else SW_ERR_UNSUPPORTED).
 */
#ifndef SLIMWISE_H
#define SLIMWISE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SW_OK = 0,
  SW_ERR_NULL = 1,        /* a required pointer is NULL */
  SW_ERR_SHAPE = 2,       /* a size is out of range (dims <= 0, n_keep < k, ...) */
  SW_ERR_ALIGN = 3,       /* pointer not 16-byte aligned, or H / I not multiples of 8 */
  SW_ERR_UNSUPPORTED = 4, /* valid but outside the kernels' limits */
  SW_ERR_WORKSPACE = 5,   /* workspace smaller than the queried size */
  SW_ERR_DEVICE = 6       /* a HIP launch failed */
} sw_status;

/* Layout of the expert weights handed to sw_moe_forward (see
 * sw_moe_pack_experts). */
typedef enum {
  SW_LAYOUT_ROW_MAJOR = 0, /* w13 [m, 2I, H], w2 [m, H, I] as documented above */
  SW_LAYOUT_TILED = 1      /* the fragment-major layout of sw_moe_pack_experts */
} sw_weight_layout;

typedef struct {
  int32_t hidden;    /* H */
  int32_t inter;     /* I, the per-expert intermediate width */
  int32_t n_experts; /* experts in the pool passed to the call */
  int32_t top_k;     /* k, experts per token */
} sw_moe_dims;

/* Human-readable name of a status code (static string, never NULL). */
const char* sw_status_str(int status);

/* Kernel families of the expert FFN calls, as sw_moe_forward_kernels
 * reports them.  Every family computes the same products; the split-K
 * family adds a tile's K slices in a different order than the others, so
 * its results can differ from theirs in the last bits. */
typedef enum {
  SW_KERNELS_NONE = 0,    /* T == 0: nothing is launched */
  SW_KERNELS_PREFILL = 1, /* >= 16 pairs per expert, pool >= 16, H and I multiples of 128 */
  SW_KERNELS_SPLIT_K = 2, /* few tiles with a long K (a token or two, the shared expert) */
  SW_KERNELS_WAVE = 3,    /* the decode streaming kernels (and any tiled pool otherwise) */
  SW_KERNELS_GENERIC = 4  /* row-major shapes outside the others' limits */
} sw_kernel_family;

/* ABI version of this header (bumped on any signature change). */
#define SW_ABI_VERSION 10
int32_t sw_abi_version(void);

/*
 * Prune and compact one layer's pool (Section 3.1: K'_l is the top m' experts
 * of the layer by an importance criterion; the pruned decoder is either a
 * checkpoint with only the retained experts and their router entries, or the
 * full pool with a router mask).  Offline; not on the decode path.
 *
 *   full        dims of the full pool (n_experts = m)
 *   importance  fp32 [m]: higher = more important.  Order is (score desc,
 *               expert id asc); NaN scores give a valid but unspecified set.
 *   n_keep      m', with top_k <= m' <= m (else SW_ERR_SHAPE)
 *   kept        out int32 [m']: retained original ids, ascending
 *   remap       out int32 [m]: compact index of each original id, -1 if pruned
 *   keep_mask   out uint8 [m]: 1 = retained (the router mask of Eq. 2)
 *   w13_c, w2_c, wr_c, bias_c
 *               out, each nullable: the compacted pool [m', ...] in kept
 *               order.  A non-NULL output needs its non-NULL source
 *               (w13, w2, wr, bias); passing all four as NULL gives the
 *               mask-only form for phase-aware masking.
 */
sw_status sw_moe_prune_compact(const sw_moe_dims* full, const float* importance, int32_t n_keep,
                               const uint16_t* w13, const uint16_t* w2, const float* wr,
                               const float* bias, int32_t* kept, int32_t* remap, uint8_t* keep_mask,
                               uint16_t* w13_c, uint16_t* w2_c, float* wr_c, float* bias_c,
                               void* stream);

/* Workspace bytes sw_moe_route and sw_moe_route_dispatch need for T tokens
 * (0 if T == 0): the logit partials, plus, for batches of more than 2048
 * pairs, the scratch of the chunked multi-block dispatch. */
size_t sw_moe_route_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens);

/*
 * Route T tokens (Section 3.1, Eq. 2 and the renormalisation after it):
 * fp32 logits z = wr . x (+ bias); experts with keep_mask[e] == 0 are
 * excluded from selection (tau = -inf); the top-k by (z desc, id asc) are
 * emitted in that order; gates are the softmax of the k selected logits
 * (equal to a softmax over all experts followed by renormalisation over the
 * k), so a gate never depends on the masked experts.
 *
 *   keep_mask  nullable uint8 [m]; NULL = every expert eligible
 *   bias       nullable fp32 [m]
 *   topk_ids   out int32 [T, k], pool ids
 *   topk_w     out fp32  [T, k]
 *   gap        nullable out fp32 [T]: z_(k) - z_(k+1) over the eligible
 *              experts (+inf when exactly k are eligible): tokens with a
 *              tiny gap are near ties whose k-th choice depends on rounding.
 *   workspace  >= sw_moe_route_workspace_bytes(d, T) bytes, 16-byte aligned
 * In-band error: if fewer than k experts are eligible, the missing slots get
 * id -1 and gate 0 and gap is NaN (sw_moe_dispatch then flags the batch).
 */
sw_status sw_moe_route(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens, const float* wr,
                       const float* bias, const uint8_t* keep_mask, int32_t* topk_ids,
                       float* topk_w, float* gap, void* workspace, size_t workspace_bytes,
                       void* stream);

/*
 * Dispatch plan of the step (Section 2.1: the step streams the union of the
 * experts selected across the batch; n_active is the realised E_distinct
 * of Eq. 1).
 *
 *   topk_ids  int32 [T, k]
 *   counts    out int32 [m]: pairs (t, j) routed to each expert
 *   offsets   out int32 [m + 1]: exclusive prefix sum of counts, offsets[m] = T*k
 *   perm      out int32 [T*k]: flat pair ids p = t*k + j grouped by expert
 *             (ascending expert id), ascending p within an expert
 *   active    out int32 [m]: experts with a nonzero count, ascending; the
 *             first *n_active entries are valid
 *   n_active  out int32 [1] (device)
 * In-band error: an id outside [0, m) sets *n_active = -1, counts and
 * offsets to 0 and perm to the identity; sw_moe_forward then writes NaN.
 */
sw_status sw_moe_dispatch(const sw_moe_dims* d, const int32_t* topk_ids, int32_t n_tokens,
                          int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* active,
                          int32_t* n_active, void* stream);

/*
 * Route, then dispatch, in one call (Section 3.1, Eq. 2; Section 2.1, Eq. 1):
 * every output is bit for bit what sw_moe_route followed by sw_moe_dispatch
 * of its topk_ids would write, with the same arguments, workspace
 * (sw_moe_route_workspace_bytes) and in-band errors.  For small decode
 * batches (T <= 32, m <= 256, k <= 16) the selection and the dispatch plan
 * are built by one block (one wave for T <= 4), which saves a kernel launch per step; above 2048
 * pairs the dispatch runs as chunked multi-block kernels whose scratch is in
 * the workspace (sw_moe_dispatch, which has no workspace, keeps one block).
 * T = 0 writes the empty plan (counts and offsets 0, *n_active = 0).
 */
sw_status sw_moe_route_dispatch(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                const float* wr, const float* bias, const uint8_t* keep_mask,
                                int32_t* topk_ids, float* topk_w, float* gap, int32_t* counts,
                                int32_t* offsets, int32_t* perm, int32_t* active,
                                int32_t* n_active, void* workspace, size_t workspace_bytes,
                                void* stream);

/* Workspace bytes sw_moe_route_dispatch_shared needs (0 on invalid
 * arguments). */
size_t sw_moe_route_shared_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens,
                                           int32_t n_shared, int32_t n_groups);

/*
 * Route + dispatch with the always-on shared expert folded into the plan
 * (Section 3.3: the distilled pruned decoder keeps a shared SwiGLU expert,
 * the frozen SE1 plus the added SE2, behind one sigmoid gate).  The shared
 * expert's SwiGLU is separable over its intermediate units, so a shared
 * expert of width n_shared * I is n_shared experts of the routed width I
 * whose down projections add.  The pool holds n_groups copies of those
 * parts after the m routed experts, and token t of the batch uses copy
 * g(t) = t * n_groups / T (contiguous runs of about T / n_groups tokens).
 * This call gives every token, after its k routed slots, n_shared more
 * slots naming its copy's parts, each with the gate sigmoid(wr[m] . x_t):
 *   topk_ids[t, k + s] = m + g(t) * n_shared + s,
 *   topk_w[t, k + s]   = sigmoid(wr[m] . x_t),
 * and builds the plan over the m + n_groups * n_shared experts.
 * sw_moe_forward with dims {H, I, m + n_groups * n_shared, k + n_shared} on
 * that pool (part s of every copy: the gate and up rows of the shared
 * expert's intermediate units s*I .. (s+1)*I - 1, and the matching I
 * columns of its down projection) then adds
 *   sigmoid(wr[m] . x_t) * W2s (silu(W1s x_t) * W3s x_t)
 * to each token's output on the routed experts' launches, bit for bit the
 * same for every n_groups.  n_groups trades weight bytes for pass shape:
 * each copy's parts receive one pair per token of their group, so with
 * groups of at most 32 tokens every part is a one-pass expert, where one
 * copy of a batch of more than 32 tokens gives parts with every token
 * (two passes, or sliced ones); each further copy streams the parts' weights
 * once more.
 *
 *   d          the routed dims: n_experts = m, top_k = k
 *   wr         fp32 [m + 1, H]: the router rows, then the shared gate row
 *   bias, keep_mask  as for sw_moe_route (over the m routed experts)
 *   n_shared   parts of the shared expert, >= 1; k + n_shared <= 32
 *   n_groups   copies of the parts in the pool, >= 1; m + n_groups * n_shared
 *              <= 1024 (else SW_ERR_UNSUPPORTED)
 *   topk_ids, topk_w  out [T, k + n_shared]
 *   gap        nullable out fp32 [T], of the routed selection
 *   counts, active  out int32 [m + n_groups * n_shared]; offsets
 *              [m + n_groups * n_shared + 1]; perm [T (k + n_shared)];
 *              n_active [1]
 *   workspace  >= sw_moe_route_shared_workspace_bytes(d, T, n_shared, n_groups)
 *              bytes
 * In-band errors as sw_moe_route_dispatch.
 */
sw_status sw_moe_route_dispatch_shared(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                       const float* wr, const float* bias,
                                       const uint8_t* keep_mask, int32_t n_shared,
                                       int32_t n_groups, int32_t* topk_ids, float* topk_w,
                                       float* gap, int32_t* counts, int32_t* offsets,
                                       int32_t* perm, int32_t* active, int32_t* n_active,
                                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * Re-lay an expert pool out for streaming (offline, once per pool; a device
 * layout choice, not part of the paper's method).  SW_LAYOUT_TILED stores
 * each expert's weights so that every 16-row MFMA operand fragment a wave
 * loads is one contiguous KiB and every tile of 16 rows is contiguous:
 *   w13_tiled: expert e, tile b (0 <= b < I/8) covers the gate rows 8b..8b+7
 *     and the up rows I+8b..I+8b+7; its H/32 fragments follow each other;
 *     fragment s holds, for lane l = 0..63, the 8 bf16 of tile row (l % 16)
 *     at columns 32s + 8(l / 16) .. +7.  Element offset:
 *     e*2IH + b*16H + s*512 + l*8 + j.
 *   w2_tiled: expert e, tile b (0 <= b < H/16) covers output rows
 *     16b..16b+15 over I the same way: e*HI + b*16I + s*512 + l*8 + j.
 * Both have the size of their row-major sources.  Requires H and I to be
 * multiples of 32, H <= 2048 and I <= 1024 (else SW_ERR_UNSUPPORTED).
 * Either source may be NULL to skip it.  sw_moe_prune_compact copies whole
 * experts, so it compacts tiled pools as well as row-major ones.
 */
sw_status sw_moe_pack_experts(const sw_moe_dims* d, const uint16_t* w13, const uint16_t* w2,
                              uint16_t* w13_tiled, uint16_t* w2_tiled, void* stream);

/* Workspace bytes sw_moe_forward (and its phases) need for T tokens. */
size_t sw_moe_forward_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens);

/*
 * The kernel families (sw_kernel_family) that sw_moe_forward, and
 * sw_moe_forward_gate_up / sw_moe_forward_down, launch for T tokens of this
 * shape and weight layout.  Host-side only: no device work, no stream.
 *   gate_up_family, down_family   out, one int32 each
 * Errors: SW_ERR_NULL (d or an output NULL), SW_ERR_SHAPE (bad dims, T < 0,
 * unknown layout), SW_ERR_UNSUPPORTED (a tiled layout the kernels do not
 * take for this shape), as sw_moe_forward would return them.
 */
sw_status sw_moe_forward_kernels(const sw_moe_dims* d, int32_t n_tokens, int32_t layout,
                                 int32_t* gate_up_family, int32_t* down_family);

/*
 * Expert FFNs and combine (Section 2.1 / 3.1: each token is processed by
 * its k experts, whose outputs are combined with the renormalised gates).
 * For every active expert e and every pair routed to it, the SwiGLU FFN
 *     g = W13[e, 0:I] x_t,  u = W13[e, I:2I] x_t,  a = silu(g) * u,
 *     y = W2[e] a                          (fp32 accumulation)
 * and out[t] = sum_j topk_w[t, j] * y(t, j), summed in slot order.  The
 * same call serves the full pool (prefill shape) and the pruned pool
 * (decode shape).  Weight traffic: each active expert's weights are read
 * from HBM once per pass over its tokens.  One pass holds up to 32 of an
 * expert's pairs in batches of up to 64 tokens; in larger batches up to 128
 * in the gate/up projection and 96 in the down projection (passes whose
 * tokens do not fit in LDS with the whole contraction stage it in slices),
 * and 160 on the prefill-sized kernels.  So every expert of a routed batch
 * of up to 32 tokens, every expert with at most 32 pairs of a batch of up
 * to 64, and every expert with at most 96 pairs of a larger batch is read
 * exactly once (an expert takes at most one pair a token); the split-K
 * kernels of batches of one or two tokens read each expert once.
 *
 *   layout     sw_weight_layout of w13 and w2 (SW_LAYOUT_TILED needs the
 *              shapes sw_moe_pack_experts accepts, and 4*T*k*H < 2^31)
 *   topk_w     fp32 [T, k] gates from sw_moe_route
 *   counts/offsets/perm/active/n_active  the dispatch plan of the same
 *              routing, from sw_moe_dispatch
 *   out        out fp32 [T, H]
 *   workspace  >= sw_moe_forward_workspace_bytes(d, T) bytes, 16-byte aligned
 * In-band error: *n_active < 0 (a flagged dispatch) fills out with NaN.
 * Deterministic: repeated calls on the same inputs give identical bits.
 */
sw_status sw_moe_forward(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                         const uint16_t* w13, const uint16_t* w2, int32_t layout,
                         const float* topk_w, const int32_t* counts, const int32_t* offsets,
                         const int32_t* perm, const int32_t* active, const int32_t* n_active,
                         float* out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * sw_moe_forward without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  It runs the same kernels as
 * sw_moe_forward (bit for bit the same output) with their scratch (the
 * per-pair h and y of the call) in a static device array of
 * SW_NO_ALLOC_SCRATCH_BYTES inside the library, so it allocates nothing:
 * no hipMalloc, no hipFree, no allocating library routine.
 *
 *   arguments   as for sw_moe_forward, minus workspace / workspace_bytes
 * Errors: as sw_moe_forward, and SW_ERR_WORKSPACE when the call needs more
 * scratch than the array holds (sw_moe_forward_workspace_bytes(d, T) >
 * SW_NO_ALLOC_SCRATCH_BYTES: T * k above 2978 routed pairs at H 2048, I 768,
 * i.e. 372 tokens at top-8; the scratch is (4 I + 4 H) bytes a pair), and
 * SW_ERR_DEVICE if the array's device address cannot be found.
 * The array is per device: each GPU the library runs on holds its own copy
 * until the process ends, and the first call on a device looks up its
 * address (kept for later calls).  Every call on one GPU shares that GPU's
 * array and leaves the last call's contents in it (each call writes all the
 * scratch it reads before reading it, so nothing needs clearing): calls
 * that can overlap on one GPU -- on different streams, or from different
 * host threads onto different streams -- race and must be serialised by
 * the caller.
 */
#define SW_NO_ALLOC_SCRATCH_BYTES ((size_t)32 << 20)
sw_status sw_moe_forward_no_alloc(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                  const uint16_t* w13, const uint16_t* w2, int32_t layout,
                                  const float* topk_w, const int32_t* counts,
                                  const int32_t* offsets, const int32_t* perm,
                                  const int32_t* active, const int32_t* n_active, float* out,
                                  void* stream);

/*
 * The three phases of sw_moe_forward, in order, for callers that time them
 * or interleave other work between them.  Arguments have the meaning given
 * for sw_moe_forward, and the phases communicate through `workspace`:
 *   gate_up: h = silu(W13_gate x) * (W13_up x) for every routed pair
 *   down:    y = W2 h for every routed pair
 *   combine: out[t] = sum_j topk_w[t, j] * y(t, j)
 */
sw_status sw_moe_forward_gate_up(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                 const uint16_t* w13, int32_t layout, const int32_t* counts,
                                 const int32_t* offsets, const int32_t* perm,
                                 const int32_t* active, const int32_t* n_active, void* workspace,
                                 size_t workspace_bytes, void* stream);
sw_status sw_moe_forward_down(const sw_moe_dims* d, int32_t n_tokens, const uint16_t* w2,
                              int32_t layout, const int32_t* counts, const int32_t* offsets,
                              const int32_t* perm, const int32_t* active, const int32_t* n_active,
                              void* workspace, size_t workspace_bytes, void* stream);
sw_status sw_moe_forward_combine(const sw_moe_dims* d, int32_t n_tokens, const float* topk_w,
                                 const int32_t* n_active, float* out, void* workspace,
                                 size_t workspace_bytes, void* stream);

/*
 * Whether the gate/up phase builds the dispatch plan itself for T tokens of
 * this shape and layout (the forward's dims: the pool's m and slots per
 * token): 1 for decode batches of 3 to 64 tokens that the 32-token streaming
 * kernels serve, with m <= 512, T*k <= 1024 and 3m + 2 + T*k <= 2464 (the
 * plan's LDS), else 0 (also on invalid arguments).  Host-side only.
 */
int32_t sw_moe_gate_up_builds_plan(const sw_moe_dims* d, int32_t n_tokens, int32_t layout);

/*
 * The gate/up phase (as sw_moe_forward_gate_up) that builds the dispatch
 * plan of topk_ids on the way (Section 2.1): every block of the launch builds
 * the plan in LDS, one of them writes counts, offsets, perm, active and
 * n_active -- what sw_moe_dispatch writes for the same ids, bit for bit,
 * in-band flag included -- and the down and combine phases then read them.
 * sw_moe_layer runs this launch in place of the dispatch kernel.
 *   topk_ids   int32 [T, k] (k = d->top_k, ids into the pool of d->n_experts)
 *   counts, offsets, perm, active, n_active  out, as for sw_moe_dispatch
 * Errors: as sw_moe_forward_gate_up, and SW_ERR_UNSUPPORTED where
 * sw_moe_gate_up_builds_plan is 0 (T = 0 included).
 */
sw_status sw_moe_forward_gate_up_plan(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                      const uint16_t* w13, int32_t layout,
                                      const int32_t* topk_ids, int32_t* counts, int32_t* offsets,
                                      int32_t* perm, int32_t* active, int32_t* n_active,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes sw_moe_layer needs (0 on invalid arguments). */
size_t sw_moe_layer_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens, int32_t n_shared,
                                    int32_t n_groups);

/*
 * One MoE layer in one call: routing (Section 3.1, Eq. 2 and the
 * renormalisation), the dispatch plan (Section 2.1, Eq. 1), the expert FFNs
 * and the weighted combine.  Every output is bit for bit what
 * sw_moe_route_dispatch (n_shared = 0) or sw_moe_route_dispatch_shared
 * (n_shared > 0) followed by sw_moe_forward would write with the same
 * arguments, the forward taking the dims {H, I, m + n_groups * n_shared,
 * k + n_shared}.  On decode batches that the 32-token streaming kernels
 * serve (3 to 64 tokens; at most 512 plan experts and 1024 pairs, within the
 * kernels' LDS), the plan is built inside the gate/up launch: each of its
 * blocks builds it in LDS from the selected ids, and one of them writes it
 * out, which saves the dispatch launch of the step.  Other shapes run the
 * two calls' kernels.
 *
 *   d, x, wr, bias, keep_mask   as for sw_moe_route (n_shared = 0) or
 *              sw_moe_route_dispatch_shared (n_shared > 0: wr has the shared
 *              gate row after the m router rows)
 *   n_shared   parts of a folded shared expert, 0 for none; n_groups their
 *              copies in the pool (ignored when n_shared = 0; as
 *              sw_moe_route_dispatch_shared otherwise)
 *   w13, w2, layout   the pool of m + n_groups * n_shared experts, as for
 *              sw_moe_forward
 *   topk_ids, topk_w  out [T, k + n_shared]; gap nullable out fp32 [T]
 *   counts, offsets, perm, active, n_active  out: the plan, as for
 *              sw_moe_dispatch over the m + n_groups * n_shared experts
 *   out        out fp32 [T, H]
 *   workspace  >= sw_moe_layer_workspace_bytes(d, T, n_shared, n_groups)
 * In-band errors as the two calls (a flagged plan fills out with NaN).
 * T = 0 writes the empty plan and nothing else.
 */
sw_status sw_moe_layer(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens, const float* wr,
                       const float* bias, const uint8_t* keep_mask, int32_t n_shared,
                       int32_t n_groups, const uint16_t* w13, const uint16_t* w2, int32_t layout,
                       int32_t* topk_ids, float* topk_w, float* gap, int32_t* counts,
                       int32_t* offsets, int32_t* perm, int32_t* active, int32_t* n_active,
                       float* out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * One of the four phases of sw_moe_layer, for callers that time them or
 * interleave other work: calling phases 0, 1, 2, 3 in order with the same
 * arguments is sw_moe_layer.  Phase 0 routes (plus the dispatch where the
 * gate/up launch does not build the plan), 1 is the gate/up launch, 2 the
 * down projection, 3 the combine.  The phases communicate through `workspace` and the plan
 * arrays.  Arguments, errors and outputs as sw_moe_layer; a phase outside
 * 0..3 is SW_ERR_SHAPE; with T = 0 phase 0 writes the empty plan and the
 * others do nothing.
 */
sw_status sw_moe_layer_phase(int32_t phase, const sw_moe_dims* d, const uint16_t* x,
                             int32_t n_tokens, const float* wr, const float* bias,
                             const uint8_t* keep_mask, int32_t n_shared, int32_t n_groups,
                             const uint16_t* w13, const uint16_t* w2, int32_t layout,
                             int32_t* topk_ids, float* topk_w, float* gap, int32_t* counts,
                             int32_t* offsets, int32_t* perm, int32_t* active, int32_t* n_active,
                             float* out, void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes sw_moe_routing_mass needs for T tokens (0 if T == 0). */
size_t sw_moe_routing_mass_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens);

/*
 * Routing-mass statistics of a batch of calibration tokens (Section 2.3:
 * the routing-mass importance criterion aggregates the router's gate
 * probabilities), accumulated into the caller's arrays:
 *   mass_softmax[e] += sum_t softmax(z_t)[e], over the eligible experts'
 *                      logits z_t = wr . x_t (+ bias);
 *   mass_topk[e]    += sum of the renormalised gates e receives as one of a
 *                      token's top-k (sw_moe_route's selection).
 * Pruning then keeps the experts with the largest mass (pass it as the
 * importance of sw_moe_prune_compact).  Masked experts receive nothing.
 *
 *   d                hidden, n_experts = m, top_k (inter is not used)
 *   x, wr, bias,     as for sw_moe_route
 *   keep_mask
 *   mass_softmax,    nullable fp32 [m] each, read and written
 *   mass_topk
 *   workspace        >= sw_moe_routing_mass_workspace_bytes(d, T) bytes,
 *                    16-byte aligned
 * In-band error: if fewer than k experts are eligible, mass_topk is left
 * unchanged (mass_softmax is still accumulated).
 */
sw_status sw_moe_routing_mass(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                              const float* wr, const float* bias, const uint8_t* keep_mask,
                              float* mass_softmax, float* mass_topk, void* workspace,
                              size_t workspace_bytes, void* stream);

/* Workspace bytes sw_moe_shared_expert needs for T tokens (0 if T == 0). */
size_t sw_moe_shared_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens);

/*
 * The always-on shared expert of the distilled pruned decoder (Section 3.3:
 * the frozen shared expert SE1 and the added SE2, whose down projection
 * starts at zero, share one sigmoid gate and are exported as one expert of
 * twice the intermediate width), added onto the layer output:
 *   out[t] += sigmoid(gate_w . x[t]) * W2s (silu(W1s x[t]) * W3s x[t]).
 *
 *   d          hidden = H, inter = the shared expert's width I_s,
 *              n_experts = 1, top_k = 1
 *   x          bf16 [T, H]
 *   w13, w2    bf16 [2 I_s, H] (gate rows, then up rows) and [H, I_s], in
 *              `layout` (SW_LAYOUT_TILED: packed by sw_moe_pack_experts with
 *              n_experts = 1)
 *   gate_w     fp32 [H], 16-byte aligned
 *   out        fp32 [T, H], read and written (the routed layer output)
 *   workspace  >= sw_moe_shared_workspace_bytes(d, T) bytes, 16-byte aligned
 * Calls that share `out` or `workspace` must be ordered on one stream.
 */
sw_status sw_moe_shared_expert(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                               const uint16_t* w13, const uint16_t* w2, int32_t layout,
                               const float* gate_w, float* out, void* workspace,
                               size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif
