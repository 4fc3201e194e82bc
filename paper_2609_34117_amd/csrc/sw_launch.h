// Host-side launchers of the libslimwise kernels.  Each enqueues on `stream`
// and returns the launch status; arguments are validated by the ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sw {

__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Largest H and I whose 32-token activation tiles fit the wave-streaming
// kernels' LDS staging.
constexpr int kMaxStreamH = 2048;
constexpr int kMaxStreamI = 1024;

size_t route_workspace_bytes(int T, int H, int m, int k);
size_t forward_workspace_bytes(int T, int H, int I, int k);
// y [T*k, H] fp32 inside a forward workspace
const float* forward_y(const void* workspace, int T, int H, int I, int k = 1);
size_t shared_workspace_bytes(int T, int H, int I);
size_t routing_mass_workspace_bytes(int T, int H, int m, int k);
hipError_t launch_routing_mass(const uint16_t* x, int T, const float* wr, const float* bias,
                               const uint8_t* keep_mask, int H, int m, int k, float* mass_softmax,
                               float* mass_topk, void* workspace, hipStream_t stream);
hipError_t launch_shared_expert(const uint16_t* x, int T, const uint16_t* w13, const uint16_t* w2,
                                bool tiled, const float* gate_w, float* out, int H, int I,
                                void* workspace, hipStream_t stream);

hipError_t launch_prune_select(const float* importance, int m, int n_keep, int32_t* kept,
                               int32_t* remap, uint8_t* keep_mask, hipStream_t stream);
hipError_t launch_compact_gather(const int32_t* kept, int n_keep, int H, int I,
                                 const uint16_t* w13, const uint16_t* w2, const float* wr,
                                 const float* bias, uint16_t* w13_c, uint16_t* w2_c, float* wr_c,
                                 float* bias_c, hipStream_t stream);

hipError_t launch_route(const uint16_t* x, int T, const float* wr, const float* bias,
                        const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                        float* topk_w, float* gap, void* workspace, hipStream_t stream);

// Dispatch of n_pairs expert ids; batches above a few thousand pairs run as
// chunked multi-block kernels when `workspace` (dispatch_workspace_bytes)
// is given, else in one block.
size_t dispatch_workspace_bytes(int n_pairs, int m);
hipError_t launch_dispatch(const int* topk_ids, int n_pairs, int m, int* counts, int* offsets,
                           int* perm, int* active, int* n_active, hipStream_t stream,
                           void* workspace = nullptr);

// Route, then dispatch of the selected ids; one select + dispatch block when
// fused_route_dispatch_supported, else the separate kernels.
// With n_shared > 0 the router has a last row, the shared expert's gate,
// and every token gets n_shared more slots after its k routed ones: the
// shared expert's parts with the sigmoid of that gate logit.  The pool
// holds n_groups copies of the parts; token t of T uses copy
// g = t * n_groups / T, pool ids m + g * n_shared .. + n_shared - 1, and the
// plan covers m + n_groups * n_shared experts.
bool fused_route_dispatch_supported(int T, int m, int k, int n_shared = 0, int n_groups = 1);
// The routing half of launch_route_dispatch alone (logits and top-k, same
// outputs), for a caller that builds the plan elsewhere.
hipError_t launch_route_select(const uint16_t* x, int T, const float* wr, const float* bias,
                               const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                               float* topk_w, float* gap, void* workspace, hipStream_t stream,
                               int n_shared = 0, int n_groups = 1);
size_t route_shared_workspace_bytes(int T, int H, int m, int k, int n_shared, int n_groups);
hipError_t launch_route_dispatch(const uint16_t* x, int T, const float* wr, const float* bias,
                                 const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                                 float* topk_w, float* gap, int* counts, int* offsets, int* perm,
                                 int* active, int* n_active, void* workspace, hipStream_t stream,
                                 int n_shared = 0, int n_groups = 1);

// Kernel family serving a gate/up or a down call of a shape; the launchers
// dispatch on it (values as sw_kernel_family in the ABI header).
enum class Kernels : int { kNone = 0, kPrefill = 1, kSplitK = 2, kWave = 3, kGeneric = 4 };
Kernels gate_up_kernels(int T, int H, int I, int m, int k, bool tiled);
Kernels down_kernels(int T, int H, int I, int m, int k, bool tiled);

// `tiled`: weights in the fragment-major layout of sw_moe_pack_experts.
// `identity_plan`: the caller guarantees perm[offsets[e] + s] = offsets[e] + s
// (the shared expert's one-expert plan), so kernels may skip reading perm.
hipError_t launch_gate_up(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                          const int* counts, const int* offsets, const int* perm,
                          const int* active, const int* n_active, int H, int I, int m, int k,
                          void* workspace, hipStream_t stream, bool identity_plan = false);
hipError_t launch_down(int T, const uint16_t* w2, bool tiled, const int* counts,
                       const int* offsets, const int* perm, const int* active,
                       const int* n_active, int H, int I, int m, int k, void* workspace,
                       hipStream_t stream, bool identity_plan = false);
// launch_gate_up for a shape wave_plan_supported takes, building the plan of
// topk_ids on the way (see launch_gate_up_wave_plan).
hipError_t launch_gate_up_building_plan(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                       const int* topk_ids, int* counts, int* offsets, int* perm,
                                       int* active, int* n_active, int H, int I, int m, int k,
                                       void* workspace, hipStream_t stream);
bool wave_stream_supported(int T, int H, int I, int k);
hipError_t launch_gate_up_wave(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                               const int* counts, const int* offsets, const int* perm,
                               const int* active, const int* n_active, int H, int I, int m, int k,
                               uint16_t* h_hi, uint16_t* h_lo, hipStream_t stream);
hipError_t launch_down_wave(int T, const uint16_t* w2, bool tiled, const int* counts,
                            const int* offsets, const int* perm, const int* active,
                            const int* n_active, int H, int I, int m, int k, const uint16_t* h_hi,
                            const uint16_t* h_lo, float* y, hipStream_t stream);
// Decode batches whose gate/up launch can build the dispatch plan itself
// (the 32-token wave kernels, at most 512 experts and 1024 pairs): every
// block builds it in LDS from topk_ids, and block 0 writes counts, offsets,
// perm, active and n_active (the dispatch kernel's outputs, bit for bit)
// for the launches after it.
bool wave_plan_supported(int T, int H, int I, int m, int k, bool tiled);
hipError_t launch_gate_up_wave_plan(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                    const int* topk_ids, int* counts, int* offsets, int* perm,
                                    int* active, int* n_active, int H, int I, int m, int k,
                                    uint16_t* h_hi, uint16_t* h_lo, hipStream_t stream);
// Batches of 16 or more pairs per expert (prefill, large decode): each weight
// tile is streamed once per 160-token pass (expert_prefill.hip).
bool prefill_supported(int T, int H, int I, int m, int k);
hipError_t launch_gate_up_prefill(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                  const int* counts, const int* offsets, const int* perm,
                                  const int* active, const int* n_active, int H, int I, int m,
                                  int k, uint16_t* h_hi, uint16_t* h_lo, hipStream_t stream);
hipError_t launch_down_prefill(int T, const uint16_t* w2, bool tiled, const int* counts,
                               const int* offsets, const int* perm, const int* active,
                               const int* n_active, int H, int I, int m, int k,
                               const uint16_t* h_hi, const uint16_t* h_lo, float* y,
                               hipStream_t stream);
// Few tiles (a decode batch of one or two tokens, the shared expert): each
// tile's K is split over the waves of a block (expert_skinny.hip).
bool skinny_gate_up_supported(int T, int H, int I, int m, int k);
bool skinny_down_supported(int T, int H, int I, int m, int k);
hipError_t launch_gate_up_skinny(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                 const int* counts, const int* offsets, const int* perm,
                                 const int* active, const int* n_active, int H, int I, int m,
                                 int k, uint16_t* h_hi, uint16_t* h_lo, bool identity,
                                 hipStream_t stream);
hipError_t launch_down_skinny(int T, const uint16_t* w2, bool tiled, const int* counts,
                              const int* offsets, const int* perm, const int* active,
                              const int* n_active, int H, int I, int m, int k,
                              const uint16_t* h_hi, const uint16_t* h_lo, float* y,
                              bool identity, hipStream_t stream);
hipError_t launch_pack_experts(const uint16_t* w13, const uint16_t* w2, uint16_t* w13_t,
                               uint16_t* w2_t, int H, int I, int m, hipStream_t stream);
hipError_t launch_combine(int T, const float* topk_w, const int* n_active, float* out, int H,
                          int I, int m, int k, void* workspace, hipStream_t stream);

}  // namespace sw
