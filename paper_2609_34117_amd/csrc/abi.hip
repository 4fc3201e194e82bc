// C ABI of libslimwise: argument validation, then kernel launches on the
// caller's stream.  Nothing is launched unless every check passes.
#include <hip/hip_runtime.h>

#include <atomic>

#include "../../include/slimwise.h"
#include "sw_launch.h"

// Scratch of sw_moe_forward_no_alloc (the per-pair h and y of one call).
// Each device the library runs on holds its own copy until the process
// ends.  In host code `scratch` names a host-side stand-in, never the device
// memory: every use goes through the device address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[SW_NO_ALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxExperts = 1024;
constexpr int kMaxTopK = 32;
constexpr int64_t kMaxBufferBytes = (int64_t)1 << 31;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

sw_status check_dims(const sw_moe_dims* d) {
  if (d == nullptr) return SW_ERR_NULL;
  if (d->hidden <= 0 || d->inter <= 0 || d->n_experts <= 0 || d->top_k <= 0) return SW_ERR_SHAPE;
  if (d->top_k > d->n_experts) return SW_ERR_SHAPE;
  if ((d->hidden & 7) != 0 || (d->inter & 7) != 0) return SW_ERR_ALIGN;
  if (d->n_experts > kMaxExperts || d->top_k > kMaxTopK) return SW_ERR_UNSUPPORTED;
  // each expert's gate/up block is addressed through one 32-bit-ranged buffer
  if (4 * (int64_t)d->inter * d->hidden >= kMaxBufferBytes) return SW_ERR_UNSUPPORTED;
  // ... and so is the router weight
  if (4 * (int64_t)d->n_experts * d->hidden >= kMaxBufferBytes) return SW_ERR_UNSUPPORTED;
  return SW_OK;
}

sw_status check_tokens(const sw_moe_dims* d, int32_t n_tokens) {
  if (n_tokens < 0) return SW_ERR_SHAPE;
  if ((int64_t)n_tokens * d->top_k >= ((int64_t)1 << 31)) return SW_ERR_UNSUPPORTED;
  // token activations and the per-pair intermediate are read through
  // 32-bit-ranged buffers
  if (2 * (int64_t)n_tokens * d->hidden >= kMaxBufferBytes) return SW_ERR_UNSUPPORTED;
  if (2 * (int64_t)n_tokens * d->top_k * d->inter >= kMaxBufferBytes) return SW_ERR_UNSUPPORTED;
  // keeps the per-pair fp32 workspace (T * k * H elements) under 4 TiB
  if ((int64_t)n_tokens * d->top_k * d->hidden >= ((int64_t)1 << 40)) return SW_ERR_UNSUPPORTED;
  return SW_OK;
}

sw_status launched(hipError_t err) { return err == hipSuccess ? SW_OK : SW_ERR_DEVICE; }

bool tiled_shape_ok(const sw_moe_dims* d) {
  return d->hidden % 32 == 0 && d->inter % 32 == 0 && d->hidden <= sw::kMaxStreamH &&
         d->inter <= sw::kMaxStreamI;
}

// Layout argument of the forward calls: known value, and a tiled pool only
// for the shapes (and token counts) the tiled kernels take.
sw_status check_layout(const sw_moe_dims* d, int32_t n_tokens, int32_t layout) {
  if (layout != SW_LAYOUT_ROW_MAJOR && layout != SW_LAYOUT_TILED) return SW_ERR_SHAPE;
  if (layout == SW_LAYOUT_TILED &&
      (!tiled_shape_ok(d) || !sw::wave_stream_supported(n_tokens, d->hidden, d->inter, d->top_k)))
    return SW_ERR_UNSUPPORTED;
  return SW_OK;
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

#define SW_TRY(expr)                 \
  do {                               \
    const sw_status st_ = (expr);    \
    if (st_ != SW_OK) return st_;    \
  } while (0)

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

sw_status scratch_on_current_device(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SW_ERR_DEVICE;
  if (dev < 0 || dev >= kMaxDevices) return SW_ERR_UNSUPPORTED;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    const hipError_t err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return SW_ERR_DEVICE;
    }
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return SW_OK;
}

sw_status check_forward_common(const sw_moe_dims* d, int32_t n_tokens, const int32_t* counts,
                               const int32_t* offsets, const int32_t* perm,
                               const int32_t* active, const int32_t* n_active, void* workspace,
                               size_t workspace_bytes) {
  SW_TRY(check_dims(d));
  SW_TRY(check_tokens(d, n_tokens));
  if (n_tokens == 0) return SW_OK;
  if (!counts || !offsets || !perm || !active || !n_active || !workspace) return SW_ERR_NULL;
  if (!aligned4(counts) || !aligned4(offsets) || !aligned4(perm) || !aligned4(active) ||
      !aligned4(n_active) || !aligned16(workspace))
    return SW_ERR_ALIGN;
  if (workspace_bytes < sw::forward_workspace_bytes(n_tokens, d->hidden, d->inter, d->top_k))
    return SW_ERR_WORKSPACE;
  return SW_OK;
}

// The forward's operands other than the plan and the workspace (T > 0).
sw_status check_forward_operands(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                 const uint16_t* w13, const uint16_t* w2, int32_t layout,
                                 const float* topk_w, const float* out) {
  SW_TRY(check_layout(d, n_tokens, layout));
  if (!x || !w13 || !w2 || !topk_w || !out) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(w13) || !aligned16(w2) || !aligned16(out) || !aligned4(topk_w))
    return SW_ERR_ALIGN;
  return SW_OK;
}

// Routed dims plus n_groups copies of n_shared parts of a shared expert: the
// extended pool and slots must stay within the kernels' limits, and so must
// the router with its gate row.
sw_status check_shared(const sw_moe_dims* d, int32_t n_shared, int32_t n_groups) {
  if (n_shared < 1 || n_groups < 1) return SW_ERR_SHAPE;
  if ((int64_t)d->n_experts + (int64_t)n_groups * n_shared > kMaxExperts ||
      d->top_k + n_shared > kMaxTopK)
    return SW_ERR_UNSUPPORTED;
  if (4 * ((int64_t)d->n_experts + 1) * d->hidden >= kMaxBufferBytes) return SW_ERR_UNSUPPORTED;
  return SW_OK;
}

// gate/up, down and combine on `workspace` (arguments already validated).
sw_status launch_forward(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                         const uint16_t* w13, const uint16_t* w2, int32_t layout,
                         const float* topk_w, const int32_t* counts, const int32_t* offsets,
                         const int32_t* perm, const int32_t* active, const int32_t* n_active,
                         float* out, void* workspace, hipStream_t s) {
  (void)hipGetLastError();
  const int H = d->hidden, I = d->inter, m = d->n_experts, k = d->top_k;
  const bool tiled = layout == SW_LAYOUT_TILED;
  SW_TRY(launched(sw::launch_gate_up(x, n_tokens, w13, tiled, counts, offsets, perm, active,
                                     n_active, H, I, m, k, workspace, s)));
  SW_TRY(launched(sw::launch_down(n_tokens, w2, tiled, counts, offsets, perm, active, n_active, H,
                                  I, m, k, workspace, s)));
  return launched(sw::launch_combine(n_tokens, topk_w, n_active, out, H, I, m, k, workspace, s));
}

// The dims of the pool a layer call's forward runs on: the routed pool, and
// the shared expert's parts after it.
sw_moe_dims layer_pool_dims(const sw_moe_dims* d, int32_t n_shared, int32_t n_groups) {
  if (n_shared == 0) return *d;
  return sw_moe_dims{d->hidden, d->inter, d->n_experts + n_groups * n_shared,
                     d->top_k + n_shared};
}

size_t layer_route_bytes(const sw_moe_dims* d, int32_t T, int32_t n_shared, int32_t n_groups) {
  if (n_shared == 0) return sw::route_workspace_bytes(T, d->hidden, d->n_experts, d->top_k);
  return sw::route_shared_workspace_bytes(T, d->hidden, d->n_experts, d->top_k, n_shared,
                                          n_groups);
}

// Dims, shared-expert and token arguments of a layer call.
sw_status check_layer_dims(const sw_moe_dims* d, int32_t n_tokens, int32_t n_shared,
                           int32_t n_groups) {
  SW_TRY(check_dims(d));
  if (n_shared < 0) return SW_ERR_SHAPE;
  if (n_shared > 0) SW_TRY(check_shared(d, n_shared, n_groups));
  const sw_moe_dims pool = layer_pool_dims(d, n_shared, n_groups);
  SW_TRY(check_dims(&pool));
  return check_tokens(&pool, n_tokens);
}

size_t layer_workspace_bytes(const sw_moe_dims* d, int32_t T, int32_t n_shared,
                             int32_t n_groups) {
  if (T <= 0) return 0;
  const sw_moe_dims pool = layer_pool_dims(d, n_shared, n_groups);
  return sw::align_up(layer_route_bytes(d, T, n_shared, n_groups), 256) +
         sw::forward_workspace_bytes(T, pool.hidden, pool.inter, pool.top_k);
}

}  // namespace

extern "C" {

const char* sw_status_str(int status) {
  switch (status) {
    case SW_OK: return "SW_OK";
    case SW_ERR_NULL: return "SW_ERR_NULL: a required pointer is NULL";
    case SW_ERR_SHAPE: return "SW_ERR_SHAPE: a size is out of range";
    case SW_ERR_ALIGN: return "SW_ERR_ALIGN: pointer not 16-byte aligned or H/I not a multiple of 8";
    case SW_ERR_UNSUPPORTED: return "SW_ERR_UNSUPPORTED: outside the kernels' limits";
    case SW_ERR_WORKSPACE: return "SW_ERR_WORKSPACE: workspace too small";
    case SW_ERR_DEVICE: return "SW_ERR_DEVICE: a HIP launch failed";
    default: return "unknown sw_status";
  }
}

int32_t sw_abi_version(void) { return SW_ABI_VERSION; }

sw_status sw_moe_prune_compact(const sw_moe_dims* full, const float* importance, int32_t n_keep,
                               const uint16_t* w13, const uint16_t* w2, const float* wr,
                               const float* bias, int32_t* kept, int32_t* remap, uint8_t* keep_mask,
                               uint16_t* w13_c, uint16_t* w2_c, float* wr_c, float* bias_c,
                               void* stream) {
  SW_TRY(check_dims(full));
  if (n_keep < full->top_k || n_keep > full->n_experts) return SW_ERR_SHAPE;
  if (!importance || !kept || !remap || !keep_mask) return SW_ERR_NULL;
  if ((w13_c && !w13) || (w2_c && !w2) || (wr_c && !wr) || (bias_c && !bias)) return SW_ERR_NULL;
  if (!aligned4(importance) || !aligned4(kept) || !aligned4(remap)) return SW_ERR_ALIGN;
  if ((w13_c && (!aligned16(w13) || !aligned16(w13_c))) ||
      (w2_c && (!aligned16(w2) || !aligned16(w2_c))) ||
      (wr_c && (!aligned16(wr) || !aligned16(wr_c))) ||
      (bias_c && (!aligned4(bias) || !aligned4(bias_c))))
    return SW_ERR_ALIGN;
  (void)hipGetLastError();
  const hipStream_t s = as_stream(stream);
  SW_TRY(launched(sw::launch_prune_select(importance, full->n_experts, n_keep, kept, remap,
                                          keep_mask, s)));
  return launched(sw::launch_compact_gather(kept, n_keep, full->hidden, full->inter, w13, w2, wr,
                                            bias, w13_c, w2_c, wr_c, bias_c, s));
}

sw_status sw_moe_pack_experts(const sw_moe_dims* d, const uint16_t* w13, const uint16_t* w2,
                              uint16_t* w13_tiled, uint16_t* w2_tiled, void* stream) {
  SW_TRY(check_dims(d));
  if (!tiled_shape_ok(d)) return SW_ERR_UNSUPPORTED;
  if ((w13 && !w13_tiled) || (w2 && !w2_tiled)) return SW_ERR_NULL;
  if ((w13 && (!aligned16(w13) || !aligned16(w13_tiled))) ||
      (w2 && (!aligned16(w2) || !aligned16(w2_tiled))))
    return SW_ERR_ALIGN;
  (void)hipGetLastError();
  return launched(sw::launch_pack_experts(w13, w2, w13_tiled, w2_tiled, d->hidden, d->inter,
                                          d->n_experts, as_stream(stream)));
}

size_t sw_moe_route_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens) {
  if (check_dims(d) != SW_OK || n_tokens <= 0) return 0;
  return sw::route_workspace_bytes(n_tokens, d->hidden, d->n_experts, d->top_k);
}

sw_status sw_moe_route(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens, const float* wr,
                       const float* bias, const uint8_t* keep_mask, int32_t* topk_ids,
                       float* topk_w, float* gap, void* workspace, size_t workspace_bytes,
                       void* stream) {
  SW_TRY(check_dims(d));
  SW_TRY(check_tokens(d, n_tokens));
  if (n_tokens == 0) return SW_OK;
  if (!x || !wr || !topk_ids || !topk_w || !workspace) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(wr) || !aligned16(workspace) || !aligned4(topk_ids) ||
      !aligned4(topk_w) || (gap && !aligned4(gap)) || (bias && !aligned4(bias)))
    return SW_ERR_ALIGN;
  if (workspace_bytes < sw::route_workspace_bytes(n_tokens, d->hidden, d->n_experts, d->top_k))
    return SW_ERR_WORKSPACE;
  (void)hipGetLastError();
  return launched(sw::launch_route(x, n_tokens, wr, bias, keep_mask, d->hidden, d->n_experts,
                                   d->top_k, topk_ids, topk_w, gap, workspace,
                                   as_stream(stream)));
}

sw_status sw_moe_dispatch(const sw_moe_dims* d, const int32_t* topk_ids, int32_t n_tokens,
                          int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* active,
                          int32_t* n_active, void* stream) {
  SW_TRY(check_dims(d));
  SW_TRY(check_tokens(d, n_tokens));
  if (!counts || !offsets || !active || !n_active) return SW_ERR_NULL;
  if (n_tokens > 0 && (!topk_ids || !perm)) return SW_ERR_NULL;
  if (!aligned4(counts) || !aligned4(offsets) || !aligned4(active) || !aligned4(n_active) ||
      (n_tokens > 0 && (!aligned4(topk_ids) || !aligned4(perm))))
    return SW_ERR_ALIGN;
  (void)hipGetLastError();
  return launched(sw::launch_dispatch(topk_ids, n_tokens * d->top_k, d->n_experts, counts,
                                      offsets, perm, active, n_active, as_stream(stream)));
}

sw_status sw_moe_route_dispatch(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                const float* wr, const float* bias, const uint8_t* keep_mask,
                                int32_t* topk_ids, float* topk_w, float* gap, int32_t* counts,
                                int32_t* offsets, int32_t* perm, int32_t* active,
                                int32_t* n_active, void* workspace, size_t workspace_bytes,
                                void* stream) {
  SW_TRY(check_dims(d));
  SW_TRY(check_tokens(d, n_tokens));
  if (!counts || !offsets || !active || !n_active) return SW_ERR_NULL;
  if (!aligned4(counts) || !aligned4(offsets) || !aligned4(active) || !aligned4(n_active))
    return SW_ERR_ALIGN;
  if (n_tokens == 0) {
    (void)hipGetLastError();
    return launched(sw::launch_dispatch(nullptr, 0, d->n_experts, counts, offsets, nullptr,
                                        active, n_active, as_stream(stream)));
  }
  if (!x || !wr || !topk_ids || !topk_w || !perm || !workspace) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(wr) || !aligned16(workspace) || !aligned4(topk_ids) ||
      !aligned4(topk_w) || !aligned4(perm) || (gap && !aligned4(gap)) ||
      (bias && !aligned4(bias)))
    return SW_ERR_ALIGN;
  if (workspace_bytes < sw::route_workspace_bytes(n_tokens, d->hidden, d->n_experts, d->top_k))
    return SW_ERR_WORKSPACE;
  (void)hipGetLastError();
  return launched(sw::launch_route_dispatch(x, n_tokens, wr, bias, keep_mask, d->hidden,
                                            d->n_experts, d->top_k, topk_ids, topk_w, gap, counts,
                                            offsets, perm, active, n_active, workspace,
                                            as_stream(stream)));
}

size_t sw_moe_route_shared_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens,
                                           int32_t n_shared, int32_t n_groups) {
  if (check_dims(d) != SW_OK || check_tokens(d, n_tokens) != SW_OK ||
      check_shared(d, n_shared, n_groups) != SW_OK)
    return 0;
  return sw::route_shared_workspace_bytes(n_tokens, d->hidden, d->n_experts, d->top_k, n_shared,
                                          n_groups);
}

sw_status sw_moe_route_dispatch_shared(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                       const float* wr, const float* bias,
                                       const uint8_t* keep_mask, int32_t n_shared,
                                       int32_t n_groups, int32_t* topk_ids, float* topk_w,
                                       float* gap, int32_t* counts, int32_t* offsets,
                                       int32_t* perm, int32_t* active, int32_t* n_active,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  SW_TRY(check_dims(d));
  SW_TRY(check_shared(d, n_shared, n_groups));
  const sw_moe_dims ext{d->hidden, d->inter, d->n_experts + n_groups * n_shared,
                        d->top_k + n_shared};
  SW_TRY(check_tokens(&ext, n_tokens));
  if (!counts || !offsets || !active || !n_active) return SW_ERR_NULL;
  if (!aligned4(counts) || !aligned4(offsets) || !aligned4(active) || !aligned4(n_active))
    return SW_ERR_ALIGN;
  if (n_tokens == 0) {
    (void)hipGetLastError();
    return launched(sw::launch_dispatch(nullptr, 0, ext.n_experts, counts, offsets, nullptr,
                                        active, n_active, as_stream(stream)));
  }
  if (!x || !wr || !topk_ids || !topk_w || !perm || !workspace) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(wr) || !aligned16(workspace) || !aligned4(topk_ids) ||
      !aligned4(topk_w) || !aligned4(perm) || (gap && !aligned4(gap)) ||
      (bias && !aligned4(bias)))
    return SW_ERR_ALIGN;
  if (workspace_bytes < sw::route_shared_workspace_bytes(n_tokens, d->hidden, d->n_experts,
                                                         d->top_k, n_shared, n_groups))
    return SW_ERR_WORKSPACE;
  (void)hipGetLastError();
  return launched(sw::launch_route_dispatch(x, n_tokens, wr, bias, keep_mask, d->hidden,
                                            d->n_experts, d->top_k, topk_ids, topk_w, gap, counts,
                                            offsets, perm, active, n_active, workspace,
                                            as_stream(stream), n_shared, n_groups));
}

size_t sw_moe_forward_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens) {
  if (check_dims(d) != SW_OK || n_tokens <= 0) return 0;
  return sw::forward_workspace_bytes(n_tokens, d->hidden, d->inter, d->top_k);
}

sw_status sw_moe_forward_kernels(const sw_moe_dims* d, int32_t n_tokens, int32_t layout,
                                 int32_t* gate_up_family, int32_t* down_family) {
  if (!d || !gate_up_family || !down_family) return SW_ERR_NULL;
  SW_TRY(check_dims(d));
  if (n_tokens < 0) return SW_ERR_SHAPE;
  SW_TRY(check_layout(d, n_tokens, layout));
  const bool tiled = layout == SW_LAYOUT_TILED;
  *gate_up_family = (int32_t)sw::gate_up_kernels(n_tokens, d->hidden, d->inter, d->n_experts,
                                                 d->top_k, tiled);
  *down_family = (int32_t)sw::down_kernels(n_tokens, d->hidden, d->inter, d->n_experts,
                                           d->top_k, tiled);
  return SW_OK;
}

sw_status sw_moe_forward_gate_up(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                 const uint16_t* w13, int32_t layout, const int32_t* counts,
                                 const int32_t* offsets, const int32_t* perm,
                                 const int32_t* active, const int32_t* n_active, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  SW_TRY(check_forward_common(d, n_tokens, counts, offsets, perm, active, n_active, workspace,
                              workspace_bytes));
  if (n_tokens == 0) return SW_OK;
  SW_TRY(check_layout(d, n_tokens, layout));
  if (!x || !w13) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(w13)) return SW_ERR_ALIGN;
  (void)hipGetLastError();
  return launched(sw::launch_gate_up(x, n_tokens, w13, layout == SW_LAYOUT_TILED, counts, offsets,
                                     perm, active, n_active,
                                     d->hidden, d->inter, d->n_experts, d->top_k, workspace,
                                     as_stream(stream)));
}

int32_t sw_moe_gate_up_builds_plan(const sw_moe_dims* d, int32_t n_tokens, int32_t layout) {
  if (check_dims(d) != SW_OK || check_tokens(d, n_tokens) != SW_OK || n_tokens == 0 ||
      check_layout(d, n_tokens, layout) != SW_OK)
    return 0;
  return sw::wave_plan_supported(n_tokens, d->hidden, d->inter, d->n_experts, d->top_k,
                                 layout == SW_LAYOUT_TILED)
             ? 1
             : 0;
}

sw_status sw_moe_forward_gate_up_plan(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                      const uint16_t* w13, int32_t layout,
                                      const int32_t* topk_ids, int32_t* counts, int32_t* offsets,
                                      int32_t* perm, int32_t* active, int32_t* n_active,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  SW_TRY(check_forward_common(d, n_tokens, counts, offsets, perm, active, n_active, workspace,
                              workspace_bytes));
  if (n_tokens == 0) return SW_ERR_UNSUPPORTED;
  SW_TRY(check_layout(d, n_tokens, layout));
  if (!x || !w13 || !topk_ids) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(w13) || !aligned4(topk_ids)) return SW_ERR_ALIGN;
  if (!sw_moe_gate_up_builds_plan(d, n_tokens, layout)) return SW_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  return launched(sw::launch_gate_up_building_plan(
      x, n_tokens, w13, layout == SW_LAYOUT_TILED, topk_ids, counts, offsets, perm, active,
      n_active, d->hidden, d->inter, d->n_experts, d->top_k, workspace, as_stream(stream)));
}

sw_status sw_moe_forward_down(const sw_moe_dims* d, int32_t n_tokens, const uint16_t* w2,
                              int32_t layout, const int32_t* counts, const int32_t* offsets,
                              const int32_t* perm, const int32_t* active, const int32_t* n_active,
                              void* workspace, size_t workspace_bytes, void* stream) {
  SW_TRY(check_forward_common(d, n_tokens, counts, offsets, perm, active, n_active, workspace,
                              workspace_bytes));
  if (n_tokens == 0) return SW_OK;
  SW_TRY(check_layout(d, n_tokens, layout));
  if (!w2) return SW_ERR_NULL;
  if (!aligned16(w2)) return SW_ERR_ALIGN;
  (void)hipGetLastError();
  return launched(sw::launch_down(n_tokens, w2, layout == SW_LAYOUT_TILED, counts, offsets, perm,
                                  active, n_active,
                                  d->hidden, d->inter, d->n_experts, d->top_k, workspace,
                                  as_stream(stream)));
}

sw_status sw_moe_forward_combine(const sw_moe_dims* d, int32_t n_tokens, const float* topk_w,
                                 const int32_t* n_active, float* out, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  SW_TRY(check_dims(d));
  SW_TRY(check_tokens(d, n_tokens));
  if (n_tokens == 0) return SW_OK;
  if (!topk_w || !n_active || !out || !workspace) return SW_ERR_NULL;
  if (!aligned4(topk_w) || !aligned4(n_active) || !aligned16(out) || !aligned16(workspace))
    return SW_ERR_ALIGN;
  if (workspace_bytes < sw::forward_workspace_bytes(n_tokens, d->hidden, d->inter, d->top_k))
    return SW_ERR_WORKSPACE;
  (void)hipGetLastError();
  return launched(sw::launch_combine(n_tokens, topk_w, n_active, out, d->hidden, d->inter,
                                     d->n_experts, d->top_k, workspace, as_stream(stream)));
}

size_t sw_moe_layer_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens, int32_t n_shared,
                                    int32_t n_groups) {
  if (check_layer_dims(d, n_tokens, n_shared, n_groups) != SW_OK) return 0;
  return layer_workspace_bytes(d, n_tokens, n_shared, n_groups);
}

sw_status sw_moe_layer_phase(int32_t phase, const sw_moe_dims* d, const uint16_t* x,
                             int32_t n_tokens, const float* wr, const float* bias,
                             const uint8_t* keep_mask, int32_t n_shared, int32_t n_groups,
                             const uint16_t* w13, const uint16_t* w2, int32_t layout,
                             int32_t* topk_ids, float* topk_w, float* gap, int32_t* counts,
                             int32_t* offsets, int32_t* perm, int32_t* active, int32_t* n_active,
                             float* out, void* workspace, size_t workspace_bytes, void* stream) {
  if (phase < 0 || phase > 3) return SW_ERR_SHAPE;
  SW_TRY(check_layer_dims(d, n_tokens, n_shared, n_groups));
  const sw_moe_dims pool = layer_pool_dims(d, n_shared, n_groups);
  if (!counts || !offsets || !active || !n_active) return SW_ERR_NULL;
  if (!aligned4(counts) || !aligned4(offsets) || !aligned4(active) || !aligned4(n_active))
    return SW_ERR_ALIGN;
  const hipStream_t s = as_stream(stream);
  if (n_tokens == 0) {
    if (phase != 0) return SW_OK;
    (void)hipGetLastError();
    return launched(sw::launch_dispatch(nullptr, 0, pool.n_experts, counts, offsets, nullptr,
                                        active, n_active, s));
  }
  if (!x || !wr || !topk_ids || !topk_w || !perm || !workspace) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(wr) || !aligned16(workspace) || !aligned4(topk_ids) ||
      !aligned4(topk_w) || !aligned4(perm) || (gap && !aligned4(gap)) ||
      (bias && !aligned4(bias)))
    return SW_ERR_ALIGN;
  SW_TRY(check_forward_operands(&pool, x, n_tokens, w13, w2, layout, topk_w, out));
  if (workspace_bytes < layer_workspace_bytes(d, n_tokens, n_shared, n_groups))
    return SW_ERR_WORKSPACE;
  (void)hipGetLastError();
  const int H = d->hidden, I = d->inter, m = d->n_experts, k = d->top_k;
  const int mp = pool.n_experts, kp = pool.top_k;
  const bool tiled = layout == SW_LAYOUT_TILED;
  void* fws = static_cast<char*>(workspace) +
              sw::align_up(layer_route_bytes(d, n_tokens, n_shared, n_groups), 256);
  if (phase == 2)
    return launched(sw::launch_down(n_tokens, w2, tiled, counts, offsets, perm, active, n_active,
                                    H, I, mp, kp, fws, s));
  if (phase == 3)
    return launched(sw::launch_combine(n_tokens, topk_w, n_active, out, H, I, mp, kp, fws, s));
  if (sw::wave_plan_supported(n_tokens, H, I, mp, kp, tiled)) {
    // 0: the routing; 1: gate/up, building the plan on the way
    if (phase == 0)
      return launched(sw::launch_route_select(x, n_tokens, wr, bias, keep_mask, H, m, k,
                                              topk_ids, topk_w, gap, workspace, s, n_shared,
                                              n_groups));
    return launched(sw::launch_gate_up_building_plan(x, n_tokens, w13, tiled, topk_ids, counts,
                                                     offsets, perm, active, n_active, H, I, mp,
                                                     kp, fws, s));
  }
  // 0: routing and dispatch; 1: gate/up
  if (phase == 0)
    return launched(sw::launch_route_dispatch(x, n_tokens, wr, bias, keep_mask, H, m, k,
                                              topk_ids, topk_w, gap, counts, offsets, perm,
                                              active, n_active, workspace, s, n_shared,
                                              n_groups));
  return launched(sw::launch_gate_up(x, n_tokens, w13, tiled, counts, offsets, perm, active,
                                     n_active, H, I, mp, kp, fws, s));
}

sw_status sw_moe_layer(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens, const float* wr,
                       const float* bias, const uint8_t* keep_mask, int32_t n_shared,
                       int32_t n_groups, const uint16_t* w13, const uint16_t* w2, int32_t layout,
                       int32_t* topk_ids, float* topk_w, float* gap, int32_t* counts,
                       int32_t* offsets, int32_t* perm, int32_t* active, int32_t* n_active,
                       float* out, void* workspace, size_t workspace_bytes, void* stream) {
  for (int32_t phase = 0; phase < 4; ++phase)
    SW_TRY(sw_moe_layer_phase(phase, d, x, n_tokens, wr, bias, keep_mask, n_shared, n_groups,
                              w13, w2, layout, topk_ids, topk_w, gap, counts, offsets, perm,
                              active, n_active, out, workspace, workspace_bytes, stream));
  return SW_OK;
}

size_t sw_moe_routing_mass_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens) {
  if (check_dims(d) != SW_OK || n_tokens <= 0) return 0;
  return sw::routing_mass_workspace_bytes(n_tokens, d->hidden, d->n_experts, d->top_k);
}

sw_status sw_moe_routing_mass(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                              const float* wr, const float* bias, const uint8_t* keep_mask,
                              float* mass_softmax, float* mass_topk, void* workspace,
                              size_t workspace_bytes, void* stream) {
  SW_TRY(check_dims(d));
  SW_TRY(check_tokens(d, n_tokens));
  if (n_tokens == 0 || (!mass_softmax && !mass_topk)) return SW_OK;
  if (!x || !wr || !workspace) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(wr) || !aligned16(workspace) || (bias && !aligned4(bias)) ||
      (mass_softmax && !aligned4(mass_softmax)) || (mass_topk && !aligned4(mass_topk)))
    return SW_ERR_ALIGN;
  if (workspace_bytes <
      sw::routing_mass_workspace_bytes(n_tokens, d->hidden, d->n_experts, d->top_k))
    return SW_ERR_WORKSPACE;
  (void)hipGetLastError();
  return launched(sw::launch_routing_mass(x, n_tokens, wr, bias, keep_mask, d->hidden,
                                          d->n_experts, d->top_k, mass_softmax, mass_topk,
                                          workspace, as_stream(stream)));
}

size_t sw_moe_shared_workspace_bytes(const sw_moe_dims* d, int32_t n_tokens) {
  if (check_dims(d) != SW_OK || n_tokens <= 0) return 0;
  return sw::shared_workspace_bytes(n_tokens, d->hidden, d->inter);
}

sw_status sw_moe_shared_expert(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                               const uint16_t* w13, const uint16_t* w2, int32_t layout,
                               const float* gate_w, float* out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  SW_TRY(check_dims(d));
  if (d->n_experts != 1 || d->top_k != 1) return SW_ERR_SHAPE;
  SW_TRY(check_tokens(d, n_tokens));
  if (n_tokens == 0) return SW_OK;
  SW_TRY(check_layout(d, n_tokens, layout));
  if (!x || !w13 || !w2 || !gate_w || !out || !workspace) return SW_ERR_NULL;
  if (!aligned16(x) || !aligned16(w13) || !aligned16(w2) || !aligned16(gate_w) ||
      !aligned16(out) || !aligned16(workspace))
    return SW_ERR_ALIGN;
  if (workspace_bytes < sw::shared_workspace_bytes(n_tokens, d->hidden, d->inter))
    return SW_ERR_WORKSPACE;
  (void)hipGetLastError();
  return launched(sw::launch_shared_expert(x, n_tokens, w13, w2, layout == SW_LAYOUT_TILED, gate_w,
                                           out, d->hidden, d->inter, workspace,
                                           as_stream(stream)));
}

sw_status sw_moe_forward(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                         const uint16_t* w13, const uint16_t* w2, int32_t layout,
                         const float* topk_w, const int32_t* counts, const int32_t* offsets,
                         const int32_t* perm, const int32_t* active, const int32_t* n_active,
                         float* out, void* workspace, size_t workspace_bytes, void* stream) {
  SW_TRY(check_forward_common(d, n_tokens, counts, offsets, perm, active, n_active, workspace,
                              workspace_bytes));
  if (n_tokens == 0) return SW_OK;
  SW_TRY(check_forward_operands(d, x, n_tokens, w13, w2, layout, topk_w, out));
  return launch_forward(d, x, n_tokens, w13, w2, layout, topk_w, counts, offsets, perm, active,
                        n_active, out, workspace, as_stream(stream));
}

sw_status sw_moe_forward_no_alloc(const sw_moe_dims* d, const uint16_t* x, int32_t n_tokens,
                                  const uint16_t* w13, const uint16_t* w2, int32_t layout,
                                  const float* topk_w, const int32_t* counts,
                                  const int32_t* offsets, const int32_t* perm,
                                  const int32_t* active, const int32_t* n_active, float* out,
                                  void* stream) {
  SW_TRY(check_dims(d));
  SW_TRY(check_tokens(d, n_tokens));
  if (n_tokens == 0) return SW_OK;
  if (sw::forward_workspace_bytes(n_tokens, d->hidden, d->inter, d->top_k) >
      SW_NO_ALLOC_SCRATCH_BYTES)
    return SW_ERR_WORKSPACE;
  if (!counts || !offsets || !perm || !active || !n_active) return SW_ERR_NULL;
  if (!aligned4(counts) || !aligned4(offsets) || !aligned4(perm) || !aligned4(active) ||
      !aligned4(n_active))
    return SW_ERR_ALIGN;
  SW_TRY(check_forward_operands(d, x, n_tokens, w13, w2, layout, topk_w, out));
  // every argument is valid: only now is the device touched
  void* ws = nullptr;
  SW_TRY(scratch_on_current_device(&ws));
  return launch_forward(d, x, n_tokens, w13, w2, layout, topk_w, counts, offsets, perm, active,
                        n_active, out, ws, as_stream(stream));
}

}  // extern "C"
