// The always-on shared expert (Section 3.3: the distilled pruned decoder
// keeps a shared SwiGLU expert behind a sigmoid gate; the frozen SE1 and the
// added SE2 share that gate and are exported as one expert of twice the
// intermediate width).  For every token t:
//   out[t] += sigmoid(gate_w . x[t]) * W2s (silu(W1s x[t]) * W3s x[t]).
// The expert is run by the routed expert kernels on a plan of one expert
// that every token selects once (k = 1), then added onto the layer output.
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

// One wave per token: the sigmoid gate and the token's plan entry; block 0
// also writes the one-expert histogram, offsets and active list.
__global__ __launch_bounds__(256) void shared_init_kernel(
    const uint16_t* __restrict__ x, const float* __restrict__ gate_w, int T, int H,
    int* __restrict__ counts, int* __restrict__ offsets, int* __restrict__ perm,
    int* __restrict__ active, int* __restrict__ n_active, float* __restrict__ gates) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    counts[0] = T;
    offsets[0] = 0;
    offsets[1] = T;
    active[0] = 0;
    *n_active = 1;
  }
  if (t >= T) return;  // wave-uniform
  const uint16_t* xt = x + (size_t)t * H;
  float z = 0.f;
  for (int h = lane * 8; h < H; h += 64 * 8) {
    const u32x4 v = ld128(xt + h);
    const float4 ga = *reinterpret_cast<const float4*>(gate_w + h);
    const float4 gb = *reinterpret_cast<const float4*>(gate_w + h + 4);
    const float g[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint16_t b = static_cast<uint16_t>((v[i / 2] >> (16 * (i & 1))) & 0xFFFFu);
      z += g[i] * bf16_to_f32(b);
    }
  }
  z = wave_sum_f32(z);
  if (lane == 0) {
    gates[t] = 1.0f / (1.0f + expf(-z));
    perm[t] = t;
  }
}

// out[t, 4c .. 4c+3] += gate[t] * y[t, 4c .. 4c+3]
__global__ __launch_bounds__(256) void shared_add_kernel(const float* __restrict__ y,
                                                        const float* __restrict__ gates,
                                                        float* __restrict__ out, int T, int H) {
  const int hq = H >> 2;
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)T * hq) return;
  const int t = (int)(idx / hq), c = (int)(idx - (size_t)t * hq);
  const float4 v = *reinterpret_cast<const float4*>(y + (size_t)t * H + 4 * c);
  float4* o = reinterpret_cast<float4*>(out + (size_t)t * H + 4 * c);
  const float g = gates[t];
  float4 r = *o;
  r.x += g * v.x;
  r.y += g * v.y;
  r.z += g * v.z;
  r.w += g * v.w;
  *o = r;
}

struct SharedWs {
  int* counts;   // [1]
  int* offsets;  // [2]
  int* active;   // [1]
  int* n_active; // [1]
  int* perm;     // [T]
  float* gates;  // [T]
  void* fwd;     // the expert kernels' workspace for T pairs
};

SharedWs carve_shared(void* ws, int T) {
  char* p = static_cast<char*>(ws);
  SharedWs s;
  s.counts = reinterpret_cast<int*>(p);
  s.offsets = s.counts + 1;
  s.active = s.counts + 3;
  s.n_active = s.counts + 4;
  p += 256;
  s.perm = reinterpret_cast<int*>(p);
  p += align_up((size_t)T * sizeof(int), 256);
  s.gates = reinterpret_cast<float*>(p);
  p += align_up((size_t)T * sizeof(float), 256);
  s.fwd = p;
  return s;
}

}  // namespace

size_t shared_workspace_bytes(int T, int H, int I) {
  if (T <= 0) return 0;
  return 256 + 2 * align_up((size_t)T * 4, 256) + forward_workspace_bytes(T, H, I, 1);
}

hipError_t launch_shared_expert(const uint16_t* x, int T, const uint16_t* w13, const uint16_t* w2,
                                bool tiled, const float* gate_w, float* out, int H, int I,
                                void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const SharedWs s = carve_shared(workspace, T);
  shared_init_kernel<<<(T + 3) / 4, 256, 0, stream>>>(x, gate_w, T, H, s.counts, s.offsets,
                                                      s.perm, s.active, s.n_active, s.gates);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  // the one-expert plan is the identity (perm[t] = t)
  err = launch_gate_up(x, T, w13, tiled, s.counts, s.offsets, s.perm, s.active, s.n_active, H, I,
                       1, 1, s.fwd, stream, true);
  if (err != hipSuccess) return err;
  err = launch_down(T, w2, tiled, s.counts, s.offsets, s.perm, s.active, s.n_active, H, I, 1, 1,
                    s.fwd, stream, true);
  if (err != hipSuccess) return err;
  const float* y = static_cast<const float*>(forward_y(s.fwd, T, H, I));
  const size_t threads = (size_t)T * (H / 4);
  shared_add_kernel<<<(unsigned)((threads + 255) / 256), 256, 0, stream>>>(y, s.gates, out, T, H);
  return hipGetLastError();
}

}  // namespace sw
