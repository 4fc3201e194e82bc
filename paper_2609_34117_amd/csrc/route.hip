// Router of the MoE layer on gfx950: fp32 logits, masked top-k selection and
// renormalised gates (Section 3.1, Eq. 2 and the renormalisation after it).
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kRouteTokens = 16;                  // tokens per block
constexpr int kRouteExpertsPerWave = 2;
constexpr int kRouteExperts = 4 * kRouteExpertsPerWave;  // experts per block
constexpr int kRouteChunk = 512;                  // hidden columns staged per step
constexpr int kMaxPool = 1024;
constexpr int kKeysPerLane = kMaxPool / kWave;

// In-register transposing butterfly: each lane starts with N partial sums
// (N a power of two <= 64); after the steps, lane l holds the wave-wide total
// of value index (l >> (6 - log2 N)) in v[0].  Every exchange halves the
// number of live values, so the cost is ~N shuffles instead of 6N.
template <int N, int S>
struct TransposeReduce {
  static __device__ __forceinline__ void run(float* v, int lane) {
    if constexpr (S == 0) {
      return;
    } else if constexpr (N > 1) {
      constexpr int half = N / 2;
      const bool upper = (lane & S) != 0;
#pragma unroll
      for (int i = 0; i < half; ++i) {
        const float send = upper ? v[i] : v[i + half];
        const float keep = upper ? v[i + half] : v[i];
        v[i] = keep + __shfl_xor(send, S);
      }
      TransposeReduce<half, S / 2>::run(v, lane);
    } else {
      v[0] += __shfl_xor(v[0], S);
      TransposeReduce<1, S / 2>::run(v, lane);
    }
  }
};

// z[t, e] = sum_h x[t, h] * wr[e, h]  (+ bias[e]), fp32.
// Block = 4 waves; tile = 8 experts x 16 tokens.  x is staged through LDS in
// 512-column chunks; each lane owns 8 columns of a chunk, so router rows and
// staged x are read with 128-bit accesses.
__global__ __launch_bounds__(256) void route_logits_kernel(const uint16_t* __restrict__ x,
                                                          const float* __restrict__ wr,
                                                          const float* __restrict__ bias,
                                                          float* __restrict__ z, int T, int H,
                                                          int m) {
  __shared__ u32x4 xs[kRouteTokens][kRouteChunk / 8];
  const int t0 = blockIdx.x * kRouteTokens;
  const int e0 = blockIdx.y * kRouteExperts;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int NV = kRouteExpertsPerWave * kRouteTokens;
  float acc[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) acc[i] = 0.f;

  for (int k0 = 0; k0 < H; k0 += kRouteChunk) {
    for (int c = threadIdx.x; c < kRouteTokens * (kRouteChunk / 8); c += 256) {
      const int tt = c / (kRouteChunk / 8), cc = c % (kRouteChunk / 8);
      const int col = k0 + cc * 8;
      xs[tt][cc] = (t0 + tt < T && col < H) ? ld128(x + (size_t)(t0 + tt) * H + col) : zero4();
    }
    __syncthreads();
    const int col = k0 + lane * 8;
    if (col < H) {
      float wv[kRouteExpertsPerWave][8];
#pragma unroll
      for (int ex = 0; ex < kRouteExpertsPerWave; ++ex) {
        const int e = e0 + wave * kRouteExpertsPerWave + ex;
        if (e < m) {
          const float4* p = reinterpret_cast<const float4*>(wr + (size_t)e * H + col);
          const float4 a = p[0], b = p[1];
          wv[ex][0] = a.x; wv[ex][1] = a.y; wv[ex][2] = a.z; wv[ex][3] = a.w;
          wv[ex][4] = b.x; wv[ex][5] = b.y; wv[ex][6] = b.z; wv[ex][7] = b.w;
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) wv[ex][i] = 0.f;
        }
      }
#pragma unroll
      for (int tt = 0; tt < kRouteTokens; ++tt) {
        const u32x4 xv = xs[tt][lane];
        float xf[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          xf[2 * q] = __uint_as_float(xv[q] << 16);
          xf[2 * q + 1] = __uint_as_float(xv[q] & 0xffff0000u);
        }
#pragma unroll
        for (int ex = 0; ex < kRouteExpertsPerWave; ++ex) {
          float s = acc[ex * kRouteTokens + tt];
#pragma unroll
          for (int i = 0; i < 8; ++i) s = fmaf(wv[ex][i], xf[i], s);
          acc[ex * kRouteTokens + tt] = s;
        }
      }
    }
    __syncthreads();
  }

  TransposeReduce<NV, 32>::run(acc, lane);
  // NV = 32: lanes 2v and 2v+1 both hold value v.
  if ((lane & 1) == 0) {
    const int v = lane >> 1;
    const int ex = v / kRouteTokens, tt = v % kRouteTokens;
    const int e = e0 + wave * kRouteExpertsPerWave + ex;
    const int t = t0 + tt;
    if (e < m && t < T) z[(size_t)t * m + e] = bias ? acc[0] + bias[e] : acc[0];
  }
}

// One wave per token: top-k over the eligible experts by (z desc, id asc),
// then softmax over the k selected logits.  Keys pack the order-preserving
// image of z with the complemented expert id, so one 64-bit max picks the
// largest logit and, among equal logits, the smallest id.
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ z,
                                                        const uint8_t* __restrict__ keep_mask,
                                                        int T, int m, int k,
                                                        int* __restrict__ topk_ids,
                                                        float* __restrict__ topk_w,
                                                        float* __restrict__ gap) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float* zt = z + (size_t)t * m;
  const int nq = (m + 63) >> 6;
  uint64_t key[kKeysPerLane];
#pragma unroll
  for (int q = 0; q < kKeysPerLane; ++q) {
    key[q] = 0;
    const int e = q * 64 + lane;
    if (q < nq && e < m && (keep_mask == nullptr || keep_mask[e] != 0))
      key[q] = (static_cast<uint64_t>(f32_order_key(zt[e])) << 32) | (0xffffffffu - (uint32_t)e);
  }

  int my_id = -1;
  float my_z = 0.f, zk = 0.f, zk1 = 0.f;
  bool complete = true, have_next = false;
  for (int j = 0; j <= k; ++j) {
    uint64_t best = 0;
#pragma unroll
    for (int q = 0; q < kKeysPerLane; ++q)
      if (q < nq) best = key[q] > best ? key[q] : best;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) {
      const uint64_t o = shfl_xor_u64(best, s);
      best = o > best ? o : best;
    }
    if (best == 0) {  // wave-uniform: no eligible expert left
      if (j < k) complete = false;
      break;
    }
    const int e = static_cast<int>(0xffffffffu - static_cast<uint32_t>(best));
    const float ze = f32_from_order_key(static_cast<uint32_t>(best >> 32));
    if (j == k) {
      zk1 = ze;
      have_next = true;
      break;
    }
    if (lane == j) {
      my_id = e;
      my_z = ze;
    }
    if (j == k - 1) zk = ze;
    if ((e & 63) == lane) {
#pragma unroll
      for (int q = 0; q < kKeysPerLane; ++q)
        if (q == (e >> 6)) key[q] = 0;
    }
  }

  const float z0 = __shfl(my_z, 0);
  const float ex = (lane < k && my_id >= 0) ? expf(my_z - z0) : 0.f;
  float s = ex;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  if (lane < k) {
    topk_ids[(size_t)t * k + lane] = my_id;
    topk_w[(size_t)t * k + lane] = my_id >= 0 ? ex / s : 0.f;
  }
  if (gap != nullptr && lane == 0)
    gap[t] = !complete ? __builtin_nanf("") : (have_next ? zk - zk1 : __builtin_inff());
}

}  // namespace

size_t route_workspace_bytes(int T, int m) {
  return T > 0 ? align_up((size_t)T * m * sizeof(float), 256) : 0;
}

hipError_t launch_route(const uint16_t* x, int T, const float* wr, const float* bias,
                        const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                        float* topk_w, float* gap, void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  float* z = static_cast<float*>(workspace);
  dim3 g1((T + kRouteTokens - 1) / kRouteTokens, (m + kRouteExperts - 1) / kRouteExperts);
  route_logits_kernel<<<g1, 256, 0, stream>>>(x, wr, bias, z, T, H, m);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  route_topk_kernel<<<(T + 3) / 4, 256, 0, stream>>>(z, keep_mask, T, m, k, topk_ids, topk_w, gap);
  return hipGetLastError();
}

}  // namespace sw
