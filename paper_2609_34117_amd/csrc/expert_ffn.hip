// Expert FFNs of the MoE layer on gfx950 (Section 2.1: each step reads the
// weights of every distinct expert selected across the batch).
//
// Every active expert's bf16 weights are streamed from HBM exactly once per
// call with 128-bit loads straight into matrix-core operand registers; the
// expert's tokens form the narrow side of a 16x16x32 bf16 MFMA (padded to
// 16 columns), so decode's handful of tokens per expert costs almost no
// issue time and there is no cross-lane reduction over the hidden size.
//
//   gate_up: block = 4 waves, tile = (expert, 8 intermediate indices).  The
//            16 A rows are the 8 gate rows and the 8 matching up rows; the
//            waves split H four ways and add their partial tiles in LDS.
//            Epilogue: h = silu(g) * u, stored as a bf16 hi/lo pair
//            (h ~= hi + lo to ~16 mantissa bits) in dispatch-slot order.
//   down:    block = 4 waves, tile = (expert, 64 output rows); each wave
//            owns 16 rows over the full I.  B = h hi and lo, two MFMAs.
//   combine: out[t] = sum_j w[t, j] y[t*k + j] in slot order.
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kKSteps = 16;   // 32-column K steps of weights held in registers per wave
constexpr int kNBlocks = 4;   // 16-token column blocks per pass (64 tokens)
constexpr int kPassTokens = 16 * kNBlocks;

struct ForwardWs {
  uint16_t* h_hi;
  uint16_t* h_lo;
  float* y;
};

__host__ __device__ inline size_t h_bytes(int n_pairs, int I) {
  return align_up((size_t)n_pairs * I * sizeof(uint16_t), 256);
}

__host__ __device__ inline ForwardWs carve(void* ws, int n_pairs, int I) {
  char* p = static_cast<char*>(ws);
  ForwardWs w;
  w.h_hi = reinterpret_cast<uint16_t*>(p);
  w.h_lo = reinterpret_cast<uint16_t*>(p + h_bytes(n_pairs, I));
  w.y = reinterpret_cast<float*>(p + 2 * h_bytes(n_pairs, I));
  return w;
}

// Resolves a streaming tile to (expert, count, first slot); false if the
// tile is surplus or the dispatch plan is inconsistent.
__device__ __forceinline__ bool tile_expert(int tile, int tpe, const int* active,
                                            const int* counts, const int* offsets, int m,
                                            int n_pairs, int* a_out, int* e_out, int* cnt_out,
                                            int* base_out) {
  if (tile < 0) return false;
  const int a = tile / tpe;
  const int e = active[a];
  if (e < 0 || e >= m) return false;
  const int cnt = counts[e], base = offsets[e];
  if (cnt <= 0 || base < 0 || cnt > n_pairs - base) return false;
  *a_out = a;
  *e_out = e;
  *cnt_out = cnt;
  *base_out = base;
  return true;
}

__global__ __launch_bounds__(256) void gate_up_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w13,
    const int* __restrict__ counts, const int* __restrict__ offsets,
    const int* __restrict__ perm, const int* __restrict__ active,
    const int* __restrict__ n_active_p, uint16_t* __restrict__ h_hi,
    uint16_t* __restrict__ h_lo, int H, int I, int m, int k, int n_pairs) {
  __shared__ f32x4 part[4][kNBlocks][kWave];
  const int n_act = *n_active_p;
  if (n_act <= 0 || n_act > m) return;
  const int tpe = I / 8;
  int a, e, cnt, base;
  const int tile = xcd_tile(blockIdx.x, n_act * tpe);
  if (!tile_expert(tile, tpe, active, counts, offsets, m, n_pairs, &a, &e, &cnt, &base)) return;
  const int ib = tile - a * tpe;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, kg = lane >> 4;
  const int wrow = r < 8 ? ib * 8 + r : I + ib * 8 + (r - 8);
  const uint16_t* arow = w13 + ((size_t)e * 2 * I + wrow) * H + kg * 8;
  const int nsteps = (H + 31) >> 5;
  const int s_lo = (wave * nsteps) >> 2, s_hi = ((wave + 1) * nsteps) >> 2;

  for (int t0 = 0; t0 < cnt; t0 += kPassTokens) {
    const int nbn = (min(kPassTokens, cnt - t0) + 15) >> 4;
    const uint16_t* xrow[kNBlocks];
#pragma unroll
    for (int nb = 0; nb < kNBlocks; ++nb) {
      xrow[nb] = nullptr;
      const int slot = t0 + nb * 16 + r;
      if (slot < cnt) {
        const int p = perm[base + slot];
        if (p >= 0 && p < n_pairs) xrow[nb] = x + (size_t)(p / k) * H + kg * 8;
      }
    }
    f32x4 acc[kNBlocks];
#pragma unroll
    for (int nb = 0; nb < kNBlocks; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int s0 = s_lo; s0 < s_hi; s0 += kKSteps) {
      u32x4 A[kKSteps];
#pragma unroll
      for (int s = 0; s < kKSteps; ++s) {
        const int col = (s0 + s) * 32;
        A[s] = (s0 + s < s_hi && col + kg * 8 < H) ? ld128_stream(arow + col) : zero4();
      }
#pragma unroll
      for (int nb = 0; nb < kNBlocks; ++nb) {
        if (nb < nbn) {
#pragma unroll
          for (int s = 0; s < kKSteps; ++s) {
            if (s0 + s < s_hi) {
              const int col = (s0 + s) * 32;
              const u32x4 B =
                  (xrow[nb] != nullptr && col + kg * 8 < H) ? ld128(xrow[nb] + col) : zero4();
              acc[nb] = mfma_16x16x32(A[s], B, acc[nb]);
            }
          }
        }
      }
    }

#pragma unroll
    for (int nb = 0; nb < kNBlocks; ++nb)
      if (nb < nbn) part[wave][nb][lane] = acc[nb];
    __syncthreads();
    if (wave < nbn) {
      const int nb = wave;
      const f32x4 c = ((part[0][nb][lane] + part[1][nb][lane]) + part[2][nb][lane]) +
                      part[3][nb][lane];
      // rows 0-7 (gate) live in lanes 0-31, the matching up rows 8-15 in
      // lanes 32-63 at the same token column
      f32x4 u;
#pragma unroll
      for (int q = 0; q < 4; ++q) u[q] = __shfl_xor(c[q], 32);
      const int slot = t0 + nb * 16 + r;
      if (lane < 32 && slot < cnt) {
        uint32_t hw[2], lw[2];
#pragma unroll
        for (int q = 0; q < 4; q += 2) {
          uint16_t hb[2], lb[2];
#pragma unroll
          for (int d = 0; d < 2; ++d) {
            const float g = c[q + d];
            const float hv = (g / (1.0f + expf(-g))) * u[q + d];
            hb[d] = f32_to_bf16(hv);
            lb[d] = f32_to_bf16(hv - bf16_to_f32(hb[d]));
          }
          hw[q / 2] = (uint32_t)hb[0] | ((uint32_t)hb[1] << 16);
          lw[q / 2] = (uint32_t)lb[0] | ((uint32_t)lb[1] << 16);
        }
        const size_t off = (size_t)(base + slot) * I + ib * 8 + kg * 4;
        *reinterpret_cast<uint2*>(h_hi + off) = make_uint2(hw[0], hw[1]);
        *reinterpret_cast<uint2*>(h_lo + off) = make_uint2(lw[0], lw[1]);
      }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void down_kernel(
    const uint16_t* __restrict__ h_hi, const uint16_t* __restrict__ h_lo,
    const uint16_t* __restrict__ w2, const int* __restrict__ counts,
    const int* __restrict__ offsets, const int* __restrict__ perm,
    const int* __restrict__ active, const int* __restrict__ n_active_p, float* __restrict__ y,
    int H, int I, int m, int n_pairs) {
  const int n_act = *n_active_p;
  if (n_act <= 0 || n_act > m) return;
  const int tpe = (H + 63) / 64;
  int a, e, cnt, base;
  const int tile = xcd_tile(blockIdx.x, n_act * tpe);
  if (!tile_expert(tile, tpe, active, counts, offsets, m, n_pairs, &a, &e, &cnt, &base)) return;
  const int ob = tile - a * tpe;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, kg = lane >> 4;
  const int orow = ob * 64 + wave * 16 + r;
  const bool row_ok = orow < H;
  const uint16_t* arow = w2 + ((size_t)e * H + (row_ok ? orow : 0)) * I + kg * 8;
  const int nsteps = (I + 31) >> 5;
  const int o_store = ob * 64 + wave * 16 + kg * 4;  // first of the 4 rows this lane stores

  for (int t0 = 0; t0 < cnt; t0 += kPassTokens) {
    const int nbn = (min(kPassTokens, cnt - t0) + 15) >> 4;
    long hoff[kNBlocks];
#pragma unroll
    for (int nb = 0; nb < kNBlocks; ++nb) {
      const int slot = t0 + nb * 16 + r;
      hoff[nb] = slot < cnt ? (long)(base + slot) * I + kg * 8 : -1;
    }
    f32x4 acc[kNBlocks];
#pragma unroll
    for (int nb = 0; nb < kNBlocks; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int s0 = 0; s0 < nsteps; s0 += kKSteps) {
      u32x4 A[kKSteps];
#pragma unroll
      for (int s = 0; s < kKSteps; ++s) {
        const int col = (s0 + s) * 32;
        A[s] = (s0 + s < nsteps && row_ok && col + kg * 8 < I) ? ld128_stream(arow + col)
                                                                : zero4();
      }
#pragma unroll
      for (int nb = 0; nb < kNBlocks; ++nb) {
        if (nb < nbn) {
#pragma unroll
          for (int s = 0; s < kKSteps; ++s) {
            if (s0 + s < nsteps) {
              const int col = (s0 + s) * 32;
              const bool ok = hoff[nb] >= 0 && col + kg * 8 < I;
              const u32x4 bh = ok ? ld128(h_hi + hoff[nb] + col) : zero4();
              const u32x4 bl = ok ? ld128(h_lo + hoff[nb] + col) : zero4();
              acc[nb] = mfma_16x16x32(A[s], bh, acc[nb]);
              acc[nb] = mfma_16x16x32(A[s], bl, acc[nb]);
            }
          }
        }
      }
    }

#pragma unroll
    for (int nb = 0; nb < kNBlocks; ++nb) {
      const int slot = t0 + nb * 16 + r;
      if (nb < nbn && slot < cnt && o_store < H) {
        const int p = perm[base + slot];
        if (p >= 0 && p < n_pairs) {
          const f32x4 c = acc[nb];
          *reinterpret_cast<float4*>(y + (size_t)p * H + o_store) = make_float4(c[0], c[1], c[2], c[3]);
        }
      }
    }
  }
}

__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ y,
                                                     const float* __restrict__ topk_w,
                                                     const int* __restrict__ n_active_p,
                                                     float* __restrict__ out, int T, int H,
                                                     int k, int m) {
  const int hq = H >> 2;
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)T * hq) return;
  const int t = (int)(idx / hq), c = (int)(idx - (size_t)t * hq);
  const int na = *n_active_p;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (na < 0 || na > m) {
    const float nan = __builtin_nanf("");
    acc = make_float4(nan, nan, nan, nan);
  } else {
    for (int j = 0; j < k; ++j) {
      const float wj = topk_w[(size_t)t * k + j];
      const float4 v = *reinterpret_cast<const float4*>(y + ((size_t)t * k + j) * H + 4 * c);
      acc.x = fmaf(wj, v.x, acc.x);
      acc.y = fmaf(wj, v.y, acc.y);
      acc.z = fmaf(wj, v.z, acc.z);
      acc.w = fmaf(wj, v.w, acc.w);
    }
  }
  *reinterpret_cast<float4*>(out + (size_t)t * H + 4 * c) = acc;
}

}  // namespace

size_t forward_workspace_bytes(int T, int H, int I, int k) {
  if (T <= 0) return 0;
  const int n_pairs = T * k;
  return 2 * h_bytes(n_pairs, I) + align_up((size_t)n_pairs * H * sizeof(float), 256);
}

hipError_t launch_gate_up(const uint16_t* x, int T, const uint16_t* w13, const int* counts,
                          const int* offsets, const int* perm, const int* active,
                          const int* n_active, int H, int I, int m, int k, void* workspace,
                          hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const ForwardWs ws = carve(workspace, T * k, I);
  const long tiles = (long)m * (I / 8);
  const int blocks = (int)align_up((size_t)tiles, 8);
  gate_up_kernel<<<blocks, 256, 0, stream>>>(x, w13, counts, offsets, perm, active, n_active,
                                             ws.h_hi, ws.h_lo, H, I, m, k, T * k);
  return hipGetLastError();
}

hipError_t launch_down(int T, const uint16_t* w2, const int* counts, const int* offsets,
                       const int* perm, const int* active, const int* n_active, int H, int I,
                       int m, int k, void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const ForwardWs ws = carve(workspace, T * k, I);
  const long tiles = (long)m * ((H + 63) / 64);
  const int blocks = (int)align_up((size_t)tiles, 8);
  down_kernel<<<blocks, 256, 0, stream>>>(ws.h_hi, ws.h_lo, w2, counts, offsets, perm, active,
                                          n_active, ws.y, H, I, m, T * k);
  return hipGetLastError();
}

hipError_t launch_combine(int T, const float* topk_w, const int* n_active, float* out, int H,
                          int I, int m, int k, void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const ForwardWs ws = carve(workspace, T * k, I);
  const size_t threads = (size_t)T * (H / 4);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  combine_kernel<<<blocks, 256, 0, stream>>>(ws.y, topk_w, n_active, out, T, H, k, m);
  return hipGetLastError();
}

}  // namespace sw
