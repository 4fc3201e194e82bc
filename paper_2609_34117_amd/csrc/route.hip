// Router of the MoE layer on gfx950: fp32 logits, masked top-k selection and
// renormalised gates (Section 3.1, Eq. 2 and the renormalisation after it).
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kMaxPool = 1024;

// fp32 w = hi + mid + lo exactly, each piece a bf16 (truncating split: hi
// keeps the top 8 significand bits, mid the next 8, lo the last 8), for
// eight weights at once; returns the three packed bf16x8 operands.
__device__ __forceinline__ void split3_bf16x8(const float4& a, const float4& b, u32x4& hi,
                                              u32x4& mid, u32x4& lo) {
  const float w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  uint32_t h[8], md[8], l[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t u = __float_as_uint(w[i]);
    h[i] = u & 0xffff0000u;
    const float r1 = w[i] - __uint_as_float(h[i]);
    md[i] = __float_as_uint(r1) & 0xffff0000u;
    l[i] = __float_as_uint(r1 - __uint_as_float(md[i]));
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    hi[q] = (h[2 * q] >> 16) | h[2 * q + 1];
    mid[q] = (md[2 * q] >> 16) | md[2 * q + 1];
    lo[q] = (l[2 * q] >> 16) | (l[2 * q + 1] & 0xffff0000u);
  }
}

// z[t, e] = sum_h x[t, h] * wr[e, h]  (+ bias[e]), fp32.
// Block = KW waves; tile = 16 experts x 16 tokens; the waves split H.  The
// router row is split exactly into three bf16 pieces, so each 32-wide K
// step is three bf16 MFMAs whose products are exact in fp32.
template <int KW>
__global__ __launch_bounds__(64 * KW) void route_logits_kernel(const uint16_t* __restrict__ x,
                                                              const float* __restrict__ wr,
                                                              const float* __restrict__ bias,
                                                              float* __restrict__ z, int T, int H,
                                                              int m) {
  constexpr int kChunk = 4;  // K steps whose loads are issued together
  __shared__ f32x4 part[KW][kWave];
  const int t0 = blockIdx.x * 16, e0 = blockIdx.y * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, kg = lane >> 4;
  const auto w_rsrc = make_rsrc(wr, 4u * (uint32_t)m * (uint32_t)H);
  const auto x_rsrc = make_rsrc(x, 2u * (uint32_t)T * (uint32_t)H);
  const bool e_ok = e0 + r < m, t_ok = t0 + r < T;
  const uint32_t w_row = (uint32_t)(e0 + r) * H * 4u, x_row = (uint32_t)(t0 + r) * H * 2u;
  const int nsteps = (H + 31) >> 5;
  const int s_lo = (wave * nsteps) / KW, s_hi = ((wave + 1) * nsteps) / KW;

  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int sb = s_lo; sb < s_hi; sb += kChunk) {
    u32x4 wa[kChunk], wb[kChunk], xb[kChunk];
#pragma unroll
    for (int c = 0; c < kChunk; ++c) {
      const int col = (sb + c) * 32 + kg * 8;
      const bool ok = sb + c < s_hi && col < H;
      const uint32_t wo = (ok && e_ok) ? w_row + (uint32_t)col * 4u : kOutOfRange;
      wa[c] = buf_ld128(w_rsrc, wo);
      wb[c] = buf_ld128(w_rsrc, wo + 16u);
      xb[c] = buf_ld128(x_rsrc, (ok && t_ok) ? x_row + (uint32_t)col * 2u : kOutOfRange);
    }
#pragma unroll
    for (int c = 0; c < kChunk; ++c) {
      u32x4 hi, mid, lo;
      split3_bf16x8(__builtin_bit_cast(float4, wa[c]), __builtin_bit_cast(float4, wb[c]), hi, mid, lo);
      acc = mfma_16x16x32(hi, xb[c], acc);
      acc = mfma_16x16x32(mid, xb[c], acc);
      acc = mfma_16x16x32(lo, xb[c], acc);
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    f32x4 c = part[0][lane];
#pragma unroll
    for (int w = 1; w < KW; ++w) c += part[w][lane];
    // c[i] = z for expert e0 + 4*kg + i, token t0 + r
    const int t = t0 + r;
    if (t < T) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = e0 + 4 * kg + i;
        if (e < m) z[(size_t)t * m + e] = bias ? c[i] + bias[e] : c[i];
      }
    }
  }
}

// One wave per token: top-k over the eligible experts by (z desc, id asc),
// then softmax over the k selected logits.  Each round takes the largest
// remaining order key with a DPP max and, among lanes holding it, the
// smallest expert id with a DPP min.  KPL = keys per lane (ceil(m / 64)).
template <int KPL>
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
  // order key of each logit; 0 marks "not eligible or already taken" (the
  // one logit whose key is 0, a NaN, is nudged to 1)
  uint32_t key[KPL];
#pragma unroll
  for (int q = 0; q < KPL; ++q) {
    const int e = q * 64 + lane;
    const bool ok = e < m && (keep_mask == nullptr || keep_mask[e] != 0);
    key[q] = ok ? max(f32_order_key(zt[e]), 1u) : 0u;
  }

  int my_id = -1;
  float my_z = 0.f, zk = 0.f, zk1 = 0.f;
  bool complete = true, have_next = false;
  for (int j = 0; j <= k; ++j) {
    uint32_t lm = key[0];
#pragma unroll
    for (int q = 1; q < KPL; ++q) lm = key[q] > lm ? key[q] : lm;
    const uint32_t best = wave_max_u32(lm);
    if (best == 0) {  // wave-uniform: no eligible expert left
      if (j < k) complete = false;
      break;
    }
    const float ze = f32_from_order_key(best);
    if (j == k) {
      zk1 = ze;
      have_next = true;
      break;
    }
    uint32_t cand = 0xffffffffu;
#pragma unroll
    for (int q = KPL - 1; q >= 0; --q) cand = key[q] == best ? (uint32_t)(q * 64 + lane) : cand;
    const int e = (int)wave_min_u32(cand);
    if (lane == j) {
      my_id = e;
      my_z = ze;
    }
    if (j == k - 1) zk = ze;
#pragma unroll
    for (int q = 0; q < KPL; ++q)
      if (q * 64 + lane == e) key[q] = 0u;
  }

  const float z0 = __shfl(my_z, 0);
  const float ex = (lane < k && my_id >= 0) ? expf(my_z - z0) : 0.f;
  const float s = wave_sum_f32(ex);
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

template <int KPL>
static void launch_topk_t(const float* z, const uint8_t* keep_mask, int T, int m, int k,
                          int* topk_ids, float* topk_w, float* gap, hipStream_t stream) {
  route_topk_kernel<KPL><<<(T + 3) / 4, 256, 0, stream>>>(z, keep_mask, T, m, k, topk_ids, topk_w,
                                                          gap);
}

hipError_t launch_route(const uint16_t* x, int T, const float* wr, const float* bias,
                        const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                        float* topk_w, float* gap, void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  float* z = static_cast<float*>(workspace);
  const dim3 grid((T + 15) / 16, (m + 15) / 16);
  // few output tiles: spread H over 16 waves per tile (one load round trip
  // per wave at H = 2048); many: 2 waves
  if ((long)grid.x * grid.y < 1024)
    route_logits_kernel<16><<<grid, 1024, 0, stream>>>(x, wr, bias, z, T, H, m);
  else
    route_logits_kernel<2><<<grid, 128, 0, stream>>>(x, wr, bias, z, T, H, m);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int kpl = (m + 63) / 64;
  if (kpl <= 1)
    launch_topk_t<1>(z, keep_mask, T, m, k, topk_ids, topk_w, gap, stream);
  else if (kpl <= 2)
    launch_topk_t<2>(z, keep_mask, T, m, k, topk_ids, topk_w, gap, stream);
  else if (kpl <= 4)
    launch_topk_t<4>(z, keep_mask, T, m, k, topk_ids, topk_w, gap, stream);
  else if (kpl <= 8)
    launch_topk_t<8>(z, keep_mask, T, m, k, topk_ids, topk_w, gap, stream);
  else
    launch_topk_t<16>(z, keep_mask, T, m, k, topk_ids, topk_w, gap, stream);
  return hipGetLastError();
}

}  // namespace sw
