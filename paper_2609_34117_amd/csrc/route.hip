// Router of the MoE layer on gfx950: fp32 logits, masked top-k selection and
// renormalised gates (Section 3.1, Eq. 2 and the renormalisation after it),
// and the fused route + dispatch of small (decode-sized) batches.
#include "dispatch_block.h"
#include "sw_launch.h"

namespace sw {
namespace {

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

// Partial logits part[ks][t][e] = sum over the ks-th slice of H of
// x[t, h] * wr[e, h], fp32.  Grid (token tiles, expert tiles, KS); a block
// is KW waves that split its slice; tile = 16 experts x 16 tokens.  The
// router row is split exactly into three bf16 pieces, so each 32-wide K step
// is three bf16 MFMAs whose products are exact in fp32.  Spreading H over KS
// blocks lets a decode-sized batch (few tiles) use many compute units.
template <int KW>
__global__ __launch_bounds__(64 * KW) void route_logits_kernel(const uint16_t* __restrict__ x,
                                                              const float* __restrict__ wr,
                                                              float* __restrict__ part, int T,
                                                              int H, int m) {
  constexpr int kChunk = 4;  // K steps whose loads are issued together
  __shared__ f32x4 red[KW][kWave];
  const int t0 = blockIdx.x * 16, e0 = blockIdx.y * 16, ks = blockIdx.z, KS = gridDim.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, kg = lane >> 4;
  const auto w_rsrc = make_rsrc(wr, 4u * (uint32_t)m * (uint32_t)H);
  const auto x_rsrc = make_rsrc(x, 2u * (uint32_t)T * (uint32_t)H);
  const bool e_ok = e0 + r < m, t_ok = t0 + r < T;
  const uint32_t w_row = (uint32_t)(e0 + r) * H * 4u, x_row = (uint32_t)(t0 + r) * H * 2u;
  const int nsteps = (H + 31) >> 5;
  const int b_lo = (ks * nsteps) / KS, b_hi = ((ks + 1) * nsteps) / KS;
  const int s_lo = b_lo + (wave * (b_hi - b_lo)) / KW;
  const int s_hi = b_lo + ((wave + 1) * (b_hi - b_lo)) / KW;

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
  red[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    f32x4 c = red[0][lane];
#pragma unroll
    for (int w = 1; w < KW; ++w) c += red[w][lane];
    // c[i] = partial z of expert e0 + 4*kg + i, token t0 + r
    const int t = t0 + r;
    if (t < T) {
      float* dst = part + ((size_t)ks * T + t) * m;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = e0 + 4 * kg + i;
        if (e < m) dst[e] = c[i];
      }
    }
  }
}

// Router logits of prefill-sized batches: a block of 4 waves computes a
// 64-token x 64-expert tile over slice blockIdx.z of H (KS = gridDim.z
// slices of whole 128-column chunks, so that several blocks share a compute
// unit and hide each other's load latency).  The tile's x
// rows are staged in LDS one 128-column chunk at a time (double-buffered),
// so each token row is read once per 64 experts instead of once per 16, and
// wave w reads the router rows of experts e0 + 16 w .. e0 + 16 w + 15
// directly: every router fragment, split into its three bf16 pieces once,
// feeds the 4 token blocks of the tile.  Same exact three-piece products as
// route_logits_kernel, accumulated over H in ascending order.
constexpr int kWideT = 64, kWideE = 64, kWideKc = 128, kWideRow = kWideKc + 8;

__global__ __launch_bounds__(256) void route_logits_wide_kernel(const uint16_t* __restrict__ x,
                                                               const float* __restrict__ wr,
                                                               float* __restrict__ part, int T,
                                                               int H, int m) {
  __shared__ uint16_t xs[2][kWideT * kWideRow];
  const int t0 = blockIdx.x * kWideT, e0 = blockIdx.y * kWideE;
  const int ks = blockIdx.z, KS = gridDim.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, kg = lane >> 4;
  const auto w_rsrc = make_rsrc(wr, 4u * (uint32_t)m * (uint32_t)H);
  const auto x_rsrc = make_rsrc(x, 2u * (uint32_t)T * (uint32_t)H);
  const int e = e0 + wave * 16 + r;
  const uint32_t w_row = (uint32_t)e * H * 4u;
  const int all = H / kWideKc;
  const int c_lo = (ks * all) / KS, c_hi = ((ks + 1) * all) / KS;

  // chunk c of the tile's x: 64 rows x 16 pieces of 8 columns, 4 per thread
  auto stage_load = [&](int c, u32x4 (&v)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = (int)threadIdx.x + j * 256, row = i >> 4, c8 = i & 15;
      const int t = t0 + row;
      v[j] = buf_ld128(x_rsrc, t < T ? ((uint32_t)t * H + (uint32_t)(c * kWideKc + c8 * 8)) * 2u
                                     : kOutOfRange);
    }
  };
  auto stage_store = [&](uint16_t* buf, const u32x4 (&v)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = (int)threadIdx.x + j * 256;
      *reinterpret_cast<u32x4*>(buf + (i >> 4) * kWideRow + (i & 15) * 8) = v[j];
    }
  };
  auto w_issue = [&](int c, u32x4 (&wa)[4], u32x4 (&wb)[4]) {
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const uint32_t off =
          e < m ? w_row + (uint32_t)(c * kWideKc + st * 32 + kg * 8) * 4u : kOutOfRange;
      wa[st] = buf_ld128(w_rsrc, off);
      wb[st] = buf_ld128(w_rsrc, off == kOutOfRange ? kOutOfRange : off + 16u);
    }
  };

  f32x4 acc[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  u32x4 v[4], wa[4], wb[4], na[4], nbw[4];
  stage_load(c_lo, v);
  w_issue(c_lo, wa, wb);
  stage_store(xs[c_lo & 1], v);
  for (int c = c_lo; c < c_hi; ++c) {
    __syncthreads();  // chunk c is in LDS; the other buffer is free
    const bool more = c + 1 < c_hi;
    if (more) {
      stage_load(c + 1, v);
      w_issue(c + 1, na, nbw);
    }
    const uint16_t* buf = xs[c & 1];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      u32x4 hi, mid, lo;
      split3_bf16x8(__builtin_bit_cast(float4, wa[st]), __builtin_bit_cast(float4, wb[st]), hi, mid,
                    lo);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const u32x4 b = *reinterpret_cast<const u32x4*>(buf + (nb * 16 + r) * kWideRow + st * 32 +
                                                        kg * 8);
        acc[nb] = mfma_16x16x32(hi, b, acc[nb]);
        acc[nb] = mfma_16x16x32(mid, b, acc[nb]);
        acc[nb] = mfma_16x16x32(lo, b, acc[nb]);
      }
    }
    if (more) {
      stage_store(xs[(c + 1) & 1], v);
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        wa[st] = na[st];
        wb[st] = nbw[st];
      }
    }
  }
  // acc[nb][i]: expert e0 + 16 wave + 4 kg + i, token t0 + 16 nb + r
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    const int t = t0 + nb * 16 + r;
    if (t < T) {
      float* dst = part + ((size_t)ks * T + t) * m;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ee = e0 + wave * 16 + 4 * kg + i;
        if (ee < m) dst[ee] = acc[nb][i];
      }
    }
  }
}

constexpr int kMaxSplit = 4;  // slices of H per logit tile

// Columns of a routing call: the m experts the top-k selects from, whose
// partial logits sit in rows of ld >= m columns (ld = m + 1 when the last
// column is the shared expert's gate logit), the k routed slots and the S
// slots of the shared expert's parts after them (ids m .. m + S - 1).
struct Cols {
  int m, ld, k, S;
  int R;  // token groups of the shared parts: the pool holds R copies of the S parts
  __device__ __host__ int plan_m() const { return m + R * S; }
};

// Token t's group of shared-part copies: R contiguous runs of the batch.
__device__ __forceinline__ int token_group(const Cols& c, int t, int T) {
  return c.R > 1 ? (int)((long long)t * c.R / T) : 0;
}

// Order key of token t's logit for expert e: z = sum of the KS partials in
// slice order, plus the bias; 0 marks an ineligible expert (the one logit
// whose key is 0, a NaN, is nudged to 1).  All partial loads are issued
// before the first add.
__device__ __forceinline__ uint32_t logit_key(const float* __restrict__ part, int KS, int T,
                                              const Cols& c, int t, int e,
                                              const float* __restrict__ bias,
                                              const uint8_t* __restrict__ keep_mask) {
  if (e >= c.m || (keep_mask != nullptr && keep_mask[e] == 0)) return 0u;
  const float* p = part + (size_t)t * c.ld + e;
  const size_t plane = (size_t)T * c.ld;
  float zp[kMaxSplit];
#pragma unroll
  for (int ks = 0; ks < kMaxSplit; ++ks) zp[ks] = ks < KS ? p[ks * plane] : 0.f;
  float z = zp[0];
#pragma unroll
  for (int ks = 1; ks < kMaxSplit; ++ks)
    if (ks < KS) z += zp[ks];
  if (bias != nullptr) z += bias[e];
  return max(f32_order_key(z), 1u);
}

// Gate of the shared expert for token t (Section 3.3): the sigmoid of its
// gate logit, the partials of column m summed in slice order like every
// other logit.
__device__ __forceinline__ float shared_gate(const float* __restrict__ part, int KS, int T,
                                             const Cols& c, int t) {
  const float* p = part + (size_t)t * c.ld + c.m;
  const size_t plane = (size_t)T * c.ld;
  float zp[kMaxSplit];
#pragma unroll
  for (int ks = 0; ks < kMaxSplit; ++ks) zp[ks] = ks < KS ? p[ks * plane] : 0.f;
  float z = zp[0];
#pragma unroll
  for (int ks = 1; ks < kMaxSplit; ++ks)
    if (ks < KS) z += zp[ks];
  return 1.0f / (1.0f + expf(-z));
}

// Reductions inside one 16-lane row (quad swaps, then the half-row and row
// mirrors): every lane of the row ends with the row's result.
template <typename Op>
__device__ __forceinline__ uint32_t row_reduce_u32(uint32_t v, uint32_t identity, Op op) {
  v = op(v, dpp_mov<dpp::kXor1>(identity, v));
  v = op(v, dpp_mov<dpp::kXor2>(identity, v));
  v = op(v, dpp_mov<dpp::kHalfMirror>(identity, v));
  v = op(v, dpp_mov<dpp::kMirror>(identity, v));
  return v;
}

// Result of one token's selection, held by the lanes of its row or wave:
// lane j < k holds slot j.
struct Selection {
  int id;        // expert id of this lane's slot, -1 if none
  float z;       // its logit
  float gate;    // renormalised gate (0 without an expert)
  float gap;     // z_(k) - z_(k+1); +inf if only k eligible; NaN if fewer
};

// The k + 1 selection rounds and the softmax over the k selected logits.
// Each round takes the largest remaining order key (a max reduction) and,
// among the lanes holding it, the smallest expert id (a min reduction); the
// (k+1)-th round only reads the runner-up for the gap.  The red_* functions
// reduce over the lanes that hold this token's keys (a row or the whole wave);
// `slot` is this lane's position among them.
template <int KPL, typename MaxOp, typename MinOp, typename SumOp>
__device__ __forceinline__ Selection select_topk(uint32_t (&key)[KPL], const int (&eid)[KPL],
                                                 int k, int slot, MaxOp red_max, MinOp red_min,
                                                 SumOp red_sum) {
  Selection s{-1, 0.f, 0.f, 0.f};
  float z_first = 0.f, zk = 0.f, zk1 = 0.f;
  bool complete = true, have_next = false;
  for (int j = 0; j <= k; ++j) {
    uint32_t lm = key[0];
#pragma unroll
    for (int q = 1; q < KPL; ++q) lm = key[q] > lm ? key[q] : lm;
    const uint32_t best = red_max(lm);
    const bool found = best != 0;  // uniform over the reducing lanes
    const float ze = f32_from_order_key(best);
    if (j == k) {
      if (found) {
        zk1 = ze;
        have_next = true;
      }
      break;
    }
    if (!found) complete = false;
    uint32_t cand = 0xffffffffu;
#pragma unroll
    for (int q = KPL - 1; q >= 0; --q) cand = key[q] == best ? (uint32_t)eid[q] : cand;
    const int e = (int)red_min(cand);
    if (found) {
      if (j == 0) z_first = ze;
      if (slot == j) {
        s.id = e;
        s.z = ze;
      }
      if (j == k - 1) zk = ze;
#pragma unroll
      for (int q = 0; q < KPL; ++q)
        if (eid[q] == e) key[q] = 0u;
    }
  }
  const float ex = (slot < k && s.id >= 0) ? expf(s.z - z_first) : 0.f;
  const float sum = red_sum(ex);
  s.gate = s.id >= 0 ? ex / sum : 0.f;
  s.gap = !complete ? __builtin_nanf("") : (have_next ? zk - zk1 : __builtin_inff());
  return s;
}

__device__ __forceinline__ uint32_t umax(uint32_t a, uint32_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint32_t umin(uint32_t a, uint32_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint32_t fadd_bits(uint32_t a, uint32_t b) {
  return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
}

// Top-k of one token per 16-lane row (four tokens per wave): lane r of the
// row holds the keys of experts q * 16 + r.  Needs m <= 16 * KPL and k <= 16.
// The softmax sum runs over the row with the same pairing as the wave
// variant's first four steps; the other rows only add +0 there, so both
// variants give identical gates.
template <int KPL>
__device__ __forceinline__ Selection select_row(const float* part, int KS, int T, const Cols& c,
                                                int t, const float* bias,
                                                const uint8_t* keep_mask) {
  const int r = threadIdx.x & 15;
  uint32_t key[KPL];
  int eid[KPL];
#pragma unroll
  for (int q = 0; q < KPL; ++q) {
    eid[q] = q * 16 + r;
    key[q] = t < T ? logit_key(part, KS, T, c, t, eid[q], bias, keep_mask) : 0u;
  }
  return select_topk<KPL>(
      key, eid, c.k, r, [](uint32_t v) { return row_reduce_u32(v, 0u, umax); },
      [](uint32_t v) { return row_reduce_u32(v, 0xffffffffu, umin); },
      [](float v) { return __uint_as_float(row_reduce_u32(__float_as_uint(v), 0u, fadd_bits)); });
}

// Top-k of one token per wave: lane l holds the keys of experts q * 64 + l.
template <int KPL>
__device__ __forceinline__ Selection select_wave(const float* part, int KS, int T, const Cols& c,
                                                 int t, const float* bias,
                                                 const uint8_t* keep_mask) {
  const int lane = threadIdx.x & 63;
  uint32_t key[KPL];
  int eid[KPL];
#pragma unroll
  for (int q = 0; q < KPL; ++q) {
    eid[q] = q * 64 + lane;
    key[q] = logit_key(part, KS, T, c, t, eid[q], bias, keep_mask);
  }
  return select_topk<KPL>(
      key, eid, c.k, lane, [](uint32_t v) { return wave_max_u32(v); },
      [](uint32_t v) { return wave_min_u32(v); }, [](float v) { return wave_sum_f32(v); });
}

// Slot `slot` of token t: a routed slot (slot < k) takes the selection,
// a shared slot k + s the shared expert's part m + s with the shared gate.
__device__ __forceinline__ int slot_id(const Selection& s, const Cols& c, int slot, int t, int T) {
  return slot < c.k ? s.id : c.m + token_group(c, t, T) * c.S + slot - c.k;
}

__device__ __forceinline__ void store_selection(const Selection& s, int t, int T, const Cols& c,
                                                int slot, float sgate,
                                                int* __restrict__ topk_ids,
                                                float* __restrict__ topk_w,
                                                float* __restrict__ gap) {
  const int kout = c.k + c.S;
  if (slot < kout) {
    topk_ids[(size_t)t * kout + slot] = slot_id(s, c, slot, t, T);
    topk_w[(size_t)t * kout + slot] = slot < c.k ? s.gate : sgate;
  }
  if (gap != nullptr && slot == 0) gap[t] = s.gap;
}

// ROW: one token per 16-lane row (16 tokens per 256-thread block), else one
// token per wave (4 per block).
template <int KPL, bool ROW>
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ part, int KS,
                                                        const float* __restrict__ bias,
                                                        const uint8_t* __restrict__ keep_mask,
                                                        int T, Cols c,
                                                        int* __restrict__ topk_ids,
                                                        float* __restrict__ topk_w,
                                                        float* __restrict__ gap) {
  if (ROW) {
    const int t = blockIdx.x * 16 + (threadIdx.x >> 4);
    const Selection s = select_row<KPL>(part, KS, T, c, t, bias, keep_mask);
    const float sg = (c.S > 0 && t < T) ? shared_gate(part, KS, T, c, t) : 0.f;
    if (t < T) store_selection(s, t, T, c, threadIdx.x & 15, sg, topk_ids, topk_w, gap);
  } else {
    const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;  // wave-uniform
    const Selection s = select_wave<KPL>(part, KS, T, c, t, bias, keep_mask);
    const float sg = c.S > 0 ? shared_gate(part, KS, T, c, t) : 0.f;
    store_selection(s, t, T, c, threadIdx.x & 63, sg, topk_ids, topk_w, gap);
  }
}

// Route + dispatch of a small batch in one 512-thread block: 16-lane row
// i selects token i (four tokens per wave; waves without a token skip the
// selection, so the busy waves have a SIMD each up to 16 tokens), the ids go
// to LDS as well as to memory, and the block then builds the dispatch plan
// from them (512 threads measured 0.4 us a step faster at one token than
// 1024: the plan's barriers and LDS clearing cover half the waves).  Larger
// batches take the multi-block top-k kernel and the dispatch kernel: one
// block would serialise their selections and plan (a 1024-thread block for
// 33-64 tokens measured 8.9 us at 64 tokens over 64 experts and 11.3 us
// over 128, against 9.2 us for the two kernels).
constexpr int kFusedThreads = 512;
constexpr int kFusedMaxPool = 256;
constexpr int kFusedMaxTokens = 32;
constexpr int kFusedMaxK = 16;
constexpr int kWaveFusedTokens = 4;  // one wave: 4 rows of 16 lanes, <= 64 pairs

template <int KPL>
__global__ __launch_bounds__(kFusedThreads) void route_select_dispatch_kernel(
    const float* __restrict__ part, int KS, const float* __restrict__ bias,
    const uint8_t* __restrict__ keep_mask, int T, Cols c, int* __restrict__ topk_ids,
    float* __restrict__ topk_w, float* __restrict__ gap, int* __restrict__ counts,
    int* __restrict__ offsets, int* __restrict__ perm, int* __restrict__ active,
    int* __restrict__ n_active) {
  __shared__ int ids_s[kFusedMaxTokens * kFusedMaxK];
  __shared__ int cursor[kFusedMaxPool];
  __shared__ int wave_base[(kFusedThreads / kWave) * kFusedMaxPool];
  __shared__ uint8_t wave_cnt[(kFusedThreads / kWave) * kFusedMaxPool];
  __shared__ uint32_t scan_scratch[34];
  __shared__ int bad;
  const int t = threadIdx.x >> 4, r = threadIdx.x & 15;
  const int kout = c.k + c.S;
  if ((threadIdx.x >> 6) * 4 < T) {  // wave-uniform
    const Selection s = select_row<KPL>(part, KS, T, c, t, bias, keep_mask);
    const float sg = (c.S > 0 && t < T) ? shared_gate(part, KS, T, c, t) : 0.f;
    if (t < T) {
      store_selection(s, t, T, c, r, sg, topk_ids, topk_w, gap);
      if (r < kout) ids_s[t * kout + r] = slot_id(s, c, r, t, T);
    }
  }
  __syncthreads();
  const DispatchLds lds{cursor, wave_base, wave_cnt, scan_scratch, &bad};
  dispatch_block(ids_s, T * kout, c.plan_m(), lds, counts, offsets, perm, active, n_active);
}

// Route + dispatch of at most 4 tokens (at most 64 pairs) in one wave: the
// rows of 16 lanes select the tokens as above, then lane q takes pair q's id
// and the wave builds the plan with ballots and wave scans, without a
// barrier.  Expert i's count and offset live on lane i % 64, slot i / 64
// (m <= 256).  The plan is the one dispatch_block builds, value for value.
template <int KPL>
__global__ __launch_bounds__(64) void route_select_dispatch_wave_kernel(
    const float* __restrict__ part, int KS, const float* __restrict__ bias,
    const uint8_t* __restrict__ keep_mask, int T, Cols c, int* __restrict__ topk_ids,
    float* __restrict__ topk_w, float* __restrict__ gap, int* __restrict__ counts,
    int* __restrict__ offsets, int* __restrict__ perm, int* __restrict__ active,
    int* __restrict__ n_active) {
  const int lane = threadIdx.x, t = lane >> 4, r = lane & 15;
  const Selection s = select_row<KPL>(part, KS, T, c, t, bias, keep_mask);
  const float sg = (c.S > 0 && t < T) ? shared_gate(part, KS, T, c, t) : 0.f;
  if (t < T) store_selection(s, t, T, c, r, sg, topk_ids, topk_w, gap);
  // the plan covers the m selectable experts and the S shared parts (<= 256
  // in all), kout slots a token; pair q = t' * kout + j is slot j of lane
  // 16 t' + j
  const int kout = c.k + c.S, m = c.plan_m();
  const int n_pairs = T * kout;
  const bool valid = lane < n_pairs;
  const int e = __shfl(slot_id(s, c, r, t, T), valid ? (lane / kout) * 16 + lane % kout : 0);
  if (__ballot(valid && (e < 0 || e >= m)) != 0) {  // the flagged plan
    for (int i = lane; i <= m; i += 64) {
      if (i < m) counts[i] = 0;
      offsets[i] = 0;
    }
    if (valid) perm[lane] = lane;
    if (lane == 0) *n_active = -1;
    return;
  }
  int cnt[4] = {0, 0, 0, 0};
  for (int q = 0; q < n_pairs; ++q) {
    const int eq = __builtin_amdgcn_readlane(e, q);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j == (eq >> 6) && lane == (eq & 63)) ++cnt[j];
  }
  // offsets = exclusive scan of the counts, active = the experts with pairs,
  // both in expert order (slot-major)
  int off[4] = {0, 0, 0, 0};
  uint32_t run_off = 0, run_act = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j * 64 >= m) break;  // uniform
    const int i = j * 64 + lane;
    const uint32_t c = i < m ? (uint32_t)cnt[j] : 0u, a = c > 0 ? 1u : 0u;
    const uint32_t ic = wave_inclusive_scan_u32(c), ia = wave_inclusive_scan_u32(a);
    off[j] = (int)(run_off + ic - c);
    if (i < m) {
      counts[i] = (int)c;
      offsets[i] = off[j];
      if (c > 0) active[run_act + ia - a] = i;
    }
    run_off += __builtin_amdgcn_readlane(ic, 63);
    run_act += __builtin_amdgcn_readlane(ia, 63);
  }
  if (lane == 0) {
    offsets[m] = (int)run_off;
    *n_active = (int)run_act;
  }
  // stable scatter: pair q goes after the earlier pairs of its expert
  const uint64_t peers = match_peers(e, valid, id_bits(m));
  const int rank = __popcll(peers & ((1ull << lane) - 1ull));
  int base = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = __shfl(off[j], e & 63);
    if (j == (e >> 6)) base = v;
  }
  if (valid) perm[base + rank] = lane;
}

// Split of the router contraction for T tokens and m experts: KW waves per
// block, KS slices of H (blocks per output tile).  Few tiles (decode): 4
// waves and up to 4 slices of H, so that about 256 blocks share the router
// bytes; many tiles (prefill): route_logits_wide_kernel's 64 x 64 tiles over
// slices of at least 8 chunks of H (2 at H = 2048), or, when H is not a
// whole number of chunks, 2-wave 16 x 16 tiles and no split.
struct LogitsSplit {
  int kw, ks;
  bool wide;  // route_logits_wide_kernel
};

LogitsSplit logits_split(int T, int H, int m) {
  const long tiles = (long)((T + 15) / 16) * ((m + 15) / 16);
  if (tiles >= 1024) {
    if (H % kWideKc != 0) return {2, 1, false};
    // >= 8 chunks a slice: at 4096 tokens, 2 slices of 8 chunks measured
    // faster than 4 of 4, 3 of 5-6 or one of 16
    return {4, std::min(kMaxSplit, std::max(1, H / kWideKc / 8)), true};
  }
  const int nsteps = (H + 31) / 32;
  const int max_ks = std::min(kMaxSplit, std::max(1, nsteps / 16));  // waves keep >= 4 K steps
  const long want = (256 + tiles - 1) / tiles;
  return {4, (int)std::max<long>(1, std::min<long>(want, max_ks)), false};
}

hipError_t launch_logits(const uint16_t* x, int T, const float* wr, int H, int m, float* part,
                         const LogitsSplit& sp, hipStream_t stream) {
  if (sp.wide) {
    const dim3 wgrid((T + kWideT - 1) / kWideT, (m + kWideE - 1) / kWideE, sp.ks);
    route_logits_wide_kernel<<<wgrid, 256, 0, stream>>>(x, wr, part, T, H, m);
    return hipGetLastError();
  }
  const dim3 grid((T + 15) / 16, (m + 15) / 16, sp.ks);
  if (sp.kw == 4)
    route_logits_kernel<4><<<grid, 256, 0, stream>>>(x, wr, part, T, H, m);
  else
    route_logits_kernel<2><<<grid, 128, 0, stream>>>(x, wr, part, T, H, m);
  return hipGetLastError();
}

template <int KPL, bool ROW>
void launch_topk_t(const float* part, int KS, const float* bias, const uint8_t* keep_mask, int T,
                   const Cols& c, int* topk_ids, float* topk_w, float* gap, hipStream_t stream) {
  const int per_block = ROW ? 16 : 4;
  route_topk_kernel<KPL, ROW><<<(T + per_block - 1) / per_block, 256, 0, stream>>>(
      part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap);
}

void launch_topk(const float* part, int KS, const float* bias, const uint8_t* keep_mask, int T,
                 const Cols& c, int* topk_ids, float* topk_w, float* gap, hipStream_t stream) {
  // one token per 16-lane row for small batches; from 64 tokens on, one token
  // per wave (more waves in flight) measured faster: 8.3 against 12.5 us at
  // 4096 tokens, 2-3% of a 40-layer batch-256 step, 2 us of a batch-64 step
  // over 128 experts
  if (c.k + c.S <= 16 && c.m <= 256 && T < 64) {
    const int kpl = (c.m + 15) / 16;
    if (kpl <= 4)
      launch_topk_t<4, true>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
    else if (kpl <= 8)
      launch_topk_t<8, true>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
    else
      launch_topk_t<16, true>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
    return;
  }
  const int kpl = (c.m + 63) / 64;
  if (kpl <= 1)
    launch_topk_t<1, false>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
  else if (kpl <= 2)
    launch_topk_t<2, false>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
  else if (kpl <= 4)
    launch_topk_t<4, false>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
  else if (kpl <= 8)
    launch_topk_t<8, false>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
  else
    launch_topk_t<16, false>(part, KS, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
}

// ---------------------------------------------------------------------------
// Routing-mass statistics (Section 2.3: an importance criterion aggregating
// the router's gate probabilities over calibration tokens).

// Token t's logit for expert e: the KS partials in slice order, plus bias.
__device__ __forceinline__ float logit_value(const float* __restrict__ part, int KS, int T, int m,
                                             int t, int e, const float* __restrict__ bias) {
  const float* p = part + (size_t)t * m + e;
  const size_t plane = (size_t)T * m;
  float z = p[0];
  for (int ks = 1; ks < KS; ++ks) z += p[ks * plane];
  if (bias != nullptr) z += bias[e];
  return z;
}

// One wave per token: the largest eligible logit and the softmax
// denominator over the eligible experts.
__global__ __launch_bounds__(256) void mass_token_stats_kernel(
    const float* __restrict__ part, int KS, const float* __restrict__ bias,
    const uint8_t* __restrict__ keep_mask, int T, int m, float* __restrict__ zmax,
    float* __restrict__ denom) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // wave-uniform
  uint32_t best = 0u;  // order key; 0 = no eligible expert on this lane
  for (int e = lane; e < m; e += kWave)
    if (keep_mask == nullptr || keep_mask[e] != 0)
      best = max(best, max(f32_order_key(logit_value(part, KS, T, m, t, e, bias)), 1u));
  best = wave_max_u32(best);
  const float zm = f32_from_order_key(best);
  float s = 0.f;
  for (int e = lane; e < m; e += kWave)
    if (keep_mask == nullptr || keep_mask[e] != 0)
      s += expf(logit_value(part, KS, T, m, t, e, bias) - zm);
  s = wave_sum_f32(s);
  if (lane == 0) {
    zmax[t] = zm;
    denom[t] = s;
  }
}

// One thread per expert: the token-ordered sum of its softmax share and of
// the gates it received (its dispatch slots in order), added to the masses.
__global__ __launch_bounds__(256) void mass_accumulate_kernel(
    const float* __restrict__ part, int KS, const float* __restrict__ bias,
    const uint8_t* __restrict__ keep_mask, int T, int m, const float* __restrict__ zmax,
    const float* __restrict__ denom, const float* __restrict__ topk_w,
    const int* __restrict__ counts, const int* __restrict__ offsets,
    const int* __restrict__ perm, const int* __restrict__ n_active, int n_pairs,
    float* __restrict__ mass_softmax, float* __restrict__ mass_topk) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= m) return;
  if (mass_softmax != nullptr && (keep_mask == nullptr || keep_mask[e] != 0)) {
    float acc = 0.f;
    for (int t = 0; t < T; ++t)
      acc += expf(logit_value(part, KS, T, m, t, e, bias) - zmax[t]) / denom[t];
    mass_softmax[e] += acc;
  }
  if (mass_topk != nullptr && *n_active >= 0) {
    const int b = offsets[e], c = counts[e];
    float acc = 0.f;
    if (b >= 0 && c >= 0 && c <= n_pairs - b)
      for (int i = 0; i < c; ++i) {
        const int p = perm[b + i];
        if (p >= 0 && p < n_pairs) acc += topk_w[p];
      }
    mass_topk[e] += acc;
  }
}

}  // namespace

size_t routing_mass_workspace_bytes(int T, int H, int m, int k) {
  if (T <= 0) return 0;
  const size_t P = (size_t)T * k;
  return route_workspace_bytes(T, H, m, k) + 3 * align_up(P * 4, 256) +
         3 * align_up((size_t)(m + 1) * 4, 256) + 256 + 2 * align_up((size_t)T * 4, 256);
}

hipError_t launch_routing_mass(const uint16_t* x, int T, const float* wr, const float* bias,
                               const uint8_t* keep_mask, int H, int m, int k, float* mass_softmax,
                               float* mass_topk, void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  char* p = static_cast<char*>(workspace);
  const size_t P = (size_t)T * k;
  float* part = reinterpret_cast<float*>(p);
  p += route_workspace_bytes(T, H, m, k);
  int* ids = reinterpret_cast<int*>(p);
  p += align_up(P * 4, 256);
  float* w = reinterpret_cast<float*>(p);
  p += align_up(P * 4, 256);
  int* perm = reinterpret_cast<int*>(p);
  p += align_up(P * 4, 256);
  int* counts = reinterpret_cast<int*>(p);
  p += align_up((size_t)(m + 1) * 4, 256);
  int* offsets = reinterpret_cast<int*>(p);
  p += align_up((size_t)(m + 1) * 4, 256);
  int* active = reinterpret_cast<int*>(p);
  p += align_up((size_t)(m + 1) * 4, 256);
  int* n_active = reinterpret_cast<int*>(p);
  p += 256;
  float* zmax = reinterpret_cast<float*>(p);
  p += align_up((size_t)T * 4, 256);
  float* denom = reinterpret_cast<float*>(p);
  hipError_t err = launch_route_dispatch(x, T, wr, bias, keep_mask, H, m, k, ids, w, nullptr,
                                         counts, offsets, perm, active, n_active, part, stream);
  if (err != hipSuccess) return err;
  const int KS = logits_split(T, H, m).ks;
  mass_token_stats_kernel<<<(T + 3) / 4, 256, 0, stream>>>(part, KS, bias, keep_mask, T, m, zmax,
                                                           denom);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  mass_accumulate_kernel<<<(m + 255) / 256, 256, 0, stream>>>(
      part, KS, bias, keep_mask, T, m, zmax, denom, w, counts, offsets, perm, n_active,
      (int)P, mass_softmax, mass_topk);
  return hipGetLastError();
}

// Logit partials, then the chunked dispatch's scratch (used once the
// partials have been read).
static size_t part_bytes(int T, int H, int m) {
  return align_up((size_t)logits_split(T, H, m).ks * T * m * sizeof(float), 256);
}

size_t route_workspace_bytes(int T, int H, int m, int k) {
  if (T <= 0) return 0;
  return part_bytes(T, H, m) + dispatch_workspace_bytes(T * k, m);
}

size_t route_shared_workspace_bytes(int T, int H, int m, int k, int S, int R) {
  if (T <= 0) return 0;
  return part_bytes(T, H, m + 1) + dispatch_workspace_bytes(T * (k + S), m + R * S);
}

namespace {

// Logits of the c.ld router rows, then the top-k over the first c.m.
hipError_t route_cols(const uint16_t* x, int T, const float* wr, const float* bias,
                      const uint8_t* keep_mask, int H, const Cols& c, int* topk_ids,
                      float* topk_w, float* gap, void* workspace, hipStream_t stream) {
  float* part = static_cast<float*>(workspace);
  const LogitsSplit sp = logits_split(T, H, c.ld);
  hipError_t err = launch_logits(x, T, wr, H, c.ld, part, sp, stream);
  if (err != hipSuccess) return err;
  launch_topk(part, sp.ks, bias, keep_mask, T, c, topk_ids, topk_w, gap, stream);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const uint16_t* x, int T, const float* wr, const float* bias,
                        const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                        float* topk_w, float* gap, void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  return route_cols(x, T, wr, bias, keep_mask, H, Cols{m, m, k, 0, 1}, topk_ids, topk_w, gap,
                    workspace, stream);
}

hipError_t launch_route_select(const uint16_t* x, int T, const float* wr, const float* bias,
                               const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                               float* topk_w, float* gap, void* workspace, hipStream_t stream,
                               int n_shared, int n_groups) {
  if (T == 0) return hipSuccess;
  const Cols c{m, n_shared > 0 ? m + 1 : m, k, n_shared, n_shared > 0 ? n_groups : 1};
  return route_cols(x, T, wr, bias, keep_mask, H, c, topk_ids, topk_w, gap, workspace, stream);
}

bool fused_route_dispatch_supported(int T, int m, int k, int S, int R) {
  return T > 0 && T <= kFusedMaxTokens && m + R * S <= kFusedMaxPool && k + S <= kFusedMaxK;
}

hipError_t launch_route_dispatch(const uint16_t* x, int T, const float* wr, const float* bias,
                                 const uint8_t* keep_mask, int H, int m, int k, int* topk_ids,
                                 float* topk_w, float* gap, int* counts, int* offsets, int* perm,
                                 int* active, int* n_active, void* workspace, hipStream_t stream,
                                 int n_shared, int n_groups) {
  const Cols c{m, n_shared > 0 ? m + 1 : m, k, n_shared, n_shared > 0 ? n_groups : 1};
  const int kout = k + n_shared, m_plan = c.plan_m();
  if (!fused_route_dispatch_supported(T, m, k, n_shared, c.R)) {
    if (T > 0) {
      hipError_t err = route_cols(x, T, wr, bias, keep_mask, H, c, topk_ids, topk_w, gap,
                                  workspace, stream);
      if (err != hipSuccess) return err;
    }
    return launch_dispatch(topk_ids, T * kout, m_plan, counts, offsets, perm, active, n_active,
                           stream, static_cast<char*>(workspace) + part_bytes(T, H, c.ld));
  }
  float* part = static_cast<float*>(workspace);
  const LogitsSplit sp = logits_split(T, H, c.ld);
  hipError_t err = launch_logits(x, T, wr, H, c.ld, part, sp, stream);
  if (err != hipSuccess) return err;
  const int kpl = (m + 15) / 16;
  if (T <= kWaveFusedTokens) {
#define SW_WF(KPL)                                                                             \
  route_select_dispatch_wave_kernel<KPL><<<1, 64, 0, stream>>>(part, sp.ks, bias, keep_mask, T, c, \
                                                               topk_ids, topk_w, gap, counts,      \
                                                               offsets, perm, active, n_active)
    if (kpl <= 4)
      SW_WF(4);
    else if (kpl <= 8)
      SW_WF(8);
    else
      SW_WF(16);
#undef SW_WF
    return hipGetLastError();
  }
#define SW_FD(KPL)                                                                             \
  route_select_dispatch_kernel<KPL><<<1, kFusedThreads, 0, stream>>>(                             \
      part, sp.ks, bias, keep_mask, T, c, topk_ids, topk_w, gap, counts, offsets, perm, active,   \
      n_active)
  if (kpl <= 4)
    SW_FD(4);
  else if (kpl <= 8)
    SW_FD(8);
  else
    SW_FD(16);
#undef SW_FD
  return hipGetLastError();
}

}  // namespace sw
