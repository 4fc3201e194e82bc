// Split-K expert kernels for calls with few tiles on gfx950: a decode batch
// of one or two tokens (Section 2.1, Eq. 1: a batch of B tokens reads about
// B * k distinct experts), or the single always-on shared expert (Section
// 3.3).
//
// With far fewer 16-row tiles than the chip has waves, giving each wave
// whole tiles leaves most waves idle and the step waits on one long stream
// per wave.  Here the contraction of a tile is split over S waves of a
// block (S a power of two up to the block's 8 or 16 waves, chosen so that
// every wave still reads a few 1 KiB K steps): wave w of the block works on
// tile slot w / S and K slice w % S.  A wave streams its slice of the tile's weights with all of
// its loads in flight at once and multiplies it with the matching slice of
// the tokens' activations, read straight from L2 (no LDS staging: every
// activation element is used by one wave only).  The S partial tiles meet
// in LDS, the slot's first wave adds them in slice order and runs the usual
// epilogue (SwiGLU into h for gate/up; y rows for down).
//
// A pass covers 16 * NB tokens of a tile's expert; the host picks NB from
// the batch size (an expert receives at most one pair per token), and the
// pass count of a block is the largest of its tiles', the same in every
// wave, so the barriers stay block-uniform.
#include <climits>

#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

// Block shape per token-block count: passes of 64 tokens (NB = 4) hold
// four times the activation fragments per K step, so they take 16 waves of
// 4 K steps per round; narrower passes take 8 waves of 8 steps.
template <int NB>
constexpr int waves_of() { return NB == 4 ? 16 : 8; }
template <int NB>
constexpr int steps_of() { return NB == 4 ? 4 : 8; }
// Whether a gate/up block loads its next group's first weights during the
// current group's last pass.  64-token passes leave no registers for it.
// The down kernel does not: the registers it takes cost a resident block per
// compute unit, which is worth more there.
template <int NB>
constexpr bool gate_up_prefetches() { return NB < 4; }

// The expert of tile `tile` as the active list holds it, read without
// waiting for n_active (any entry below m is safe to read): the first
// weight loads of a group go out before the plan is validated.  -1 when the
// slot is outside the list's storage.
__device__ __forceinline__ int speculative_expert(int tile, int tpe, const int* active, int m) {
  const int a = tile / tpe;
  return a < m ? active[a] : -1;
}

// Token count and first dispatch slot of tile `tile` with expert e; an
// out-of-range tile, a bad expert id or a pair range outside [0, n_pairs)
// has no tokens.
__device__ __forceinline__ void tile_tokens(int tile, int n_tiles, int e, const int* counts,
                                            const int* offsets, int m, int n_pairs, int* cnt,
                                            int* base) {
  *cnt = 0;
  *base = 0;
  if (tile >= n_tiles || e < 0 || e >= m) return;
  const int c = counts[e], b = offsets[e];
  if (c <= 0 || b < 0 || c > n_pairs - b) return;
  *cnt = c;
  *base = b;
}

// Largest token count over the block's tile slots: the block's pass count
// follows from it, identically in every wave.
__device__ __forceinline__ int group_max_count(int grp, int tps, int n_tiles, int tpe,
                                               const int* active, const int* counts,
                                               const int* offsets, int m, int n_pairs) {
  int mx = 0;
  for (int s = 0; s < tps; ++s) {
    const int tile = grp * tps + s;
    if (tile >= n_tiles) break;
    int c, b;
    tile_tokens(tile, n_tiles, active[tile / tpe], counts, offsets, m, n_pairs, &c, &b);
    mx = max(mx, c);
  }
  return mx;
}

// ---------------------------------------------------------------------------
// gate/up + SwiGLU

template <int NB, bool kTiled>
__global__ __launch_bounds__(64 * waves_of<NB>(), 1) void gate_up_skinny_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w13,
    const int* __restrict__ counts, const int* __restrict__ offsets,
    const int* __restrict__ perm, const int* __restrict__ active,
    const int* __restrict__ n_active_p, uint16_t* __restrict__ h_hi,
    uint16_t* __restrict__ h_lo, int H, int I, int m, int k, int n_pairs, int S, int identity) {
  constexpr int kNT = 16 * NB;
  constexpr int kWv = waves_of<NB>(), kKS = steps_of<NB>();
  constexpr bool kPrefetch = gate_up_prefetches<NB>();
  __shared__ f32x4 red[kWv][NB][kWave];
  __shared__ int pid_s[kWv][kNT];  // per tile slot: the pass's pair ids
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, kg = lane >> 4;
  const int tps = kWv / S, slot = wave / S, slice = wave - slot * S;
  const int tpe = I / 8, nsteps = H / 32;
  const int s_lo = (slice * nsteps) / S, s_hi = ((slice + 1) * nsteps) / S;
  const auto xr = make_rsrc(x, 2u * (uint32_t)(n_pairs / k) * (uint32_t)H);
  const int n_act = *n_active_p;
  bool first = true;

  struct Src {
    __amdgpu_buffer_rsrc_t w;
    uint32_t row;
    int e, ib;
  };
  // this wave's weights in group g (the expert read without waiting for
  // n_active); tiles from `limit` on (past the plan's tiles, once it is
  // known) get the empty resource and load nothing
  auto src_of = [&](int g, int limit) {
    Src c;
    const int tile = g * tps + slot;
    const int e = tile < limit ? speculative_expert(tile, tpe, active, m) : -1;
    const bool e_ok = e >= 0 && e < m;
    c.e = e;
    c.ib = tile - (tile / tpe) * tpe;
    c.w = make_rsrc(w13 + (size_t)(e_ok ? e : 0) * 2 * I * H, e_ok ? 4u * (uint32_t)I * H : 0u);
    if (kTiled) {
      c.row = (uint32_t)c.ib * 32u * H + (uint32_t)lane * 16u;
    } else {
      const int wrow = r < 8 ? c.ib * 8 + r : I + c.ib * 8 + (r - 8);
      c.row = (uint32_t)wrow * H * 2u + kg * 16u;
    }
    return c;
  };
  constexpr uint32_t stride = kTiled ? 1024u : 64u;
  auto issue = [&](const Src& c, u32x4 (&A)[kKS], int sb) {
#pragma unroll
    for (int j = 0; j < kKS; ++j) {
      const uint32_t off = sb + j < s_hi ? c.row + (uint32_t)(sb + j) * stride : kOutOfRange;
      A[j] = kTiled ? buf_ld128_stream(c.w, off) : buf_ld128(c.w, off);
    }
  };
  // a block walks several groups: the next group's first round of weights
  // goes out as soon as the current group's last MFMAs have read theirs
  u32x4 A[kKS];
  Src cur = src_of(blockIdx.x, INT_MAX);
  issue(cur, A, s_lo);

  for (int grp = blockIdx.x;; grp += gridDim.x) {
    const int tile = grp * tps + slot;
    const int e = cur.e, ib = cur.ib;
    if (n_act <= 0 || n_act > m) return;  // an invalid plan: no work
    const int n_tiles = n_act * tpe;
    if (grp * tps >= n_tiles) break;
    int cnt, base;
    tile_tokens(tile, n_tiles, e, counts, offsets, m, n_pairs, &cnt, &base);
    const int maxcnt =
        tps == 1 ? cnt : group_max_count(grp, tps, n_tiles, tpe, active, counts, offsets, m, n_pairs);
    const uint32_t hbytes = 2u * (uint32_t)cnt * (uint32_t)I;
    const auto hh = make_rsrc(h_hi + (size_t)base * I, hbytes);
    const auto hl = make_rsrc(h_lo + (size_t)base * I, hbytes);
    const bool more = (grp + (int)gridDim.x) * tps < n_tiles;  // a next group
    Src nxt;
    if constexpr (kPrefetch) nxt = src_of(grp + gridDim.x, n_tiles);
    bool prefetched = false;

    // at least one pass: every path then consumes the group's first weight
    // loads (the empty group of an invalid plan stores nothing)
    int p0 = 0;
    do {
      if (!first) __syncthreads();  // the previous pass's readers of red and pid_s are done
      first = false;
      const int nbn = p0 < cnt ? (min(kNT, cnt - p0) + 15) >> 4 : 0;
      // the pass's pair ids: one load per lane by the slot's first wave, into
      // LDS (an identity plan, the shared expert's, needs none)
      if (!identity) {
        if (slice == 0 && lane < kNT) {
          const int sl = p0 + lane;
          const int p = sl < cnt ? perm[base + sl] : -1;
          pid_s[slot][lane] = (p >= 0 && p < n_pairs) ? p : -1;
        }
        __syncthreads();
      }
      // activation row of column r of each 16-token block: x[pair / k]
      uint32_t xrow[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int sl = p0 + nb * 16 + r;
        const int p = identity ? base + sl : pid_s[slot][nb * 16 + r];
        xrow[nb] = (nb < nbn && sl < cnt && p >= 0 && p < n_pairs)
                       ? (uint32_t)(p / k) * H * 2u + kg * 16u : kOutOfRange;
      }
      f32x4 acc[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      int sb = s_lo;  // every slice has at least one K step
      do {
        if (sb != s_lo || p0 != 0) issue(cur, A, sb);
        u32x4 B[NB][kKS];
#pragma unroll
        for (int j = 0; j < kKS; ++j)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            B[nb][j] = buf_ld128(xr, (sb + j < s_hi && xrow[nb] != kOutOfRange)
                                         ? xrow[nb] + (uint32_t)(sb + j) * 64u : kOutOfRange);
        // keep every load of the round ahead of the first MFMA
        __builtin_amdgcn_sched_barrier(0);
        // (columns past the pass's tokens multiply zeros and are not stored)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int j = 0; j < kKS; ++j) acc[nb] = mfma_16x16x32(A[j], B[nb][j], acc[nb]);
      } while ((sb += kKS) < s_hi);
      if (kPrefetch && more && p0 + kNT >= maxcnt) {  // the group's last pass
        issue(nxt, A, s_lo);
        prefetched = true;
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) red[wave][nb][lane] = acc[nb];
      __syncthreads();
      // token block nb of the slot is finished by its wave nb % S (slice order)
      if (slice < NB && nbn > 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if (nb < nbn && nb % S == slice) {
            const int w0 = slot * S;
            f32x4 g4 = red[w0][nb][lane];
            for (int q = 1; q < S; ++q) g4 += red[w0 + q][nb][lane];
            f32x4 u4;
#pragma unroll
            for (int i = 0; i < 4; ++i) u4[i] = __shfl_xor(g4[i], 32);
            float hv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) hv[i] = swiglu(g4[i], u4[i]);
            u32x2 hw, lw;
            split_bf16x4(hv, hw, lw);
            const int sl = p0 + nb * 16 + r;
            uint32_t off = kOutOfRange;
            if (lane < 32 && sl < cnt) off = ((uint32_t)sl * I + (uint32_t)(ib * 8 + kg * 4)) * 2u;
            __builtin_amdgcn_raw_buffer_store_b64(hw, hh, off, 0, 0);
            __builtin_amdgcn_raw_buffer_store_b64(lw, hl, off, 0, 0);
          }
        }
      }
    } while ((p0 += kNT) < maxcnt);
    if (!more) break;
    if constexpr (kPrefetch) {
      if (!prefetched) issue(nxt, A, s_lo);  // a group without passes
      cur = nxt;
    } else {
      cur = src_of(grp + gridDim.x, n_tiles);
      issue(cur, A, s_lo);
    }
  }
}

// ---------------------------------------------------------------------------
// down projection

template <int NB, bool kTiled>
__global__ __launch_bounds__(64 * waves_of<NB>(), 1) void down_skinny_kernel(
    const uint16_t* __restrict__ h_hi, const uint16_t* __restrict__ h_lo,
    const uint16_t* __restrict__ w2, const int* __restrict__ counts,
    const int* __restrict__ offsets, const int* __restrict__ perm,
    const int* __restrict__ active, const int* __restrict__ n_active_p, float* __restrict__ y,
    int H, int I, int m, int n_pairs, int S, int identity) {
  constexpr int kNT = 16 * NB;
  constexpr int kWv = waves_of<NB>();
  constexpr int kHS = steps_of<NB>() / 2;  // two MFMAs (hi, lo) per weight load
  __shared__ f32x4 red[kWv][NB][kWave];
  __shared__ int pid_s[kWv][kNT];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, kg = lane >> 4;
  const int tps = kWv / S, slot = wave / S, slice = wave - slot * S;
  const int tpe = H / 16, nsteps = I / 32;
  const int s_lo = (slice * nsteps) / S, s_hi = ((slice + 1) * nsteps) / S;
  const uint32_t hbytes_all = 2u * (uint32_t)n_pairs * (uint32_t)I;
  const auto hhr = make_rsrc(h_hi, hbytes_all);
  const auto hlr = make_rsrc(h_lo, hbytes_all);
  const auto yr = make_rsrc(y, 4u * (uint32_t)n_pairs * (uint32_t)H);
  const int n_act = *n_active_p;
  bool first = true;

  struct Src {
    __amdgpu_buffer_rsrc_t w;
    uint32_t row;
    int e, ib;
  };
  // this wave's weights in group g (the expert read without waiting for
  // n_active); tiles from `limit` on (past the plan's tiles, once it is
  // known) get the empty resource and load nothing
  auto src_of = [&](int g, int limit) {
    Src c;
    const int tile = g * tps + slot;
    const int e = tile < limit ? speculative_expert(tile, tpe, active, m) : -1;
    const bool e_ok = e >= 0 && e < m;
    c.e = e;
    c.ib = tile - (tile / tpe) * tpe;
    c.w = make_rsrc(w2 + (size_t)(e_ok ? e : 0) * H * I, e_ok ? 2u * (uint32_t)H * I : 0u);
    c.row = kTiled ? (uint32_t)c.ib * 32u * I + (uint32_t)lane * 16u
                   : (uint32_t)(c.ib * 16 + r) * I * 2u + kg * 16u;
    return c;
  };
  constexpr uint32_t stride = kTiled ? 1024u : 64u;
  auto issue = [&](const Src& c, u32x4 (&A)[kHS], int sb) {
#pragma unroll
    for (int j = 0; j < kHS; ++j) {
      const uint32_t off = sb + j < s_hi ? c.row + (uint32_t)(sb + j) * stride : kOutOfRange;
      A[j] = kTiled ? buf_ld128_stream(c.w, off) : buf_ld128(c.w, off);
    }
  };
  u32x4 A[kHS];
  Src cur = src_of(blockIdx.x, INT_MAX);
  issue(cur, A, s_lo);

  for (int grp = blockIdx.x;; grp += gridDim.x) {
    const int tile = grp * tps + slot;
    const int e = cur.e, ib = cur.ib;
    if (n_act <= 0 || n_act > m) return;
    const int n_tiles = n_act * tpe;
    if (grp * tps >= n_tiles) break;
    int cnt, base;
    tile_tokens(tile, n_tiles, e, counts, offsets, m, n_pairs, &cnt, &base);
    const int maxcnt =
        tps == 1 ? cnt : group_max_count(grp, tps, n_tiles, tpe, active, counts, offsets, m, n_pairs);

    // at least one pass: every path then consumes the group's first weight
    // loads (the empty group of an invalid plan stores nothing)
    int p0 = 0;
    do {
      if (!first) __syncthreads();
      first = false;
      const int nbn = p0 < cnt ? (min(kNT, cnt - p0) + 15) >> 4 : 0;
      // h rows of the pass are the dispatch slots base + p0 + nb * 16 + r;
      // the pair ids (y rows, for the epilogue) go to LDS as in gate/up
      if (!identity && slice == 0 && lane < kNT) {
        const int sl = p0 + lane;
        const int p = sl < cnt ? perm[base + sl] : -1;
        pid_s[slot][lane] = (p >= 0 && p < n_pairs) ? p : -1;
      }
      uint32_t hrow[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int sl = p0 + nb * 16 + r;
        const bool in = nb < nbn && sl < cnt;
        hrow[nb] = in ? (uint32_t)(base + sl) * I * 2u + kg * 16u : kOutOfRange;
      }
      f32x4 acc[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      int sb = s_lo;  // every slice has at least one K step
      do {
        if (sb != s_lo || p0 != 0) issue(cur, A, sb);
        u32x4 BH[NB][kHS], BL[NB][kHS];
#pragma unroll
        for (int j = 0; j < kHS; ++j)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const uint32_t ho = (sb + j < s_hi && hrow[nb] != kOutOfRange)
                                    ? hrow[nb] + (uint32_t)(sb + j) * 64u : kOutOfRange;
            BH[nb][j] = buf_ld128(hhr, ho);
            BL[nb][j] = buf_ld128(hlr, ho);
          }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int j = 0; j < kHS; ++j) {
              acc[nb] = mfma_16x16x32(A[j], BH[nb][j], acc[nb]);
              acc[nb] = mfma_16x16x32(A[j], BL[nb][j], acc[nb]);
            }
      } while ((sb += kHS) < s_hi);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) red[wave][nb][lane] = acc[nb];
      __syncthreads();
      if (slice < NB && nbn > 0) {
        const int o = ib * 16 + kg * 4;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if (nb < nbn && nb % S == slice) {
            const int w0 = slot * S;
            f32x4 c = red[w0][nb][lane];
            for (int q = 1; q < S; ++q) c += red[w0 + q][nb][lane];
            const int sl = p0 + nb * 16 + r;
            const int p = sl >= cnt ? -1 : identity ? base + sl : pid_s[slot][nb * 16 + r];
            uint32_t off = kOutOfRange;
            if (p >= 0 && p < n_pairs) off = ((uint32_t)p * H + (uint32_t)o) * 4u;
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, c), yr, off, 0, 0);
          }
        }
      }
    } while ((p0 += kNT) < maxcnt);
    if ((grp + (int)gridDim.x) * tps >= n_tiles) break;
    cur = src_of(grp + gridDim.x, n_tiles);
    issue(cur, A, s_lo);
  }
}

// K split of a block of wv waves: the largest S in {wv, wv/2, ..., 1} that
// leaves every wave at least min_steps K steps.
int split_factor(int nsteps, int wv, int min_steps) {
  int s = wv;
  while (s > 1 && nsteps / s < min_steps) s >>= 1;
  return s;
}

// Token blocks per pass: an expert receives at most one pair per token.
int token_blocks(int T) { return T <= 16 ? 1 : T <= 32 ? 2 : 4; }

// Upper bound of the active experts of a call.
int64_t max_active(int T, int m, int k) { return std::min<int64_t>(m, (int64_t)T * k); }

// Blocks of a launch.  Kernels that prefetch get no more than fit on the
// chip at once: a block with a second group loads that group's first
// weights during its current group's last pass, where a fresh block would
// wait for a compute unit to free up.  The others get a block per group.
template <bool kPrefetch, auto kKernel>
int skinny_grid(int64_t tiles, int wv, int S) {
  const int64_t groups = std::max<int64_t>(1, (tiles + wv / S - 1) / (wv / S));
  if (!kPrefetch) return (int)std::min<int64_t>(groups, 4096);
  static const int per_cu = [&] {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kKernel, 64 * wv, 0) != hipSuccess)
      n = 1;
    return std::max(n, 1);
  }();
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 256;
  const int64_t cap = (int64_t)cus * per_cu;
  return (int)std::min(groups, cap);
}

constexpr int kMaxSkinnyTiles = 2048;

}  // namespace

bool skinny_gate_up_supported(int T, int H, int I, int m, int k) {
  return T >= 1 && H >= 1024 && H % 32 == 0 && I % 8 == 0 &&
         max_active(T, m, k) * (I / 8) <= kMaxSkinnyTiles &&
         2 * (int64_t)T * H < ((int64_t)1 << 31) && 2 * (int64_t)T * k * I < ((int64_t)1 << 31);
}

bool skinny_down_supported(int T, int H, int I, int m, int k) {
  return T >= 1 && I >= 256 && I % 32 == 0 && H % 16 == 0 &&
         max_active(T, m, k) * (H / 16) <= kMaxSkinnyTiles &&
         4 * (int64_t)T * k * H < ((int64_t)1 << 31) && 2 * (int64_t)T * k * I < ((int64_t)1 << 31);
}

template <int NB>
static void gate_up_skinny(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                           const int* counts, const int* offsets, const int* perm,
                           const int* active, const int* n_active, int H, int I, int m, int k,
                           uint16_t* h_hi, uint16_t* h_lo, bool identity, hipStream_t stream) {
  constexpr int wv = waves_of<NB>();
  const int S = split_factor(H / 32, wv, NB == 4 ? 4 : 6);
  const int64_t tiles = max_active(T, m, k) * (I / 8);
  constexpr bool kPf = gate_up_prefetches<NB>();
  if (tiled) {
    constexpr auto kern = gate_up_skinny_kernel<NB, true>;
    kern<<<skinny_grid<kPf, kern>(tiles, wv, S), 64 * wv, 0, stream>>>(
        x, w13, counts, offsets, perm, active, n_active, h_hi, h_lo, H, I, m, k, T * k, S,
        identity ? 1 : 0);
  } else {
    constexpr auto kern = gate_up_skinny_kernel<NB, false>;
    kern<<<skinny_grid<kPf, kern>(tiles, wv, S), 64 * wv, 0, stream>>>(
        x, w13, counts, offsets, perm, active, n_active, h_hi, h_lo, H, I, m, k, T * k, S,
        identity ? 1 : 0);
  }
}

hipError_t launch_gate_up_skinny(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                 const int* counts, const int* offsets, const int* perm,
                                 const int* active, const int* n_active, int H, int I, int m,
                                 int k, uint16_t* h_hi, uint16_t* h_lo, bool identity,
                                 hipStream_t stream) {
  switch (token_blocks(T)) {
    case 1:
      gate_up_skinny<1>(x, T, w13, tiled, counts, offsets, perm, active, n_active, H, I, m, k,
                        h_hi, h_lo, identity, stream);
      break;
    case 2:
      gate_up_skinny<2>(x, T, w13, tiled, counts, offsets, perm, active, n_active, H, I, m, k,
                        h_hi, h_lo, identity, stream);
      break;
    default:
      gate_up_skinny<4>(x, T, w13, tiled, counts, offsets, perm, active, n_active, H, I, m, k,
                        h_hi, h_lo, identity, stream);
  }
  return hipGetLastError();
}

template <int NB>
static void down_skinny(int T, const uint16_t* w2, bool tiled, const int* counts,
                        const int* offsets, const int* perm, const int* active,
                        const int* n_active, int H, int I, int m, int k, const uint16_t* h_hi,
                        const uint16_t* h_lo, float* y, bool identity, hipStream_t stream) {
  constexpr int wv = waves_of<NB>();
  const int S = split_factor(I / 32, wv, NB == 4 ? 2 : 6);
  const int64_t tiles = max_active(T, m, k) * (H / 16);
  if (tiled) {
    constexpr auto kern = down_skinny_kernel<NB, true>;
    kern<<<skinny_grid<false, kern>(tiles, wv, S), 64 * wv, 0, stream>>>(
        h_hi, h_lo, w2, counts, offsets, perm, active, n_active, y, H, I, m, T * k, S,
        identity ? 1 : 0);
  } else {
    constexpr auto kern = down_skinny_kernel<NB, false>;
    kern<<<skinny_grid<false, kern>(tiles, wv, S), 64 * wv, 0, stream>>>(
        h_hi, h_lo, w2, counts, offsets, perm, active, n_active, y, H, I, m, T * k, S,
        identity ? 1 : 0);
  }
}

hipError_t launch_down_skinny(int T, const uint16_t* w2, bool tiled, const int* counts,
                              const int* offsets, const int* perm, const int* active,
                              const int* n_active, int H, int I, int m, int k,
                              const uint16_t* h_hi, const uint16_t* h_lo, float* y,
                              bool identity, hipStream_t stream) {
  switch (token_blocks(T)) {
    case 1:
      down_skinny<1>(T, w2, tiled, counts, offsets, perm, active, n_active, H, I, m, k, h_hi,
                     h_lo, y, identity, stream);
      break;
    case 2:
      down_skinny<2>(T, w2, tiled, counts, offsets, perm, active, n_active, H, I, m, k, h_hi,
                     h_lo, y, identity, stream);
      break;
    default:
      down_skinny<4>(T, w2, tiled, counts, offsets, perm, active, n_active, H, I, m, k, h_hi,
                     h_lo, y, identity, stream);
  }
  return hipGetLastError();
}

}  // namespace sw
