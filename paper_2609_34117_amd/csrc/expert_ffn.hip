// Expert FFNs of the MoE layer on gfx950 (Section 2.1: each step reads the
// weights of every distinct expert selected across the batch).
//
// Every active expert's bf16 weights are streamed from HBM exactly once per
// call with 128-bit loads straight into matrix-core operand registers (plain
// loads: measured faster than non-temporal ones for this 16-row access
// pattern on MI355X); the
// expert's tokens form the narrow side of a 16x16x32 bf16 MFMA (padded to
// 16 columns), so decode's handful of tokens per expert costs almost no
// issue time and there is no cross-lane reduction over the hidden size.
// All operand loads are branch-free buffer loads: lanes with nothing to read
// use an out-of-range offset and receive zeros, so a wave issues its whole
// tile of loads back to back before the first MFMA waits on them.
//
//   gate_up: block = 4 waves, tile = (expert, 8 intermediate indices).  The
//            16 A rows are the 8 gate rows and the 8 matching up rows; the
//            waves split H four ways and add their partial tiles in LDS.
//            Epilogue: h = silu(g) * u, stored as a bf16 hi/lo pair
//            (h ~= hi + lo to ~16 mantissa bits) in dispatch-slot order.
//   down:    block = 4 waves, tile = (expert, 16*MB output rows); the waves
//            split I four ways; B = h hi and lo (two MFMAs per step).
//   combine: out[t] = sum_j w[t, j] y[t*k + j] in slot order.
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kNbGateUp = 4;  // 16-token column blocks per pass of gate_up (64 tokens)
constexpr int kNbDown = 2;    // ... of down (32 tokens)

struct ForwardWs {
  uint16_t* h_hi;
  uint16_t* h_lo;
  float* y;
};

__host__ __device__ inline size_t h_bytes(int n_pairs, int I) {
  return align_up((size_t)n_pairs * I * sizeof(uint16_t), 256);
}

__host__ __device__ inline size_t y_bytes(int n_pairs, int H) {
  return align_up((size_t)n_pairs * H * sizeof(float), 256);
}

__host__ __device__ inline ForwardWs carve(void* ws, int n_pairs, int H, int I) {
  char* p = static_cast<char*>(ws);
  ForwardWs w;
  w.h_hi = reinterpret_cast<uint16_t*>(p);
  w.h_lo = reinterpret_cast<uint16_t*>(p + h_bytes(n_pairs, I));
  w.y = reinterpret_cast<float*>(p + 2 * h_bytes(n_pairs, I));
  return w;
}

// Resolves a streaming tile to (expert slot, expert, count, first slot);
// false if the tile is surplus or the dispatch plan is inconsistent.
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

// K range of wave w when `nsteps` 32-wide K steps are split four ways.
__device__ __forceinline__ void wave_ksteps(int nsteps, int wave, int* lo, int* hi) {
  *lo = (wave * nsteps) >> 2;
  *hi = ((wave + 1) * nsteps) >> 2;
}

template <int KS>
__global__ __launch_bounds__(256) void gate_up_generic_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w13,
    const int* __restrict__ counts, const int* __restrict__ offsets,
    const int* __restrict__ perm, const int* __restrict__ active,
    const int* __restrict__ n_active_p, uint16_t* __restrict__ h_hi,
    uint16_t* __restrict__ h_lo, int H, int I, int m, int k, int n_pairs, int T) {
  __shared__ f32x4 part[4][kNbGateUp][kWave];
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
  const auto w_rsrc = make_rsrc(w13 + (size_t)e * 2 * I * H, 4u * (uint32_t)I * (uint32_t)H);
  const auto x_rsrc = make_rsrc(x, 2u * (uint32_t)T * (uint32_t)H);
  const auto p_rsrc = make_rsrc(perm + base, 4u * (uint32_t)cnt);
  const uint32_t a_row = (uint32_t)wrow * H * 2u;
  int s_lo, s_hi;
  wave_ksteps((H + 31) >> 5, wave, &s_lo, &s_hi);
  const int n_w = s_hi - s_lo;
  const int nchunks = (n_w + KS - 1) / KS;

  u32x4 A[KS];
  for (int t0 = 0; t0 < cnt; t0 += 16 * kNbGateUp) {
    const int nbn = (min(16 * kNbGateUp, cnt - t0) + 15) >> 4;
    // byte offset of each N-block's token row for this lane (out of range
    // for slots past the expert's count)
    uint32_t pv[kNbGateUp], xoff[kNbGateUp];
#pragma unroll
    for (int nb = 0; nb < kNbGateUp; ++nb) pv[nb] = buf_ld32(p_rsrc, (uint32_t)(t0 + nb * 16 + r) * 4u);
#pragma unroll
    for (int nb = 0; nb < kNbGateUp; ++nb) {
      const int slot = t0 + nb * 16 + r;
      const bool ok = slot < cnt && pv[nb] < (uint32_t)n_pairs;
      const uint32_t t = (ok ? pv[nb] : 0u) / (uint32_t)k;
      xoff[nb] = ok ? t * H * 2u : kOutOfRange;
    }
    f32x4 acc[kNbGateUp];
#pragma unroll
    for (int nb = 0; nb < kNbGateUp; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int ch = 0; ch < nchunks; ++ch) {
      const int sb = s_lo + ch * KS;
      if (t0 == 0 || nchunks > 1) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const int col = (sb + s) * 32 + kg * 8;
          const bool ok = sb + s < s_hi && col < H;
          A[s] = buf_ld128(w_rsrc, ok ? a_row + (uint32_t)col * 2u : kOutOfRange);
        }
      }
#pragma unroll
      for (int nb = 0; nb < kNbGateUp; ++nb) {
        if (nb < nbn) {
          u32x4 B[KS];
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            const int col = (sb + s) * 32 + kg * 8;
            const bool ok = sb + s < s_hi && col < H && xoff[nb] != kOutOfRange;
            B[s] = buf_ld128(x_rsrc, ok ? xoff[nb] + (uint32_t)col * 2u : kOutOfRange);
          }
#pragma unroll
          for (int s = 0; s < KS; ++s) acc[nb] = mfma_16x16x32(A[s], B[s], acc[nb]);
        }
      }
    }

#pragma unroll
    for (int nb = 0; nb < kNbGateUp; ++nb)
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
        float hv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) hv[q] = swiglu(c[q], u[q]);
        u32x2 hw, lw;
        split_bf16x4(hv, hw, lw);
        const size_t off = (size_t)(base + slot) * I + ib * 8 + kg * 4;
        *reinterpret_cast<uint2*>(h_hi + off) = make_uint2(hw[0], hw[1]);
        *reinterpret_cast<uint2*>(h_lo + off) = make_uint2(lw[0], lw[1]);
      }
    }
    __syncthreads();
  }
}

template <int KS, int MB>
__global__ __launch_bounds__(256) void down_generic_kernel(
    const uint16_t* __restrict__ h_hi, const uint16_t* __restrict__ h_lo,
    const uint16_t* __restrict__ w2, const int* __restrict__ counts,
    const int* __restrict__ offsets, const int* __restrict__ perm,
    const int* __restrict__ active, const int* __restrict__ n_active_p, float* __restrict__ y,
    int H, int I, int m, int n_pairs) {
  __shared__ f32x4 part[4][MB * kNbDown][kWave];
  const int n_act = *n_active_p;
  if (n_act <= 0 || n_act > m) return;
  constexpr int kRows = 16 * MB;
  const int tpe = (H + kRows - 1) / kRows;
  int a, e, cnt, base;
  const int tile = xcd_tile(blockIdx.x, n_act * tpe);
  if (!tile_expert(tile, tpe, active, counts, offsets, m, n_pairs, &a, &e, &cnt, &base)) return;
  const int o0 = (tile - a * tpe) * kRows;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, kg = lane >> 4;
  const auto w_rsrc = make_rsrc(w2 + (size_t)e * H * I, 2u * (uint32_t)H * (uint32_t)I);
  const auto hh_rsrc = make_rsrc(h_hi + (size_t)base * I, 2u * (uint32_t)cnt * (uint32_t)I);
  const auto hl_rsrc = make_rsrc(h_lo + (size_t)base * I, 2u * (uint32_t)cnt * (uint32_t)I);
  int s_lo, s_hi;
  wave_ksteps((I + 31) >> 5, wave, &s_lo, &s_hi);
  const int n_w = s_hi - s_lo;
  const int nchunks = (n_w + KS - 1) / KS;

  u32x4 A[MB][KS];
  for (int t0 = 0; t0 < cnt; t0 += 16 * kNbDown) {
    const int nbn = (min(16 * kNbDown, cnt - t0) + 15) >> 4;
    f32x4 acc[MB][kNbDown];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < kNbDown; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int ch = 0; ch < nchunks; ++ch) {
      const int sb = s_lo + ch * KS;
      if (t0 == 0 || nchunks > 1) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int row = o0 + mb * 16 + r;
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            const int col = (sb + s) * 32 + kg * 8;
            const bool ok = row < H && sb + s < s_hi && col < I;
            A[mb][s] = buf_ld128(
                w_rsrc, ok ? ((uint32_t)row * I + (uint32_t)col) * 2u : kOutOfRange);
          }
        }
      }
#pragma unroll
      for (int nb = 0; nb < kNbDown; ++nb) {
        if (nb < nbn) {
          const int slot = t0 + nb * 16 + r;
          u32x4 bh[KS], bl[KS];
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            const int col = (sb + s) * 32 + kg * 8;
            const bool ok = slot < cnt && sb + s < s_hi && col < I;
            const uint32_t off = ok ? ((uint32_t)slot * I + (uint32_t)col) * 2u : kOutOfRange;
            bh[s] = buf_ld128(hh_rsrc, off);
            bl[s] = buf_ld128(hl_rsrc, off);
          }
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int s = 0; s < KS; ++s) {
              acc[mb][nb] = mfma_16x16x32(A[mb][s], bh[s], acc[mb][nb]);
              acc[mb][nb] = mfma_16x16x32(A[mb][s], bl[s], acc[mb][nb]);
            }
        }
      }
    }

#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < kNbDown; ++nb)
        if (nb < nbn) part[wave][mb * kNbDown + nb][lane] = acc[mb][nb];
    __syncthreads();
    // fragment f = (mb, nb): reduced and stored by wave f % 4
    for (int f = wave; f < MB * kNbDown; f += 4) {
      const int mb = f / kNbDown, nb = f % kNbDown;
      if (nb >= nbn) continue;
      const f32x4 c = ((part[0][f][lane] + part[1][f][lane]) + part[2][f][lane]) + part[3][f][lane];
      const int slot = t0 + nb * 16 + r;
      const int o = o0 + mb * 16 + kg * 4;
      if (slot < cnt && o < H) {
        const int p = perm[base + slot];
        if (p >= 0 && p < n_pairs)
          *reinterpret_cast<float4*>(y + (size_t)p * H + o) = make_float4(c[0], c[1], c[2], c[3]);
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Persistent, software-pipelined streaming kernels (the decode fast path).
//
// Each block loops over a fixed sequence of tiles.  While tile j is being
// multiplied, reduced and stored, tile j+1's metadata, dispatch slots and
// weights are already in flight.  Loads retire in issue order for the
// vector-memory counter, so every wave issues tile j's activation loads
// BEFORE tile j+1's prefetch: waiting on tile j's operands then never waits
// on tile j+1's weights.  Two weight register buffers alternate (the loop
// body is instantiated twice with the buffers swapped), so nothing is copied.

struct StreamRange {
  int first, end, step;
};

// XCD x = block % 8 owns the contiguous tile range [x*per, (x+1)*per); its
// blocks take every (nblocks/8)-th tile of it, so concurrently streamed
// tiles of one expert share that XCD's L2 for their activations.
__device__ __forceinline__ StreamRange stream_range(int bid, int nblocks, int total) {
  const int xcd = bid & 7, local = bid >> 3;
  const int per = (total + 7) >> 3;
  return StreamRange{xcd * per + local, min(total, (xcd + 1) * per), nblocks >> 3};
}

struct ExpertTile {
  int e, cnt, base, sub;
  bool ok;
};

struct GateUpCtx {
  const uint16_t* w13;
  const int* perm;
  uint16_t* h_hi;
  uint16_t* h_lo;
  __amdgpu_buffer_rsrc_t x_rsrc;
  int H, I, k, n_pairs, s_lo, s_hi, lane, wave, r, kg;
};

template <int KS>
__device__ __forceinline__ void gu_load_a(u32x4 (&A)[KS], const GateUpCtx& c, const ExpertTile& t) {
  const auto rs = make_rsrc(c.w13 + (size_t)t.e * 2 * c.I * c.H,
                            t.ok ? 4u * (uint32_t)c.I * (uint32_t)c.H : 0u);
  const int wrow = c.r < 8 ? t.sub * 8 + c.r : c.I + t.sub * 8 + (c.r - 8);
  const uint32_t a_row = (uint32_t)wrow * c.H * 2u;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int col = (c.s_lo + s) * 32 + c.kg * 8;
    const bool ok = c.s_lo + s < c.s_hi && col < c.H;
    A[s] = buf_ld128(rs, ok ? a_row + (uint32_t)col * 2u : kOutOfRange);
  }
}

// Dispatch slots t0 + nb*16 + r of the tile's expert (pair ids; zero past
// the expert's count).
__device__ __forceinline__ void load_slots(uint32_t (&pv)[kNbGateUp], const int* perm, int r,
                                           const ExpertTile& t, int t0) {
  const auto rs = make_rsrc(perm + t.base, t.ok ? 4u * (uint32_t)t.cnt : 0u);
#pragma unroll
  for (int nb = 0; nb < kNbGateUp; ++nb) pv[nb] = buf_ld32(rs, (uint32_t)(t0 + nb * 16 + r) * 4u);
}

template <int KS>
__device__ __forceinline__ void gu_load_b(u32x4 (&B)[KS], const GateUpCtx& c, uint32_t pv,
                                          int slot, const ExpertTile& t) {
  const bool tok = t.ok && slot < t.cnt && pv < (uint32_t)c.n_pairs;
  const uint32_t xrow = (tok ? pv : 0u) / (uint32_t)c.k * (uint32_t)c.H * 2u;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int col = (c.s_lo + s) * 32 + c.kg * 8;
    const bool ok = tok && c.s_lo + s < c.s_hi && col < c.H;
    B[s] = buf_ld128(c.x_rsrc, ok ? xrow + (uint32_t)col * 2u : kOutOfRange);
  }
}

// Cross-wave sum of the partial tiles, SwiGLU, and the h hi/lo store for
// N-blocks [0, nbn) of the pass starting at slot t0.
__device__ __forceinline__ void gu_epilogue(const GateUpCtx& c, const ExpertTile& t,
                                            f32x4 (*part)[kNbGateUp][kWave],
                                            const f32x4 (&acc)[kNbGateUp], int t0, int nbn) {
#pragma unroll
  for (int nb = 0; nb < kNbGateUp; ++nb)
    if (nb < nbn) part[c.wave][nb][c.lane] = acc[nb];
  __syncthreads();
  if (c.wave < nbn) {
    const int nb = c.wave, lane = c.lane;
    const f32x4 v = ((part[0][nb][lane] + part[1][nb][lane]) + part[2][nb][lane]) + part[3][nb][lane];
    f32x4 u;
#pragma unroll
    for (int q = 0; q < 4; ++q) u[q] = __shfl_xor(v[q], 32);
    const int slot = t0 + nb * 16 + c.r;
    if (lane < 32 && slot < t.cnt) {
      float hv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) hv[q] = swiglu(v[q], u[q]);
      u32x2 hw, lw;
      split_bf16x4(hv, hw, lw);
      const size_t off = (size_t)(t.base + slot) * c.I + t.sub * 8 + c.kg * 4;
      *reinterpret_cast<uint2*>(c.h_hi + off) = make_uint2(hw[0], hw[1]);
      *reinterpret_cast<uint2*>(c.h_lo + off) = make_uint2(lw[0], lw[1]);
    }
  }
  __syncthreads();
}

// Metadata of the experts a block's tiles touch, staged in LDS once per
// block: the tiles of one XCD range cover at most kMaxRangeExperts active
// slots, so a tile's expert, count and first slot become one LDS read
// instead of two dependent global round trips per tile.
constexpr int kMaxRangeExperts = 1024 / 8 + 2;

struct TileTables {
  const int* s_e;     // LDS: expert id of staged slot i
  const int* s_cnt;   // LDS: its pair count
  const int* s_base;  // LDS: its first dispatch slot
  int a0, tpe;        // first staged active slot; tiles per expert
};

__device__ __forceinline__ ExpertTile staged_tile(const TileTables& tb, int tile) {
  const int a = tile / tb.tpe;
  const int i = a - tb.a0;
  const int e = tb.s_e[i];
  if (e < 0) return ExpertTile{0, 0, 0, 0, false};
  return ExpertTile{e, tb.s_cnt[i], tb.s_base[i], tile - a * tb.tpe, true};
}

// Stages slots [a0, a0 + n) of the active list; an entry that fails the
// consistency checks is stored with e = -1.  Ends with a block barrier.
__device__ __forceinline__ void stage_tiles(int* s_e, int* s_cnt, int* s_base, int a0, int n,
                                            const int* active, const int* counts,
                                            const int* offsets, int m, int n_pairs) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    int e = active[a0 + i];
    int cnt = 0, base = 0;
    if (e >= 0 && e < m) {
      cnt = counts[e];
      base = offsets[e];
      if (cnt <= 0 || base < 0 || cnt > n_pairs - base) e = -1;
    } else {
      e = -1;
    }
    s_e[i] = e;
    s_cnt[i] = cnt;
    s_base[i] = base;
  }
  __syncthreads();
}

// One pipelined tile: A holds this tile's weights (in flight or landed),
// pv its first 64 dispatch slots.  The next tile (`next_tile` >= 0) has its
// metadata resolved into *nx and its slots and weights requested into pvn /
// An.  The prefetch is issued unconditionally (no next tile = an empty
// buffer, so every load is out of range and touches no memory) and the
// first 16 tokens are multiplied in straight-line code: with no branch
// around loads in between, the wait-count analysis sees the exact load
// order and those MFMAs wait only on this tile's operands.
template <int KS>
__device__ __forceinline__ void gu_tile(const GateUpCtx& c, const TileTables& tb,
                                        const ExpertTile& t, int next_tile, ExpertTile* nx,
                                        u32x4 (&A)[KS], u32x4 (&An)[KS],
                                        const uint32_t (&pv)[kNbGateUp],
                                        uint32_t (&pvn)[kNbGateUp],
                                        f32x4 (*part)[kNbGateUp][kWave]) {
  u32x4 B[KS];
  gu_load_b(B, c, pv[0], c.r, t);
  ExpertTile n{0, 0, 0, 0, false};
  if (next_tile >= 0) n = staged_tile(tb, next_tile);
  *nx = n;
  load_slots(pvn, c.perm, c.r, n, 0);
  gu_load_a(An, c, n);

  f32x4 acc[kNbGateUp];
#pragma unroll
  for (int nb = 0; nb < kNbGateUp; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < KS; ++s) acc[0] = mfma_16x16x32(A[s], B[s], acc[0]);

  // the remaining 16-token blocks (rare at decode sizes)
  uint32_t pp[kNbGateUp] = {pv[0], pv[1], pv[2], pv[3]};
  for (int t0 = 0;;) {
    const int nbn = (min(16 * kNbGateUp, t.cnt - t0) + 15) >> 4;
#pragma unroll
    for (int nb = 0; nb < kNbGateUp; ++nb) {
      if ((t0 > 0 || nb > 0) && nb < nbn) {
        gu_load_b(B, c, pp[nb], t0 + nb * 16 + c.r, t);
#pragma unroll
        for (int s = 0; s < KS; ++s) acc[nb] = mfma_16x16x32(A[s], B[s], acc[nb]);
      }
    }
    gu_epilogue(c, t, part, acc, t0, nbn);
    t0 += 16 * kNbGateUp;
    if (t0 >= t.cnt) break;
    load_slots(pp, c.perm, c.r, t, t0);
#pragma unroll
    for (int nb = 0; nb < kNbGateUp; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

template <int KS>
__global__ __launch_bounds__(256, 2) void gate_up_stream_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w13,
    const int* __restrict__ counts, const int* __restrict__ offsets,
    const int* __restrict__ perm, const int* __restrict__ active,
    const int* __restrict__ n_active_p, uint16_t* __restrict__ h_hi,
    uint16_t* __restrict__ h_lo, int H, int I, int m, int k, int n_pairs, int T) {
  __shared__ f32x4 part[4][kNbGateUp][kWave];
  const int n_act = *n_active_p;
  if (n_act <= 0 || n_act > m) return;
  const int tpe = I / 8;
  const StreamRange rg = stream_range(blockIdx.x, gridDim.x, n_act * tpe);
  if (rg.first >= rg.end) return;

  GateUpCtx c;
  c.w13 = w13;
  c.perm = perm;
  c.h_hi = h_hi;
  c.h_lo = h_lo;
  c.x_rsrc = make_rsrc(x, 2u * (uint32_t)T * (uint32_t)H);
  c.H = H;
  c.I = I;
  c.k = k;
  c.n_pairs = n_pairs;
  c.lane = threadIdx.x & 63;
  c.wave = threadIdx.x >> 6;
  c.r = c.lane & 15;
  c.kg = c.lane >> 4;
  wave_ksteps((H + 31) >> 5, c.wave, &c.s_lo, &c.s_hi);

  __shared__ int s_e[kMaxRangeExperts], s_cnt[kMaxRangeExperts], s_base[kMaxRangeExperts];
  const int a0 = rg.first / tpe, a1 = (rg.end - 1) / tpe;
  stage_tiles(s_e, s_cnt, s_base, a0, a1 - a0 + 1, active, counts, offsets, m, n_pairs);
  const TileTables tb{s_e, s_cnt, s_base, a0, tpe};
  u32x4 A0[KS], A1[KS];
  uint32_t p0[kNbGateUp], p1[kNbGateUp];
  int tile = rg.first;
  ExpertTile t = staged_tile(tb, tile), nx = t;
  load_slots(p0, perm, c.r, t, 0);
  gu_load_a(A0, c, t);
  for (;;) {
    int nt = tile + rg.step < rg.end ? tile + rg.step : -1;
    gu_tile(c, tb, t, nt, &nx, A0, A1, p0, p1, part);
    if (nt < 0) break;
    tile = nt;
    t = nx;
    nt = tile + rg.step < rg.end ? tile + rg.step : -1;
    gu_tile(c, tb, t, nt, &nx, A1, A0, p1, p0, part);
    if (nt < 0) break;
    tile = nt;
    t = nx;
  }
}

struct DownCtx {
  const uint16_t* w2;
  const uint16_t* h_hi;
  const uint16_t* h_lo;
  const int* perm;
  float* y;
  int H, I, n_pairs, s_lo, s_hi, lane, wave, r, kg;
};

template <int KS, int MB>
__device__ __forceinline__ void dn_load_a(u32x4 (&A)[MB][KS], const DownCtx& c, const ExpertTile& t) {
  const auto rs = make_rsrc(c.w2 + (size_t)t.e * c.H * c.I,
                            t.ok ? 2u * (uint32_t)c.H * (uint32_t)c.I : 0u);
  const int o0 = t.sub * 16 * MB;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int row = o0 + mb * 16 + c.r;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int col = (c.s_lo + s) * 32 + c.kg * 8;
      const bool ok = row < c.H && c.s_lo + s < c.s_hi && col < c.I;
      A[mb][s] = buf_ld128(rs, ok ? ((uint32_t)row * c.I + (uint32_t)col) * 2u : kOutOfRange);
    }
  }
}

template <int KS>
__device__ __forceinline__ void dn_load_b(u32x4 (&bh)[KS], u32x4 (&bl)[KS], const DownCtx& c,
                                          const ExpertTile& t, int slot) {
  const uint32_t bytes = t.ok ? 2u * (uint32_t)t.cnt * (uint32_t)c.I : 0u;
  const auto hs = make_rsrc(c.h_hi + (size_t)t.base * c.I, bytes);
  const auto ls = make_rsrc(c.h_lo + (size_t)t.base * c.I, bytes);
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int col = (c.s_lo + s) * 32 + c.kg * 8;
    const bool ok = slot < t.cnt && c.s_lo + s < c.s_hi && col < c.I;
    const uint32_t off = ok ? ((uint32_t)slot * c.I + (uint32_t)col) * 2u : kOutOfRange;
    bh[s] = buf_ld128(hs, off);
    bl[s] = buf_ld128(ls, off);
  }
}

// Reduction across the four waves and the y store of one pass.
template <int MB>
__device__ __forceinline__ void dn_epilogue(const DownCtx& c, const ExpertTile& t,
                                            f32x4 (*part)[MB * kNbDown][kWave],
                                            const f32x4 (&acc)[MB][kNbDown],
                                            const uint32_t (&ps)[kNbDown], int t0, int nbn) {
  const int o0 = t.sub * 16 * MB;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < kNbDown; ++nb)
      if (nb < nbn) part[c.wave][mb * kNbDown + nb][c.lane] = acc[mb][nb];
  __syncthreads();
  for (int f = c.wave; f < MB * kNbDown; f += 4) {
    const int mb = f / kNbDown, nb = f % kNbDown;
    if (nb >= nbn) continue;
    const int lane = c.lane;
    const f32x4 v = ((part[0][f][lane] + part[1][f][lane]) + part[2][f][lane]) + part[3][f][lane];
    const int slot = t0 + nb * 16 + c.r;
    const int o = o0 + mb * 16 + c.kg * 4;
    const uint32_t p = ps[nb];
    if (slot < t.cnt && o < c.H && p < (uint32_t)c.n_pairs)
      *reinterpret_cast<float4*>(c.y + (size_t)p * c.H + o) = make_float4(v[0], v[1], v[2], v[3]);
  }
  __syncthreads();
}

__device__ __forceinline__ void dn_load_slots(uint32_t (&ps)[kNbDown], const DownCtx& c,
                                              const ExpertTile& t, int t0) {
  const auto rs = make_rsrc(c.perm + t.base, t.ok ? 4u * (uint32_t)t.cnt : 0u);
#pragma unroll
  for (int nb = 0; nb < kNbDown; ++nb) ps[nb] = buf_ld32(rs, (uint32_t)(t0 + nb * 16 + c.r) * 4u);
}

// One pipelined down tile (same structure as gu_tile).
template <int KS, int MB>
__device__ __forceinline__ void dn_tile(const DownCtx& c, const TileTables& tb,
                                        const ExpertTile& t, int next_tile, ExpertTile* nx,
                                        u32x4 (&A)[MB][KS], u32x4 (&An)[MB][KS],
                                        f32x4 (*part)[MB * kNbDown][kWave]) {
  u32x4 bh[KS], bl[KS];
  dn_load_b(bh, bl, c, t, c.r);
  uint32_t ps[kNbDown];
  dn_load_slots(ps, c, t, 0);
  ExpertTile n{0, 0, 0, 0, false};
  if (next_tile >= 0) n = staged_tile(tb, next_tile);
  *nx = n;
  dn_load_a(An, c, n);

  f32x4 acc[MB][kNbDown];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < kNbDown; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      acc[mb][0] = mfma_16x16x32(A[mb][s], bh[s], acc[mb][0]);
      acc[mb][0] = mfma_16x16x32(A[mb][s], bl[s], acc[mb][0]);
    }

  for (int t0 = 0;;) {
    const int nbn = (min(16 * kNbDown, t.cnt - t0) + 15) >> 4;
#pragma unroll
    for (int nb = 0; nb < kNbDown; ++nb) {
      if ((t0 > 0 || nb > 0) && nb < nbn) {
        dn_load_b(bh, bl, c, t, t0 + nb * 16 + c.r);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            acc[mb][nb] = mfma_16x16x32(A[mb][s], bh[s], acc[mb][nb]);
            acc[mb][nb] = mfma_16x16x32(A[mb][s], bl[s], acc[mb][nb]);
          }
      }
    }
    dn_epilogue<MB>(c, t, part, acc, ps, t0, nbn);
    t0 += 16 * kNbDown;
    if (t0 >= t.cnt) break;
    dn_load_slots(ps, c, t, t0);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < kNbDown; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

template <int KS, int MB>
__global__ __launch_bounds__(256, 2) void down_stream_kernel(
    const uint16_t* __restrict__ h_hi, const uint16_t* __restrict__ h_lo,
    const uint16_t* __restrict__ w2, const int* __restrict__ counts,
    const int* __restrict__ offsets, const int* __restrict__ perm,
    const int* __restrict__ active, const int* __restrict__ n_active_p, float* __restrict__ y,
    int H, int I, int m, int n_pairs) {
  __shared__ f32x4 part[4][MB * kNbDown][kWave];
  const int n_act = *n_active_p;
  if (n_act <= 0 || n_act > m) return;
  const int tpe = (H + 16 * MB - 1) / (16 * MB);
  const StreamRange rg = stream_range(blockIdx.x, gridDim.x, n_act * tpe);
  if (rg.first >= rg.end) return;

  DownCtx c;
  c.w2 = w2;
  c.h_hi = h_hi;
  c.h_lo = h_lo;
  c.perm = perm;
  c.y = y;
  c.H = H;
  c.I = I;
  c.n_pairs = n_pairs;
  c.lane = threadIdx.x & 63;
  c.wave = threadIdx.x >> 6;
  c.r = c.lane & 15;
  c.kg = c.lane >> 4;
  wave_ksteps((I + 31) >> 5, c.wave, &c.s_lo, &c.s_hi);

  __shared__ int s_e[kMaxRangeExperts], s_cnt[kMaxRangeExperts], s_base[kMaxRangeExperts];
  const int a0 = rg.first / tpe, a1 = (rg.end - 1) / tpe;
  stage_tiles(s_e, s_cnt, s_base, a0, a1 - a0 + 1, active, counts, offsets, m, n_pairs);
  const TileTables tb{s_e, s_cnt, s_base, a0, tpe};
  u32x4 A0[MB][KS], A1[MB][KS];
  int tile = rg.first;
  ExpertTile t = staged_tile(tb, tile), nx = t;
  dn_load_a(A0, c, t);
  for (;;) {
    int nt = tile + rg.step < rg.end ? tile + rg.step : -1;
    dn_tile(c, tb, t, nt, &nx, A0, A1, part);
    if (nt < 0) break;
    tile = nt;
    t = nx;
    nt = tile + rg.step < rg.end ? tile + rg.step : -1;
    dn_tile(c, tb, t, nt, &nx, A1, A0, part);
    if (nt < 0) break;
    tile = nt;
    t = nx;
  }
}

// One thread per (token, 4 consecutive outputs); the k slot loads of a
// group of 8 are issued before their fused multiply-adds, which then run in
// slot order.
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ y,
                                                     const float* __restrict__ topk_w,
                                                     const int* __restrict__ n_active_p,
                                                     float* __restrict__ out, int T, int H,
                                                     int k, int m) {
  const int hq = H >> 2;
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)T * hq) return;
  const int t = (int)(idx / hq), c = (int)(idx - (size_t)t * hq);
  // the n_active load and the y / gate loads go out together; an invalid
  // plan (n_active outside [0, m]) turns the result into NaN afterwards
  const int na = *n_active_p;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  const float* yt = y + (size_t)t * k * H + 4 * c;
  const float* wt = topk_w + (size_t)t * k;
  for (int j0 = 0; j0 < k; j0 += 8) {
    float4 v[8];
    float w[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (j0 + q < k) {
        v[q] = *reinterpret_cast<const float4*>(yt + (size_t)(j0 + q) * H);
        w[q] = wt[j0 + q];
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (j0 + q < k) {
        acc.x = fmaf(w[q], v[q].x, acc.x);
        acc.y = fmaf(w[q], v[q].y, acc.y);
        acc.z = fmaf(w[q], v[q].z, acc.z);
        acc.w = fmaf(w[q], v[q].w, acc.w);
      }
    }
  }
  if (na < 0 || na > m) {
    const float nan = __builtin_nanf("");
    acc = make_float4(nan, nan, nan, nan);
  }
  *reinterpret_cast<float4*>(out + (size_t)t * H + 4 * c) = acc;
}

int round8(long v) { return (int)align_up((size_t)v, 8); }

}  // namespace

const float* forward_y(const void* workspace, int T, int H, int I, int k) {
  return carve(const_cast<void*>(workspace), T * k, H, I).y;
}

size_t forward_workspace_bytes(int T, int H, int I, int k) {
  if (T <= 0) return 0;
  const int n_pairs = T * k;
  return 2 * h_bytes(n_pairs, I) + y_bytes(n_pairs, H);
}

// Persistent grid: `per_cu` resident blocks on every compute unit, a
// multiple of 8 so each XCD gets the same number.
static int stream_blocks(int per_cu) {
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 256;
  return round8((long)cus * per_cu);
}

Kernels gate_up_kernels(int T, int H, int I, int m, int k, bool tiled) {
  if (T <= 0) return Kernels::kNone;
  if (prefill_supported(T, H, I, m, k)) return Kernels::kPrefill;
  if (skinny_gate_up_supported(T, H, I, m, k)) return Kernels::kSplitK;
  // the tiled layout is only produced for shapes the wave kernels take
  if (tiled || wave_stream_supported(T, H, I, k)) return Kernels::kWave;
  return Kernels::kGeneric;
}

Kernels down_kernels(int T, int H, int I, int m, int k, bool tiled) {
  if (T <= 0) return Kernels::kNone;
  if (prefill_supported(T, H, I, m, k)) return Kernels::kPrefill;
  if (skinny_down_supported(T, H, I, m, k)) return Kernels::kSplitK;
  if (tiled || wave_stream_supported(T, H, I, k)) return Kernels::kWave;
  return Kernels::kGeneric;
}

hipError_t launch_gate_up(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                          const int* counts, const int* offsets, const int* perm,
                          const int* active, const int* n_active, int H, int I, int m, int k,
                          void* workspace, hipStream_t stream, bool identity_plan) {
  const Kernels family = gate_up_kernels(T, H, I, m, k, tiled);
  if (family == Kernels::kNone) return hipSuccess;
  const ForwardWs ws = carve(workspace, T * k, H, I);
  if (family == Kernels::kPrefill)
    return launch_gate_up_prefill(x, T, w13, tiled, counts, offsets, perm, active, n_active, H,
                                  I, m, k, ws.h_hi, ws.h_lo, stream);
  if (family == Kernels::kSplitK)
    return launch_gate_up_skinny(x, T, w13, tiled, counts, offsets, perm, active, n_active, H, I,
                                 m, k, ws.h_hi, ws.h_lo, identity_plan, stream);
  if (family == Kernels::kWave)
    return launch_gate_up_wave(x, T, w13, tiled, counts, offsets, perm, active, n_active, H, I, m,
                               k, ws.h_hi, ws.h_lo, stream);
  const int per_wave = (((H + 31) >> 5) + 3) >> 2;
  const long tiles = (long)m * (I / 8);
  if (per_wave <= 8) {
    const int blocks = (int)std::min<long>(round8(tiles), stream_blocks(2));
    gate_up_stream_kernel<8><<<blocks, 256, 0, stream>>>(x, w13, counts, offsets, perm, active,
                                                         n_active, ws.h_hi, ws.h_lo, H, I, m, k,
                                                         T * k, T);
  } else if (per_wave <= 16) {
    const int blocks = (int)std::min<long>(round8(tiles), stream_blocks(2));
    gate_up_stream_kernel<16><<<blocks, 256, 0, stream>>>(x, w13, counts, offsets, perm, active,
                                                          n_active, ws.h_hi, ws.h_lo, H, I, m, k,
                                                          T * k, T);
  } else {
    gate_up_generic_kernel<16><<<round8(tiles), 256, 0, stream>>>(
        x, w13, counts, offsets, perm, active, n_active, ws.h_hi, ws.h_lo, H, I, m, k, T * k, T);
  }
  return hipGetLastError();
}

hipError_t launch_gate_up_building_plan(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                       const int* topk_ids, int* counts, int* offsets, int* perm,
                                       int* active, int* n_active, int H, int I, int m, int k,
                                       void* workspace, hipStream_t stream) {
  const ForwardWs ws = carve(workspace, T * k, H, I);
  return launch_gate_up_wave_plan(x, T, w13, tiled, topk_ids, counts, offsets, perm, active,
                                  n_active, H, I, m, k, ws.h_hi, ws.h_lo, stream);
}

template <int KS, int MB>
static void launch_down_t(const ForwardWs& ws, const uint16_t* w2, const int* counts,
                          const int* offsets, const int* perm, const int* active,
                          const int* n_active, int H, int I, int m, int n_pairs,
                          hipStream_t stream) {
  const long tiles = (long)m * ((H + 16 * MB - 1) / (16 * MB));
  const int blocks = (int)std::min<long>(round8(tiles), stream_blocks(2));
  down_stream_kernel<KS, MB><<<blocks, 256, 0, stream>>>(ws.h_hi, ws.h_lo, w2, counts, offsets,
                                                         perm, active, n_active, ws.y, H, I, m,
                                                         n_pairs);
}

hipError_t launch_down(int T, const uint16_t* w2, bool tiled, const int* counts,
                       const int* offsets, const int* perm, const int* active,
                       const int* n_active, int H, int I, int m, int k, void* workspace,
                       hipStream_t stream, bool identity_plan) {
  const Kernels family = down_kernels(T, H, I, m, k, tiled);
  if (family == Kernels::kNone) return hipSuccess;
  const ForwardWs ws = carve(workspace, T * k, H, I);
  if (family == Kernels::kPrefill)
    return launch_down_prefill(T, w2, tiled, counts, offsets, perm, active, n_active, H, I, m, k,
                               ws.h_hi, ws.h_lo, ws.y, stream);
  if (family == Kernels::kSplitK)
    return launch_down_skinny(T, w2, tiled, counts, offsets, perm, active, n_active, H, I, m, k,
                              ws.h_hi, ws.h_lo, ws.y, identity_plan, stream);
  if (family == Kernels::kWave)
    return launch_down_wave(T, w2, tiled, counts, offsets, perm, active, n_active, H, I, m, k,
                            ws.h_hi, ws.h_lo, ws.y, stream);
  const int per_wave = (((I + 31) >> 5) + 3) >> 2;  // K steps of one wave
  // about 16 weight loads in flight per wave: MB row blocks x per_wave steps
  if (per_wave <= 2)
    launch_down_t<2, 4>(ws, w2, counts, offsets, perm, active, n_active, H, I, m, T * k, stream);
  else if (per_wave <= 4)
    launch_down_t<4, 4>(ws, w2, counts, offsets, perm, active, n_active, H, I, m, T * k, stream);
  else if (per_wave <= 6)
    launch_down_t<6, 2>(ws, w2, counts, offsets, perm, active, n_active, H, I, m, T * k, stream);
  else if (per_wave <= 8)
    launch_down_t<8, 2>(ws, w2, counts, offsets, perm, active, n_active, H, I, m, T * k, stream);
  else
    down_generic_kernel<16, 1><<<round8((long)m * ((H + 15) / 16)), 256, 0, stream>>>(
        ws.h_hi, ws.h_lo, w2, counts, offsets, perm, active, n_active, ws.y, H, I, m, T * k);
  return hipGetLastError();
}

hipError_t launch_combine(int T, const float* topk_w, const int* n_active, float* out, int H,
                          int I, int m, int k, void* workspace, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const ForwardWs ws = carve(workspace, T * k, H, I);
  const size_t threads = (size_t)T * (H / 4);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  combine_kernel<<<blocks, 256, 0, stream>>>(ws.y, topk_w, n_active, out, T, H, k, m);
  return hipGetLastError();
}

}  // namespace sw
