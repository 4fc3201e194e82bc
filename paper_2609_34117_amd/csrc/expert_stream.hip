// Wave-streaming expert FFN kernels for gfx950: the decode fast path of the
// MoE layer (Section 2.1: a decode step reads every distinct expert chosen
// across the batch, so the step is bound by streaming expert weights).
//
// Design:
//   - A persistent grid of one 8-wave block per compute unit.  The tiles of
//     all active experts form one list; block b owns the contiguous,
//     equal-sized range b*per .. (b+1)*per of it, which crosses at most a few
//     expert boundaries ("segments").  When some expert has more tokens than
//     a whole-K pass holds, the blocks instead own equal runs of estimated
//     cost (the cost-weighted walk below), so that the tiles of popular
//     experts, which cost more each, are spread over more blocks.
//   - Each wave owns whole tiles (16 weight rows over the full K) and
//     streams them as 8 KiB chunks through a kDepth-deep register pipeline
//     (3, or 2 where a wide pass needs the registers for its accumulators):
//     the kDepth - 1 chunks ahead are always in flight.  The B operand
//     (tokens) comes from LDS, so waiting for activations never waits on
//     weights.  The first chunks of a segment are issued as soon as its
//     expert id is known, before the activation staging and its barriers.
//   - Each tile is streamed once for all of its expert's tokens (up to
//     kNbMax * 16 of them, 64 to 128 by variant; more take further passes).  When the segment's
//     tokens fit in LDS with the whole contraction (K = H for gate/up, I for
//     down) they are staged once and the waves run through their tiles
//     with no barrier ("whole-K" pass).  Otherwise ("sliced" pass) K is cut
//     into slices of whole chunks that fit for all of the tokens: the block
//     takes one tile per wave at a time, and for each slice stages that
//     slice of every token row, then each wave streams its tile's chunks of
//     the slice into accumulators that live across the slices.  Where two
//     slices fit, they alternate between two LDS buffers and each is staged
//     a whole slice ahead of its use.  A popular expert thus costs the same
//     weight bytes as any other; its tokens are re-read from L2 once per
//     group of 8 tiles.
//   - Every step issues the same memory operations (out-of-range offsets
//     for missing chunks and for epilogue stores on non-final chunks), so
//     the compiler's wait counts are exact and the pipeline never drains on
//     a conservative wait; the slice staging waits only for its own loads
//     and the chunks before it (an explicit count, with the load order
//     pinned), not for the weights issued after it.
// Tiles:  gate_up: 8 gate rows + the 8 matching up rows; epilogue writes
//         h = silu(g) * u as a bf16 hi/lo pair.
//         down: 16 output rows of W2; epilogue writes y (fp32) per pair.
#include <cmath>

#include "dispatch_block.h"
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kWv = 8;            // waves per block
constexpr int kBlk = 64 * kWv;    // threads per block
constexpr int kKC = 8;            // 32-wide K steps per streamed chunk
constexpr int kChunkCols = 32 * kKC;
constexpr int kNT = 32;           // tokens of the whole-K pass of a small batch
constexpr int kPad = 8;           // bf16 elements of padding per staged row
constexpr int kMaxExperts = 1024;  // pool size limit of the library (routed + shared parts)
// LDS of the staged activations (bf16 elements): 32 whole rows of the
// largest H, or of both h planes at the largest I, with room to spare for
// the sliced passes' larger token counts
constexpr int kStage = 76800;
static_assert(kNT * (kMaxStreamH + kPad) <= kStage, "whole-K rows of a 32-token pass");
static_assert(2 * kNT * (kMaxStreamI + kPad) <= kStage, "whole-K h rows of a 32-token pass");
// the narrowest slice (one chunk) of the widest passes fits: 128 tokens of
// x, 96 tokens of h hi and lo
static_assert(128 * (kChunkCols + kPad) <= kStage && 2 * 96 * (kChunkCols + kPad) <= kStage,
              "one-chunk slices of the widest passes");

// One staged row of `bytes` (a multiple of 16) into LDS at `dst`, straight
// from memory: a wave's buffer load with the LDS bit moves 64 x 16 bytes,
// lane l to dst + 16 l, so the row is bytes / 1 KiB such loads, the last
// one on the lanes still inside the row.  src is the row's byte offset in
// the resource (out of range: the lanes read zeros).  dst and the loop are
// wave-uniform; the caller waits for vmcnt before the rows are read (the
// compiler does not track these LDS writes).
__device__ __forceinline__ void stage_row(__amdgpu_buffer_rsrc_t r, uint32_t src, uint16_t* dst,
                                          int bytes, int lane) {
  for (int q = 0; q * 1024 < bytes; ++q) {
    if (q * 1024 + lane * 16 < bytes)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          r, (__attribute__((address_space(3))) void*)(dst + q * 512), 16,
          src == kOutOfRange ? kOutOfRange : src + (uint32_t)(q * 1024 + lane * 16), 0, 0, 0);
  }
}

// s_waitcnt immediates (gfx9 encoding): at most n vector-memory operations
// outstanding, expcnt and lgkmcnt left alone
constexpr int vmcnt_at_most(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int kVmcntZero = vmcnt_at_most(0);
// ... and every LDS access of this wave done
constexpr int vmcnt_at_most_lds_done(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }
// only this wave's LDS accesses done (vmcnt at its maximum)
constexpr int kLdsDone = vmcnt_at_most_lds_done(63);

// The barriers around the staging of a K slice.  Plain s_barriers with
// explicit waits: a __syncthreads fence could also wait for the weight
// loads in flight, which must stay outstanding across the staging.
// Before: every wave's reads of the previous slice are done.
__device__ __forceinline__ void slice_barrier_before() {
  __builtin_amdgcn_s_waitcnt(kLdsDone);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}
// After: the slice's loads of every wave have landed; `after` loads issued
// since the staging stay outstanding.
template <int kAfter>
__device__ __forceinline__ void slice_barrier_after() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(kAfter));
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// A double-buffered slice's wait: every staging load of this wave issued
// before the last `after` vector-memory operations has landed, and this
// wave's LDS accesses are done.  `after` (wave-uniform, 0..63) is rounded
// down to a multiple of 8, which only waits for more.
__device__ __forceinline__ void wait_staged_before(int after) {
  switch (after >> 3) {
    case 0: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(0)); break;
    case 1: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(8)); break;
    case 2: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(16)); break;
    case 3: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(24)); break;
    case 4: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(32)); break;
    case 5: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(40)); break;
    case 6: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(48)); break;
    default: __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(56)); break;
  }
}

// LDS offset (elements) of slice sigma's buffer: the two halves of the
// staging area alternate on a double-buffered pass.
__device__ __forceinline__ int slice_buffer(bool dbl, int sigma) {
  return (dbl && (sigma & 1)) ? kStage / 2 : 0;
}

// Position of a wave's chunk q in its pass: tile group (or own tile) j,
// chunk c of the tile, and on a sliced pass the slice sl and the chunk's
// place ks in it.  Advanced by one step at a time, so that the chunk loops
// do no integer division per step.
struct ChunkPos {
  int j, c, sl, ks;
  __device__ __forceinline__ void start(int q, int cpt, int cps) {
    j = q / cpt;
    c = q - j * cpt;
    sl = c / cps;
    ks = c - sl * cps;
  }
  __device__ __forceinline__ void next(int cpt, int cps) {
    ++c;
    if (++ks == cps) {
      ks = 0;
      ++sl;
    }
    if (c == cpt) {
      c = ks = sl = 0;
      ++j;
    }
  }
};

struct Segment {
  int lo, hi;  // tile range [lo, hi) inside one expert
  int a, e, cnt, base;
  int w_end;   // cost position after the segment (cost-weighted walk)
  bool e_ok;   // expert id in range: its weights may be read
};

// Next segment of the block's tile range starting at tile `lo`.  With
// `all_active` (n_active == m) the active list is the identity, so the
// expert is the slot itself and active[] is not read.  The loads of the
// expert's count and offset are issued here but consumed only by
// finish_segment, so the first weight chunks can go out in between.
// Without `read_plan` the count and offset are left for the caller.
__device__ __forceinline__ Segment next_segment(int lo, int r_hi, int tpe, const int* active,
                                                const int* counts, const int* offsets, int m,
                                                bool all_active, bool read_plan = true) {
  Segment s;
  s.lo = lo;
  s.a = lo / tpe;
  s.hi = min(r_hi, (s.a + 1) * tpe);
  const int e = all_active ? s.a : active[s.a];
  s.e_ok = e >= 0 && e < m;
  s.e = s.e_ok ? e : 0;
  s.cnt = read_plan ? counts[s.e] : 0;
  s.base = read_plan ? offsets[s.e] : 0;
  s.w_end = 0;
  return s;
}

// A segment whose pair range is not inside [0, n_pairs) has no tokens.
__device__ __forceinline__ void finish_segment(Segment& s, int n_pairs) {
  const bool ok = s.e_ok && s.cnt > 0 && s.base >= 0 && s.cnt <= n_pairs - s.base;
  if (!ok) {
    s.cnt = 0;
    s.base = 0;
  }
}

// Balanced contiguous tile range of this block.
__device__ __forceinline__ void block_range(int total, int* r_lo, int* r_hi) {
  const int per = (total + (int)gridDim.x - 1) / (int)gridDim.x;
  *r_lo = min(total, (int)blockIdx.x * per);
  *r_hi = min(total, *r_lo + per);
}

// How one pass of a segment is staged.  A pass takes up to pmax tokens
// (passes of a segment are balanced); `planes` staged rows per token (1:
// x, 2: h hi and lo) of K columns.  Whole-K when all of them fit.  Else the
// widest slice of whole chunks of which two fit ("double-buffered": the
// next slice is staged while the current one is read), or failing that of
// which one fits.
struct PassShape {
  int n;       // tokens of the pass
  int nbn;     // 16-token MFMA column blocks
  int cps;     // chunks per K slice (cpt for a whole-K pass)
  int stride;  // LDS elements per staged row
  bool sliced;
  bool dbl;    // sliced into two LDS buffers (at 0 and kStage / 2)
};

__device__ __forceinline__ int pass_tokens(int cnt, int pmax) {
  const int np = (cnt + pmax - 1) / pmax;
  return (cnt + np - 1) / np;
}

__device__ __forceinline__ PassShape pass_shape(int n, int K, int cpt, int planes) {
  PassShape ps;
  ps.n = n;
  ps.nbn = (n + 15) >> 4;
  const int rows = ps.nbn * 16 * planes;
  ps.dbl = false;
  if (rows * (K + kPad) <= kStage) {
    ps.cps = cpt;
    ps.stride = K + kPad;
    ps.sliced = false;
  } else {
    const int c2 = (kStage / 2 / rows - kPad) / kChunkCols;
    const int c = c2 >= 1 ? c2 : (kStage / rows - kPad) / kChunkCols;
    ps.cps = max(1, min(c, cpt));
    ps.stride = ps.cps * kChunkCols + kPad;
    ps.sliced = true;
    ps.dbl = c2 >= 1;
  }
  return ps;
}

// Cost-weighted walk.  Equal tile ranges balance the blocks when every
// expert takes one whole-K pass.  A sliced pass costs more per tile: its
// waves meet at a barrier on every slice, its tokens are staged again for
// every group of tiles, and its wider passes take more MFMA and LDS work.
// Per-block timings put a double-buffered sliced tile of 3 to 6 column
// blocks at 2.9 to 4 times a whole-K tile, and a single-buffered slice
// (which drains the weight pipeline) at about one whole-K tile.  Every extra
// pass streams the tile again.  So when some expert needs a sliced pass or
// several passes, the blocks take equal runs of cost instead: expert slot
// a's tiles each cost tile_cost(count) units and start at wp[a] + i * cost,
// and block b owns the tiles whose start lies in its run.  A popular expert
// is then spread over more blocks instead of lengthening the few that own
// its tiles.
constexpr int kCostWholeK = 8;     // one whole-K pass over a tile
constexpr int kCostSliced = 6;     // added per tile by a double-buffered sliced pass
constexpr int kCostSlicedNb = 3;   // ... and per 16-token column block of it
constexpr int kCostSlice1 = 8;     // added per K slice of a single-buffered pass

__device__ __forceinline__ int pass_cost(int n, int K, int cpt, int planes) {
  const PassShape ps = pass_shape(n, K, cpt, planes);
  // a whole-K pass costs more with its column blocks too: per-block timings
  // put each further block of 16 tokens at about 6% of a tile for gate/up
  // and 12% for down (two h planes)
  if (!ps.sliced) return kCostWholeK + (ps.nbn - 1) * planes / 2;
  if (ps.dbl) return kCostWholeK + kCostSliced + kCostSlicedNb * ps.nbn;
  return kCostWholeK + kCostSlice1 * ((cpt + ps.cps - 1) / ps.cps);
}

// Cost of one tile of an expert with n pairs, in passes of at most pmax.
__device__ __forceinline__ int tile_cost(int n, int pmax, int K, int cpt, int planes) {
  if (n <= 0) return 0;
  const int np = (n + pmax - 1) / pmax, per = (n + np - 1) / np;
  return (np - 1) * pass_cost(per, K, cpt, planes) + pass_cost(n - (np - 1) * per, K, cpt, planes);
}

// Tokens of the largest whole-K pass.
__device__ __forceinline__ int whole_k_tokens(int pmax, int K, int planes) {
  return min(pmax, 16 * (kStage / (16 * planes * (K + kPad))));
}

// Offsets of experts 2t .. 2t + 2 (thread t): one round of independent
// loads at the kernel's start, with indices clamped to offsets[m] (past m
// the differences are 0).
struct PairCounts {
  int o0, o1, o2;
};

__device__ __forceinline__ PairCounts load_pair_counts(const int* offsets, int m) {
  const int e0 = 2 * (int)threadIdx.x;
  return PairCounts{offsets[min(e0, m)], offsets[min(e0 + 1, m)], offsets[min(e0 + 2, m)]};
}

// Whether some expert has more pairs than a whole-K pass holds (a garbage
// plan can only make this true, which takes the checked weighted walk):
// each wave posts its verdict to its own LDS slot before a barrier the
// kernel has anyway, and every thread reads the eight slots after it.
// m <= 2 * kBlk.
__device__ __forceinline__ void post_heavy_verdict(const PairCounts& c, int light, int* verdict) {
  const bool big = c.o1 - c.o0 > light || c.o2 - c.o1 > light;
  const bool any = __ballot(big) != 0;
  if ((threadIdx.x & 63) == 0) verdict[threadIdx.x >> 6] = any ? 1 : 0;
}

__device__ __forceinline__ bool read_heavy_verdict(const int* verdict) {
  int v = 0;
#pragma unroll
  for (int w = 0; w < kWv; ++w) v |= verdict[w];
  return v != 0;
}

// The same with a barrier of its own.  Every thread of the block calls it.
__device__ __forceinline__ bool some_expert_is_heavy(const PairCounts& c, int light,
                                                     int* verdict) {
  post_heavy_verdict(c, light, verdict);
  __syncthreads();
  return read_heavy_verdict(verdict);
}

// wp[a] = cost before active slot a's tiles, wp[n_act] = the total.  Every
// thread of the block calls it; n_act <= 2 * kBlk.
__device__ void weighted_work(int n_act, int tpe, const int* active, const int* counts,
                              const int* offsets, int m, int n_pairs, int pmax, int K, int cpt,
                              int planes, int* wp, uint32_t* scan) {
  auto cost = [&](int a) {
    if (a >= n_act) return 0;
    const int e = active[a];
    if (e < 0 || e >= m) return 0;
    const int c = counts[e], b = offsets[e];
    if (c <= 0 || b < 0 || c > n_pairs - b) return 0;
    return tpe * tile_cost(c, pmax, K, cpt, planes);
  };
  const int a0 = 2 * (int)threadIdx.x;
  const int c0 = cost(a0), c1 = cost(a0 + 1);
  uint32_t off, unused, total, unused_t;
  block_exclusive_scan2((uint32_t)(c0 + c1), 0u, scan, &off, &unused, &total, &unused_t);
  if (a0 < n_act) wp[a0] = (int)off;
  if (a0 + 1 < n_act) wp[a0 + 1] = (int)off + c0;
  if (threadIdx.x == 0) wp[n_act] = (int)total;
  __syncthreads();
}

// Segment of the weighted walk from cost position w: the first tile whose
// start is at or after w, and the following tiles of its expert whose starts
// lie before w_hi.  s.lo == s.hi when no tile starts in [w, w_hi).
__device__ __forceinline__ Segment weighted_segment(int w, int w_hi, int n_act, const int* wp,
                                                    int tpe, const int* active,
                                                    const int* counts, const int* offsets,
                                                    int m) {
  int a = 0, hi = n_act - 1;  // the last slot a with wp[a] <= w
  while (a < hi) {
    const int mid = (a + hi + 1) >> 1;
    if (wp[mid] <= w)
      a = mid;
    else
      hi = mid - 1;
  }
  Segment s;
  int c = (wp[a + 1] - wp[a]) / tpe, i0 = c > 0 ? (w - wp[a] + c - 1) / c : tpe;
  while (i0 >= tpe && a + 1 < n_act && wp[a + 1] < w_hi) {  // the next expert's first tile
    ++a;
    c = (wp[a + 1] - wp[a]) / tpe;
    i0 = c > 0 ? 0 : tpe;
  }
  const int i1 = c > 0 ? min(tpe, (w_hi - wp[a] + c - 1) / c) : 0;
  s.a = a;
  s.lo = a * tpe + min(i0, tpe);
  s.hi = a * tpe + max(min(i0, tpe), i1);
  s.w_end = i1 >= tpe ? wp[a + 1] : w_hi;
  const int e = active[a];
  s.e_ok = e >= 0 && e < m;
  s.e = s.e_ok ? e : 0;
  s.cnt = counts[s.e];
  s.base = offsets[s.e];
  return s;
}

// ---------------------------------------------------------------------------
// gate/up + SwiGLU

struct GuWave {
  __amdgpu_buffer_rsrc_t w, hh, hl;
  const uint16_t* xs;  // LDS activations [rows][stride]
  int H, I, nsteps, cpt, lane, r, kg, wave;
  int seg_lo, seg_hi, a, tpe, p0, cnt, nbn, cps, stride;
  int nsl;   // K slices per tile (1 on a whole-K pass)
  bool dbl;  // double-buffered slices
};

// Weight chunk q (tile j = q / cpt of this wave, chunk c) of the segment.
// Row-major: lane (r, kg) reads 16 B of weight row r at 64-byte K steps.
// Tiled: the tile's fragments are contiguous, so the wave reads 1 KiB per
// load (non-temporal: read once).  Chunks of tiles this wave does not have
// read out of range.
template <bool kTiled>
__device__ __forceinline__ void gu_issue(const GuWave& g, int j, int c, u32x4 (&A)[kKC]) {
  const int tile = g.seg_lo + g.wave + j * kWv;
  const int ib = tile - g.a * g.tpe;
  uint32_t row, stride;
  if (kTiled) {
    row = (uint32_t)ib * 32u * g.H + (uint32_t)g.lane * 16u;
    stride = 1024u;
  } else {
    const int wrow = g.r < 8 ? ib * 8 + g.r : g.I + ib * 8 + (g.r - 8);
    row = (uint32_t)wrow * g.H * 2u + g.kg * 16u;
    stride = 64u;
  }
  const bool live = tile < g.seg_hi;
#pragma unroll
  for (int s = 0; s < kKC; ++s) {
    const int step = c * kKC + s;
    const uint32_t off = (live && step < g.nsteps) ? row + (uint32_t)step * stride : kOutOfRange;
    A[s] = kTiled ? buf_ld128_stream(g.w, off) : buf_ld128(g.w, off);
  }
}

// MFMAs of chunk q for the pass's column blocks (NB at most), and on the
// tile's last chunk the SwiGLU epilogue.  The NB pairs of h stores are
// issued on every chunk (out of range unless they hold a result), so every
// chunk issues the same memory operations.
template <int NB>
__device__ __forceinline__ void gu_compute(const GuWave& g, const ChunkPos& at,
                                           const u32x4 (&A)[kKC], f32x4 (&acc)[NB]) {
  const int j = at.j, c = at.c;
  const int tile = g.seg_lo + g.wave + j * kWv;
  const bool have = tile < g.seg_hi;  // false: no tile of this wave in the group
  if (c == 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // column of a K step inside the staged slice, and the slice's buffer
  const int sl = at.sl;
  const int step0 = sl * g.cps * kKC;
  const uint16_t* xb = g.xs + slice_buffer(g.dbl, j * g.nsl + sl);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (have && nb < g.nbn) {
      const uint16_t* row = xb + (nb * 16 + g.r) * g.stride + g.kg * 8;
      u32x4 B[kKC];
#pragma unroll
      for (int s = 0; s < kKC; ++s) {
        const int step = c * kKC + s;
        const bool ok = step < g.nsteps;
        const u32x4 v = *reinterpret_cast<const u32x4*>(row + (ok ? (step - step0) * 32 : 0));
        B[s] = ok ? v : zero4();
      }
#pragma unroll
      for (int s = 0; s < kKC; ++s) acc[nb] = mfma_16x16x32(A[s], B[s], acc[nb]);
    }
  }
  // epilogue on the tile's last chunk: SwiGLU of the 8 (gate, up) row pairs
  // for every token column; lanes 0-31 own the results
  const bool last = have && c == g.cpt - 1;
  const int ib = tile - g.a * g.tpe;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    uint32_t off = kOutOfRange;
    u32x2 hw = {0u, 0u}, lw = {0u, 0u};
    if (last && nb < g.nbn) {
      const f32x4 v = acc[nb];
      f32x4 u;
#pragma unroll
      for (int i = 0; i < 4; ++i) u[i] = __shfl_xor(v[i], 32);
      float hv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) hv[i] = swiglu(v[i], u[i]);
      split_bf16x4(hv, hw, lw);
      const int slot = g.p0 + nb * 16 + g.r;
      if (g.lane < 32 && slot < g.cnt)
        off = ((uint32_t)slot * g.I + (uint32_t)(ib * 8 + g.kg * 4)) * 2u;
    }
    __builtin_amdgcn_raw_buffer_store_b64(hw, g.hh, off, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b64(lw, g.hl, off, 0, 0);
  }
}

// The chunk loop of one pass.  Chunk q lives in A[q % D]; the issue for
// q + D - 1 goes out before the compute of q.  Q is the same on every wave
// of a sliced pass, so every wave meets every barrier.
//   Single-buffered slices: slice c / cps is staged before chunk c of each
//     tile group: after a barrier (every wave is done with the previous
//     slice) its loads go out, then the chunk D - 1 ahead, then a wait that
//     leaves exactly that chunk's kKC loads outstanding, and a barrier.
//   Double-buffered slices: the slices of the pass (sigma = 0, 1, ... over
//     the tile groups) alternate between the two buffers.  At the first
//     step of slice sigma a wait lands sigma's staging (issued a whole
//     slice earlier) without waiting for the weight chunks issued after it,
//     then a barrier; after it every wave is done with slice sigma - 1, so
//     slice sigma + 1 is staged into that buffer at once, a whole slice of
//     steps before it is read.  The first slice, staged before the loop,
//     waits for everything.
template <bool kTiled, int D, int NB, typename Stage>
__device__ __forceinline__ void gu_run(const GuWave& g, u32x4 (&A)[D][kKC], int Q, bool sliced,
                                       Stage&& stage) {
  // vector-memory operations of one step (its weight chunk and its stores),
  // and those issued after a slice's staging before the slice is read (at
  // least one slice of steps)
  constexpr int kStepOps = kKC + 2 * NB;
  const int min_len = min(g.cps, g.cpt - (g.nsl - 1) * g.cps);
  const int after = min(63, min_len * kStepOps);
  const int n_slices = g.nsl * (Q / g.cpt);
  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  ChunkPos at, ahead;  // the chunk computed, and the chunk issued D - 1 steps ahead
  at.start(0, g.cpt, g.cps);
  ahead.start(D - 1, g.cpt, g.cps);
  for (int q = 0; q < Q; q += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int qd = q + d;
      const bool first = sliced && qd < Q && at.ks == 0;
      if (first && !g.dbl) {
        slice_barrier_before();
        stage(at.sl, 0);
        __builtin_amdgcn_sched_barrier(0);  // the slice's loads, then the weights
      }
      if (first && g.dbl) {
        const int sigma = at.j * g.nsl + at.sl;
        wait_staged_before(sigma == 0 ? 0 : after);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        if (sigma + 1 < n_slices) {
          stage(at.sl + 1 < g.nsl ? at.sl + 1 : 0, slice_buffer(true, sigma + 1));
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      gu_issue<kTiled>(g, ahead.j, ahead.c, A[(d + D - 1) % D]);
      if (first && !g.dbl) slice_barrier_after<kKC>();
      if (d == 0 || qd < Q) gu_compute<NB>(g, at, A[d], acc);
      at.next(g.cpt, g.cps);
      ahead.next(g.cpt, g.cps);
    }
  }
}

// The dispatch plan of a gate/up launch that builds it itself (kPlan): the
// selected ids it reads, and the arrays block 0 writes for the launches after
// it (down projection, combine) and for the caller.
struct PlanBuild {
  const int* ids;
  int *counts, *offsets, *perm, *active, *n_active;
};

// LDS words of such a plan, beside the staging area: n_active, counts[m],
// offsets[m + 1], active[m] and perm[n_pairs].
constexpr int kPlanInts = 2464;
__host__ __device__ constexpr int plan_ints(int m, int n_pairs) { return 3 * m + 2 + n_pairs; }

// Every block builds the plan of the batch in LDS from its n_pairs selected
// ids (n_pairs <= 2 kBlk, m <= kBlk): the plan the dispatch kernel writes,
// value for value, in four barriers.  ids_r holds this thread's ids (pairs
// tid and tid + kBlk), loaded before the block's first weight chunks so that
// waiting for them does not wait for those.  Pair p belongs to run
// cw = p / 64 (a wave's 64 pairs); within a run, ballots match equal ids
// (the pair's rank among them), and the run's count of each id goes to
// LDS.  The histogram is the sum of the runs' counts; offsets and the active
// list come from one block scan over the experts (expert e on thread e); a
// pair's place in perm is then its expert's offset, plus its expert's
// counts in the earlier runs, plus its rank: pairs in pair order within
// each expert.  The runs' counts live in the staging area, which nothing
// else uses yet.  Block 0 then writes the plan to memory.  Every thread of
// the block calls it.
__device__ void build_plan(const int (&ids_r)[2], int n_pairs, int m, uint16_t* xs, int* plan_s,
                           const PlanBuild& pb) {
  constexpr int kRuns = 2 * kWv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int* counts = plan_s + 1;
  int* offsets = counts + m;
  int* active = offsets + m + 1;
  int* perm = active + m;
  uint8_t* run_cnt = reinterpret_cast<uint8_t*>(xs);                   // [kRuns][m]
  uint32_t* wsum = reinterpret_cast<uint32_t*>(xs) + kRuns * m / 4;     // [2][kWv]
  int* bad = reinterpret_cast<int*>(wsum + 2 * kWv);
  for (int i = tid; i < kRuns * m / 4; i += kBlk) reinterpret_cast<uint32_t*>(run_cnt)[i] = 0u;
  if (tid < m) counts[tid] = 0;
  if (tid == 0) *bad = 0;
  __syncthreads();

  // runs: rank among equal ids, the run's count per id, the histogram
  const int nbits = id_bits(m);
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  int rank[2], key[2];
  bool ok[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int p = tid + i * kBlk;
    const int e = ids_r[i];
    ok[i] = p < n_pairs && e >= 0 && e < m;
    if (p < n_pairs && !ok[i]) *bad = 1;
    key[i] = ok[i] ? e : 0;
    const uint64_t peers = match_peers(key[i], ok[i], nbits);
    rank[i] = __popcll(peers & lt_mask);
    if (ok[i] && rank[i] == 0) {
      const int n = __popcll(peers);
      run_cnt[(i * kWv + wave) * m + key[i]] = static_cast<uint8_t>(n);
      atomicAdd(&counts[key[i]], n);
    }
  }
  __syncthreads();

  if (*bad) {  // an id outside [0, m): the flagged plan
    for (int e = tid; e <= m; e += kBlk) {
      if (e < m) counts[e] = 0;
      offsets[e] = 0;
    }
    for (int p = tid; p < n_pairs; p += kBlk) perm[p] = p;
    if (tid == 0) plan_s[0] = -1;
  } else {
    // offsets and the active list: one scan over the experts
    const uint32_t c = tid < m ? (uint32_t)counts[tid] : 0u, a = c > 0 ? 1u : 0u;
    const uint32_t ic = wave_inclusive_scan_u32(c), ia = wave_inclusive_scan_u32(a);
    if (lane == 63) {
      wsum[wave] = ic;
      wsum[kWv + wave] = ia;
    }
    __syncthreads();
    uint32_t bc = 0, ba = 0, tc = 0, ta = 0;
#pragma unroll
    for (int w = 0; w < kWv; ++w) {
      const uint32_t sc = wsum[w], sa = wsum[kWv + w];
      bc += w < wave ? sc : 0u;
      ba += w < wave ? sa : 0u;
      tc += sc;
      ta += sa;
    }
    if (tid < m) {
      offsets[tid] = (int)(bc + ic - c);
      if (a) active[ba + ia - 1] = tid;
    }
    if (tid == 0) {
      offsets[m] = (int)tc;
      plan_s[0] = (int)ta;
    }
    __syncthreads();
    // each pair's place: its expert's offset, its expert's pairs in the
    // earlier runs, its rank in its run
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (!ok[i]) continue;
      const int run = i * kWv + wave;
      int pos = offsets[key[i]] + rank[i];
      for (int r = 0; r < run; ++r) pos += run_cnt[r * m + key[i]];
      perm[pos] = tid + i * kBlk;
    }
  }
  __syncthreads();
  if (blockIdx.x == 0) {
    const int na = plan_s[0];
    for (int e = tid; e <= m; e += kBlk) {
      if (e < m) pb.counts[e] = counts[e];
      pb.offsets[e] = offsets[e];
    }
    for (int p = tid; p < n_pairs; p += kBlk) pb.perm[p] = perm[p];
    for (int a = tid; a < na; a += kBlk) pb.active[a] = active[a];
    if (tid == 0) *pb.n_active = na;
  }
}

// kSpeculate: guess n_active == m and issue the first weight chunks before
// n_active arrives (a wrong guess redoes the first segment).
// kNbMax: column blocks of the largest pass (16 kNbMax tokens): 2 for
// batches of up to 64 tokens, 8 for larger ones.
// kPlan: the plan arguments are unused; the block builds the plan from
// pb.ids instead (m <= kBlk, n_pairs <= 2 kBlk, plan_ints(m, n_pairs) <=
// kPlanInts), and block 0 writes it to pb's arrays.
template <bool kTiled, bool kSpeculate, int kNbMax, int kDepth, bool kPlan>
__global__ __launch_bounds__(kBlk, 1) void gate_up_wave_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w13,
    const int* __restrict__ counts_in, const int* __restrict__ offsets_in,
    const int* __restrict__ perm_in, const int* __restrict__ active_in,
    const int* __restrict__ n_active_p, uint16_t* __restrict__ h_hi,
    uint16_t* __restrict__ h_lo, int H, int I, int m, int k, int n_pairs, PlanBuild pb) {
  constexpr int kPmax = 16 * kNbMax;
  // the wide variant (batches of more than 64 tokens) can give an expert
  // more pairs than a whole-K pass holds: the cost-weighted walk is
  // compiled in
  constexpr bool kBalance = kNbMax > 2;
  static_assert(!(kPlan && kBalance), "the plan is built by the 32-token variants only");
  __shared__ __attribute__((aligned(16))) uint16_t xs[kStage];
  __shared__ int pid[kPmax];
  __shared__ int wp[kBalance ? kMaxExperts + 1 : 1];
  __shared__ uint32_t scan[34];
  __shared__ int verdict[kWv];
  __shared__ int plan_s[kPlan ? kPlanInts : 1];
  const int* counts = kPlan ? plan_s + 1 : counts_in;
  const int* offsets = kPlan ? plan_s + 1 + m : offsets_in;
  const int* active = kPlan ? plan_s + 2 + 2 * m : active_in;
  const int* perm = kPlan ? plan_s + 2 + 3 * m : perm_in;
  const int tpe = I / 8;
  int ids_r[2] = {0, 0};
  if constexpr (kPlan) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int p = (int)threadIdx.x + i * kBlk;
      ids_r[i] = p < n_pairs ? pb.ids[p] : 0;
    }
  }
  int n_act = kPlan ? 0 : *n_active_p;
  const auto xr = make_rsrc(x, 2u * (uint32_t)(n_pairs / k) * (uint32_t)H);

  GuWave g;
  g.xs = xs;
  g.H = H;
  g.I = I;
  g.nsteps = H / 32;
  g.cpt = (g.nsteps + kKC - 1) / kKC;
  g.lane = threadIdx.x & 63;
  g.wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  g.r = g.lane & 15;
  g.kg = g.lane >> 4;
  g.tpe = tpe;

  u32x4 A[kDepth][kKC];
  // the segment's first chunks d0 .. kDepth - 2 (tile 0 of this wave: the
  // same chunks in a whole-K and a sliced pass)
  auto issue_first = [&](int d0) {
#pragma unroll
    for (int d = 0; d < kDepth - 1; ++d) {
      if (d >= d0) {
        ChunkPos h;
        h.start(d, g.cpt, g.cpt);
        gu_issue<kTiled>(g, h.j, h.c, A[d]);
      }
    }
  };
  // weight resource of the segment's expert and its first chunks up to
  // d_end (all kDepth - 1 of them by default)
  auto begin_segment = [&](const Segment& sg, int d_end = kDepth - 1) {
    g.seg_lo = sg.lo;
    g.seg_hi = sg.hi;
    g.a = sg.a;
    g.w = make_rsrc(w13 + (size_t)sg.e * 2 * I * H, sg.e_ok ? 4u * (uint32_t)I * (uint32_t)H : 0u);
#pragma unroll
    for (int d = 0; d < kDepth - 1; ++d) {
      if (d < d_end) {
        ChunkPos h;
        h.start(d, g.cpt, g.cpt);
        gu_issue<kTiled>(g, h.j, h.c, A[d]);
      }
    }
  };

  // Speculate a fully active pool (n_active == m, the usual saturated decode
  // batch): the block's tile range and its first expert then follow from m
  // alone, so that segment's plan loads and weight chunks go out together
  // with the n_active load.  A wrong guess redoes the first segment.
  // (Without kSpeculate the first segment waits for n_active instead.)
  const int light = whole_k_tokens(kPmax, H, 1);
  const PairCounts pc = kBalance ? load_pair_counts(offsets, m) : PairCounts{0, 0, 0};
  int r_lo = 0, r_hi = 0;
  Segment sg;
  // A block that builds the plan issues only the first guessed chunk before
  // it: a wave that issues more at the kernel's start, when every compute
  // unit does, stalls on the issue (the memory system holds as many
  // requests as it can) and cannot build the plan meanwhile; the rest of
  // the chunks follow the build.
  constexpr int kEarly = kPlan ? 1 : kDepth - 1;
  if constexpr (kSpeculate) {
    block_range(m * tpe, &r_lo, &r_hi);
    // (a plan built here is not there yet: its count and offset are read
    // once it is)
    sg = next_segment(r_lo, r_hi, tpe, active, counts_in, offsets_in, m, true, !kPlan);
    begin_segment(sg, kEarly);
  }
  if constexpr (kPlan) {
    build_plan(ids_r, n_pairs, m, xs, plan_s, pb);
    n_act = plan_s[0];
    if (kSpeculate) {
      sg.cnt = counts[sg.e];
      sg.base = offsets[sg.e];
      issue_first(kEarly);
    }
  }
  if (n_act <= 0 || n_act > m) return;  // an invalid plan: no work
  const bool all = n_act == m;
  // With kBalance, whether some expert needs a sliced pass or several passes
  // is decided once, at the first barrier of the block's first pass (its
  // pair-id loads are already out then); a block without such a barrier
  // decides it on a barrier of its own.  If one does, the block switches to
  // its run of the cost-weighted walk.
  bool checked = !kBalance, weighted = false;
  int w_hi = 0;
  auto go_weighted = [&]() {
    weighted = true;
    weighted_work(n_act, tpe, active, counts, offsets, m, n_pairs, kPmax, H, g.cpt, 1, wp, scan);
    block_range(wp[n_act], &r_lo, &w_hi);
    if (r_lo >= w_hi) return false;
    sg = weighted_segment(r_lo, w_hi, n_act, wp, tpe, active, counts, offsets, m);
    if (sg.lo >= sg.hi) return false;
    begin_segment(sg);
    return true;
  };
  if (!kSpeculate || !all) {
    block_range(n_act * tpe, &r_lo, &r_hi);
    if (r_lo < r_hi) {
      sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, all);
      begin_segment(sg);
    }
  }
  if (r_lo >= r_hi) {
    if (!kBalance) return;
    checked = true;
    if (!some_expert_is_heavy(pc, light, verdict) || !go_weighted()) return;
  }

  for (;;) {
    finish_segment(sg, n_pairs);
    if (!checked && sg.cnt == 0) {  // no pass (hence no barrier) in this segment
      checked = true;
      if (some_expert_is_heavy(pc, light, verdict)) {
        if (!go_weighted()) return;
        continue;
      }
    }
    g.cnt = sg.cnt;
    const uint32_t hbytes = 2u * (uint32_t)sg.cnt * (uint32_t)I;
    g.hh = make_rsrc(h_hi + (size_t)sg.base * I, hbytes);
    g.hl = make_rsrc(h_lo + (size_t)sg.base * I, hbytes);
    const int per_pass = sg.cnt > 0 ? pass_tokens(sg.cnt, kPmax) : 1;
    // this wave's tiles of the segment (seg_lo + wave, + kWv, ...), and the
    // tile groups every wave walks on a sliced pass
    const int seg_n = sg.hi - sg.lo;
    const int ntw = seg_n > g.wave ? (seg_n - g.wave + kWv - 1) / kWv : 0;
    const int ngroups = (seg_n + kWv - 1) / kWv;
    bool restart = false;
    for (int p0 = 0; p0 < sg.cnt; p0 += per_pass) {
      const PassShape ps = pass_shape(min(per_pass, sg.cnt - p0), H, g.cpt, 1);
      g.p0 = p0;
      g.nbn = ps.nbn;
      g.cps = ps.cps;
      g.stride = ps.stride;
      g.nsl = (g.cpt + ps.cps - 1) / ps.cps;
      g.dbl = ps.dbl;
      const int Q = (ps.sliced ? ngroups : ntw) * g.cpt;
      if (p0 > 0) {
#pragma unroll
        for (int d = 0; d < kDepth - 1; ++d) {
      ChunkPos h;
      h.start(d, g.cpt, g.cpt);
      gu_issue<kTiled>(g, h.j, h.c, A[d]);
    }
      }
      // the pass's pair ids (loaded before the barrier that waits for the
      // previous pass's readers of pid and xs)
      int pv = -1;
      if ((int)threadIdx.x < ps.n) {
        const int p = perm[sg.base + p0 + (int)threadIdx.x];
        pv = (p >= 0 && p < n_pairs) ? p : -1;
      }
      if (!checked) post_heavy_verdict(pc, light, verdict);
      __syncthreads();
      if (!checked) {
        checked = true;
        if (read_heavy_verdict(verdict)) {
          restart = true;
          break;
        }
      }
      if ((int)threadIdx.x < kPmax) pid[threadIdx.x] = pv;
      __syncthreads();
      // K slice `sl` (all of K on a whole-K pass) of the pass's token rows
      // of x, straight into the LDS buffer at element `boff`: wave w stages
      // rows w, w + kWv, ... (rows without a pair read zeros)
      auto stage = [&](int sl, int boff) {
        const int col0 = sl * g.cps * kChunkCols;
        const int bytes = 2 * min(g.cps * kChunkCols, H - col0);
        for (int tok = g.wave; tok < g.nbn * 16; tok += kWv) {
          const int p = pid[tok];
          stage_row(xr, p >= 0 ? ((uint32_t)(p / k) * (uint32_t)H + (uint32_t)col0) * 2u
                               : kOutOfRange,
                    xs + boff + tok * g.stride, bytes, g.lane);
        }
      };
      if (!ps.sliced) {
        stage(0, 0);
        __builtin_amdgcn_s_waitcnt(kVmcntZero);
        __syncthreads();
      } else if (ps.dbl) {
        stage(0, 0);  // landed by the wait at the loop's first step
      }
      if (kNbMax == 2 || ps.nbn <= 2)
        gu_run<kTiled, kDepth, 2>(g, A, Q, ps.sliced, stage);
      else
        gu_run<kTiled, kDepth, kNbMax>(g, A, Q, ps.sliced, stage);
    }
    if (restart) {
      if (!go_weighted()) return;
      continue;
    }
    if (weighted) {
      if (sg.w_end >= w_hi) break;
      sg = weighted_segment(sg.w_end, w_hi, n_act, wp, tpe, active, counts, offsets, m);
      if (sg.lo >= sg.hi) break;
    } else {
      if (sg.hi >= r_hi) break;
      sg = next_segment(sg.hi, r_hi, tpe, active, counts, offsets, m, all);
    }
    begin_segment(sg);
  }
}

// ---------------------------------------------------------------------------
// down projection

struct DnWave {
  __amdgpu_buffer_rsrc_t w, y;
  const uint16_t* hs;  // LDS h hi rows [rows][stride], then the lo rows
  const int* pid;      // LDS pair ids of the pass
  int H, I, nsteps, cpt, lane, r, kg, wave;
  int seg_lo, seg_hi, a, tpe, nbn, cps, stride, lo_off;
  int nsl;   // K slices per tile (1 on a whole-K pass)
  bool dbl;  // double-buffered slices
};

template <bool kTiled>
__device__ __forceinline__ void dn_issue(const DnWave& g, int j, int c, u32x4 (&A)[kKC]) {
  const int tile = g.seg_lo + g.wave + j * kWv;
  const int ob = tile - g.a * g.tpe;
  const int o = ob * 16 + g.r;
  uint32_t row, stride;
  if (kTiled) {
    row = (uint32_t)ob * 32u * g.I + (uint32_t)g.lane * 16u;
    stride = 1024u;
  } else {
    row = (uint32_t)o * g.I * 2u + g.kg * 16u;
    stride = 64u;
  }
  const bool live = tile < g.seg_hi;
#pragma unroll
  for (int s = 0; s < kKC; ++s) {
    const int step = c * kKC + s;
    const bool ok = live && step < g.nsteps && o < g.H;
    const uint32_t off = ok ? row + (uint32_t)step * stride : kOutOfRange;
    A[s] = kTiled ? buf_ld128_stream(g.w, off) : buf_ld128(g.w, off);
  }
}

template <int NB>
__device__ __forceinline__ void dn_compute(const DnWave& g, const ChunkPos& at,
                                           const u32x4 (&A)[kKC], f32x4 (&acc)[NB]) {
  const int j = at.j, c = at.c;
  const int tile = g.seg_lo + g.wave + j * kWv;
  const bool have = tile < g.seg_hi;
  if (c == 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int sl = at.sl;
  const int step0 = sl * g.cps * kKC;
  const uint16_t* hb = g.hs + slice_buffer(g.dbl, j * g.nsl + sl);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (have && nb < g.nbn) {
      const uint16_t* row = hb + (nb * 16 + g.r) * g.stride + g.kg * 8;
#pragma unroll
      for (int s = 0; s < kKC; ++s) {
        const int step = c * kKC + s;
        const bool ok = step < g.nsteps;
        const int col = ok ? (step - step0) * 32 : 0;
        const u32x4 bh = *reinterpret_cast<const u32x4*>(row + col);
        const u32x4 bl = *reinterpret_cast<const u32x4*>(row + g.lo_off + col);
        acc[nb] = mfma_16x16x32(A[s], ok ? bh : zero4(), acc[nb]);
        acc[nb] = mfma_16x16x32(A[s], ok ? bl : zero4(), acc[nb]);
      }
    }
  }
  const bool last = have && c == g.cpt - 1;
  const int o = (tile - g.a * g.tpe) * 16 + g.kg * 4;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    uint32_t off = kOutOfRange;
    if (last && nb < g.nbn) {
      const int p = g.pid[nb * 16 + g.r];
      if (p >= 0 && o < g.H) off = ((uint32_t)p * g.H + (uint32_t)o) * 4u;
    }
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[nb]), g.y, off, 0, 0);
  }
}

// As gu_run; a down step stores one y fragment per column block.
template <bool kTiled, int D, int NB, typename Stage>
__device__ __forceinline__ void dn_run(const DnWave& g, u32x4 (&A)[D][kKC], int Q, bool sliced,
                                       Stage&& stage) {
  constexpr int kStepOps = kKC + NB;
  const int min_len = min(g.cps, g.cpt - (g.nsl - 1) * g.cps);
  const int after = min(63, min_len * kStepOps);
  const int n_slices = g.nsl * (Q / g.cpt);
  f32x4 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  ChunkPos at, ahead;  // the chunk computed, and the chunk issued D - 1 steps ahead
  at.start(0, g.cpt, g.cps);
  ahead.start(D - 1, g.cpt, g.cps);
  for (int q = 0; q < Q; q += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int qd = q + d;
      const bool first = sliced && qd < Q && at.ks == 0;
      if (first && !g.dbl) {
        slice_barrier_before();
        stage(at.sl, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (first && g.dbl) {
        const int sigma = at.j * g.nsl + at.sl;
        wait_staged_before(sigma == 0 ? 0 : after);
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        if (sigma + 1 < n_slices) {
          stage(at.sl + 1 < g.nsl ? at.sl + 1 : 0, slice_buffer(true, sigma + 1));
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      dn_issue<kTiled>(g, ahead.j, ahead.c, A[(d + D - 1) % D]);
      if (first && !g.dbl) slice_barrier_after<kKC>();
      if (d == 0 || qd < Q) dn_compute<NB>(g, at, A[d], acc);
      at.next(g.cpt, g.cps);
      ahead.next(g.cpt, g.cps);
    }
  }
}

template <bool kTiled, bool kSpeculate, int kNbMax, int kDepth>
__global__ __launch_bounds__(kBlk, 1) void down_wave_kernel(
    const uint16_t* __restrict__ h_hi, const uint16_t* __restrict__ h_lo,
    const uint16_t* __restrict__ w2, const int* __restrict__ counts,
    const int* __restrict__ offsets, const int* __restrict__ perm,
    const int* __restrict__ active, const int* __restrict__ n_active_p, float* __restrict__ y,
    int H, int I, int m, int n_pairs) {
  constexpr int kPmax = 16 * kNbMax;
  constexpr bool kBalance = kNbMax > 2;  // as in gate_up_wave_kernel
  __shared__ __attribute__((aligned(16))) uint16_t hs[kStage];
  __shared__ int pid[kPmax];
  __shared__ int wp[kBalance ? kMaxExperts + 1 : 1];
  __shared__ uint32_t scan[34];
  __shared__ int verdict[kWv];
  const int tpe = (H + 15) / 16;
  const int n_act = *n_active_p;

  DnWave g;
  g.hs = hs;
  g.pid = pid;
  g.y = make_rsrc(y, 4u * (uint32_t)n_pairs * (uint32_t)H);
  g.H = H;
  g.I = I;
  g.nsteps = I / 32;
  g.cpt = (g.nsteps + kKC - 1) / kKC;
  g.lane = threadIdx.x & 63;
  g.wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  g.r = g.lane & 15;
  g.kg = g.lane >> 4;
  g.tpe = tpe;
  const uint32_t hbytes = 2u * (uint32_t)n_pairs * (uint32_t)I;
  const auto hhr = make_rsrc(h_hi, hbytes);
  const auto hlr = make_rsrc(h_lo, hbytes);

  u32x4 A[kDepth][kKC];
  auto begin_segment = [&](const Segment& sg) {
    g.seg_lo = sg.lo;
    g.seg_hi = sg.hi;
    g.a = sg.a;
    g.w = make_rsrc(w2 + (size_t)sg.e * H * I, sg.e_ok ? 2u * (uint32_t)H * (uint32_t)I : 0u);
#pragma unroll
    for (int d = 0; d < kDepth - 1; ++d) {
      ChunkPos h;
      h.start(d, g.cpt, g.cpt);
      dn_issue<kTiled>(g, h.j, h.c, A[d]);
    }
  };

  // Speculate a fully active pool, and walk by cost when some expert needs
  // a sliced pass or several passes, as in gate_up_wave_kernel.
  const int light = whole_k_tokens(kPmax, I, 2);
  const PairCounts pc = kBalance ? load_pair_counts(offsets, m) : PairCounts{0, 0, 0};
  int r_lo = 0, r_hi = 0;
  Segment sg;
  if constexpr (kSpeculate) {
    block_range(m * tpe, &r_lo, &r_hi);
    sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, true);
    begin_segment(sg);
  }
  if (n_act <= 0 || n_act > m) return;  // an invalid plan: no work
  const bool all = n_act == m;
  bool checked = !kBalance, weighted = false;
  int w_hi = 0;
  auto go_weighted = [&]() {
    weighted = true;
    weighted_work(n_act, tpe, active, counts, offsets, m, n_pairs, kPmax, I, g.cpt, 2, wp, scan);
    block_range(wp[n_act], &r_lo, &w_hi);
    if (r_lo >= w_hi) return false;
    sg = weighted_segment(r_lo, w_hi, n_act, wp, tpe, active, counts, offsets, m);
    if (sg.lo >= sg.hi) return false;
    begin_segment(sg);
    return true;
  };
  if (!kSpeculate || !all) {
    block_range(n_act * tpe, &r_lo, &r_hi);
    if (r_lo < r_hi) {
      sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, all);
      begin_segment(sg);
    }
  }
  if (r_lo >= r_hi) {
    if (!kBalance) return;
    checked = true;
    if (!some_expert_is_heavy(pc, light, verdict) || !go_weighted()) return;
  }

  for (;;) {
    finish_segment(sg, n_pairs);
    if (!checked && sg.cnt == 0) {  // no pass (hence no barrier) in this segment
      checked = true;
      if (some_expert_is_heavy(pc, light, verdict)) {
        if (!go_weighted()) return;
        continue;
      }
    }
    const int per_pass = sg.cnt > 0 ? pass_tokens(sg.cnt, kPmax) : 1;
    const int seg_n = sg.hi - sg.lo;
    const int ntw = seg_n > g.wave ? (seg_n - g.wave + kWv - 1) / kWv : 0;
    const int ngroups = (seg_n + kWv - 1) / kWv;
    bool restart = false;
    for (int p0 = 0; p0 < sg.cnt; p0 += per_pass) {
      const PassShape ps = pass_shape(min(per_pass, sg.cnt - p0), I, g.cpt, 2);
      g.nbn = ps.nbn;
      g.cps = ps.cps;
      g.stride = ps.stride;
      g.lo_off = ps.nbn * 16 * ps.stride;
      g.nsl = (g.cpt + ps.cps - 1) / ps.cps;
      g.dbl = ps.dbl;
      const int Q = (ps.sliced ? ngroups : ntw) * g.cpt;
      if (p0 > 0) {
#pragma unroll
        for (int d = 0; d < kDepth - 1; ++d) {
      ChunkPos h;
      h.start(d, g.cpt, g.cpt);
      dn_issue<kTiled>(g, h.j, h.c, A[d]);
    }
      }
      // the pass's pair ids (for the y rows); its h rows are contiguous in
      // dispatch-slot order
      int pv = -1;
      if ((int)threadIdx.x < ps.n) {
        const int p = perm[sg.base + p0 + (int)threadIdx.x];
        pv = (p >= 0 && p < n_pairs) ? p : -1;
      }
      if (!checked) post_heavy_verdict(pc, light, verdict);
      __syncthreads();  // the previous pass's readers of hs and pid are done
      if (!checked) {
        checked = true;
        if (read_heavy_verdict(verdict)) {
          restart = true;
          break;
        }
      }
      if ((int)threadIdx.x < kPmax) pid[threadIdx.x] = pv;
      // K slice `sl` of the pass's h rows (hi, then lo), straight into the
      // LDS buffer at element `boff`: wave w stages rows w, w + kWv, ... of
      // both halves
      auto stage = [&](int sl, int boff) {
        const int col0 = sl * g.cps * kChunkCols;
        const int bytes = 2 * min(g.cps * kChunkCols, I - col0);
        for (int tok = g.wave; tok < g.nbn * 16; tok += kWv) {
          const uint32_t src =
              tok < ps.n ? ((uint32_t)(sg.base + p0 + tok) * (uint32_t)I + (uint32_t)col0) * 2u
                         : kOutOfRange;
          stage_row(hhr, src, hs + boff + tok * g.stride, bytes, g.lane);
          stage_row(hlr, src, hs + boff + g.lo_off + tok * g.stride, bytes, g.lane);
        }
      };
      if (!ps.sliced) {
        stage(0, 0);
        __builtin_amdgcn_s_waitcnt(kVmcntZero);
      } else if (ps.dbl) {
        stage(0, 0);  // landed by the wait at the loop's first step
      }
      __syncthreads();  // pid (and a whole-K pass's rows) visible to every wave
      if (kNbMax == 2 || ps.nbn <= 2)
        dn_run<kTiled, kDepth, 2>(g, A, Q, ps.sliced, stage);
      else
        dn_run<kTiled, kDepth, kNbMax>(g, A, Q, ps.sliced, stage);
    }
    if (restart) {
      if (!go_weighted()) return;
      continue;
    }
    if (weighted) {
      if (sg.w_end >= w_hi) break;
      sg = weighted_segment(sg.w_end, w_hi, n_act, wp, tpe, active, counts, offsets, m);
      if (sg.lo >= sg.hi) break;
    } else {
      if (sg.hi >= r_hi) break;
      sg = next_segment(sg.hi, r_hi, tpe, active, counts, offsets, m, all);
    }
    begin_segment(sg);
  }
}

// Tiled ("fragment-major") expert layout.  Gate/up: tile ib of an expert
// holds the 16 A rows (gate rows 8ib..8ib+7, then up rows I+8ib..) over all
// of H as H/32 consecutive 1 KiB fragments; fragment s stores, for lane l =
// 0..63, the 8 bf16 of row (l % 16), columns 32s + 8(l / 16) .. +7.  Down:
// tile ob holds output rows 16ob..16ob+15 over I the same way.  One thread
// moves one 16-byte fragment piece.
__global__ __launch_bounds__(256) void pack_w13_kernel(const uint16_t* __restrict__ src,
                                                      uint16_t* __restrict__ dst, int H, int I,
                                                      size_t n_frag) {
  const size_t f = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (f >= n_frag) return;
  const size_t per_e = (size_t)2 * I * H / 8, per_tile = (size_t)2 * H;
  const size_t e = f / per_e, rem = f - e * per_e;
  const int ib = (int)(rem / per_tile), rem2 = (int)(rem - (size_t)ib * per_tile);
  const int s = rem2 >> 6, l = rem2 & 63;
  const int rr = l & 15;
  const int row = rr < 8 ? ib * 8 + rr : I + ib * 8 + (rr - 8);
  const int col = s * 32 + (l >> 4) * 8;
  *reinterpret_cast<u32x4*>(dst + f * 8) =
      ld128(src + e * 2 * I * H + (size_t)row * H + col);
}

__global__ __launch_bounds__(256) void pack_w2_kernel(const uint16_t* __restrict__ src,
                                                     uint16_t* __restrict__ dst, int H, int I,
                                                     size_t n_frag) {
  const size_t f = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (f >= n_frag) return;
  const size_t per_e = (size_t)H * I / 8, per_tile = (size_t)2 * I;
  const size_t e = f / per_e, rem = f - e * per_e;
  const int ob = (int)(rem / per_tile), rem2 = (int)(rem - (size_t)ob * per_tile);
  const int s = rem2 >> 6, l = rem2 & 63;
  const int row = ob * 16 + (l & 15);
  const int col = s * 32 + (l >> 4) * 8;
  *reinterpret_cast<u32x4*>(dst + f * 8) = ld128(src + e * H * I + (size_t)row * I + col);
}

// Variant of a launch: the largest pass (column blocks) and the weight
// pipeline depth.  An expert receives at most one pair per token of a routed
// batch, so passes of T tokens stream every expert once.  Batches of up to
// 64 tokens take passes of 32 (2 column blocks, three chunks in flight): a
// 64-token variant needs every register and measured 2.6 us slower on the
// 64-token decode layer over 64 experts, and 10 us over 128, than the
// 32-token one, whose only extra cost is a second pass over an expert that
// receives more than 32 of the batch's tokens (heavy skew; near-uniform
// routing gives at most about 20 at 64 tokens).  Larger batches take the
// most that fit the registers with no spill -- 8 column blocks (128 tokens)
// for gate/up with two chunks in flight, 6 (96 tokens) for down with three
// -- and the cost-weighted walk.  Guessing a fully active pool pays when
// the expected number of idle experts, m (1 - k/m)^T, is well below one.
int gate_up_column_blocks(int T) { return T <= 2 * kNT ? 2 : 8; }
int down_column_blocks(int T) { return T <= 2 * kNT ? 2 : 6; }

bool speculate_full_pool(int T, int m, int k) {
  const double idle = m * std::pow(1.0 - (double)k / m, (double)T);
  return idle < 0.25;
}

int stream_grid() {
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 256;
  return cus;
}

}  // namespace

bool wave_stream_supported(int T, int H, int I, int k) {
  return H % 32 == 0 && I % 32 == 0 && H <= kMaxStreamH && I <= kMaxStreamI &&
         4 * (int64_t)T * k * H < ((int64_t)1 << 31);
}

hipError_t launch_gate_up_wave(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                               const int* counts, const int* offsets, const int* perm,
                               const int* active, const int* n_active, int H, int I, int m, int k,
                               uint16_t* h_hi, uint16_t* h_lo, hipStream_t stream) {
  const int nb = gate_up_column_blocks(T);
  const bool sp = speculate_full_pool(T, m, k);
#define SW_GU(TI, SP, NB, D)                                                                   \
  gate_up_wave_kernel<TI, SP, NB, D, false><<<stream_grid(), kBlk, 0, stream>>>(                \
      x, w13, counts, offsets, perm, active, n_active, h_hi, h_lo, H, I, m, k, T * k,           \
      PlanBuild{})
  if (nb == 2) {
    if (sp) {
      if (tiled) SW_GU(true, true, 2, 3); else SW_GU(false, true, 2, 3);
    } else {
      if (tiled) SW_GU(true, false, 2, 3); else SW_GU(false, false, 2, 3);
    }
  } else if (sp) {
    if (tiled) SW_GU(true, true, 8, 2); else SW_GU(false, true, 8, 2);
  } else {
    if (tiled) SW_GU(true, false, 8, 2); else SW_GU(false, false, 8, 2);
  }
#undef SW_GU
  return hipGetLastError();
}

bool wave_plan_supported(int T, int H, int I, int m, int k, bool tiled) {
  return gate_up_kernels(T, H, I, m, k, tiled) == Kernels::kWave && gate_up_column_blocks(T) == 2 &&
         m <= kBlk && T * k <= 2 * kBlk && plan_ints(m, T * k) <= kPlanInts;
}

hipError_t launch_gate_up_wave_plan(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                    const int* topk_ids, int* counts, int* offsets, int* perm,
                                    int* active, int* n_active, int H, int I, int m, int k,
                                    uint16_t* h_hi, uint16_t* h_lo, hipStream_t stream) {
  const PlanBuild pb{topk_ids, counts, offsets, perm, active, n_active};
  const bool sp = speculate_full_pool(T, m, k);
#define SW_GP(TI, SP)                                                                          \
  gate_up_wave_kernel<TI, SP, 2, 3, true><<<stream_grid(), kBlk, 0, stream>>>(                  \
      x, w13, nullptr, nullptr, nullptr, nullptr, nullptr, h_hi, h_lo, H, I, m, k, T * k, pb)
  if (sp) {
    if (tiled) SW_GP(true, true); else SW_GP(false, true);
  } else {
    if (tiled) SW_GP(true, false); else SW_GP(false, false);
  }
#undef SW_GP
  return hipGetLastError();
}

hipError_t launch_down_wave(int T, const uint16_t* w2, bool tiled, const int* counts,
                            const int* offsets, const int* perm, const int* active,
                            const int* n_active, int H, int I, int m, int k, const uint16_t* h_hi,
                            const uint16_t* h_lo, float* y, hipStream_t stream) {
  const int nb = down_column_blocks(T);
  const bool sp = speculate_full_pool(T, m, k);
#define SW_DN(TI, SP, NB)                                                                      \
  down_wave_kernel<TI, SP, NB, 3><<<stream_grid(), kBlk, 0, stream>>>(                          \
      h_hi, h_lo, w2, counts, offsets, perm, active, n_active, y, H, I, m, T * k)
  if (nb == 2) {
    if (sp) {
      if (tiled) SW_DN(true, true, 2); else SW_DN(false, true, 2);
    } else {
      if (tiled) SW_DN(true, false, 2); else SW_DN(false, false, 2);
    }
  } else if (sp) {
    if (tiled) SW_DN(true, true, 6); else SW_DN(false, true, 6);
  } else {
    if (tiled) SW_DN(true, false, 6); else SW_DN(false, false, 6);
  }
#undef SW_DN
  return hipGetLastError();
}

hipError_t launch_pack_experts(const uint16_t* w13, const uint16_t* w2, uint16_t* w13_t,
                               uint16_t* w2_t, int H, int I, int m, hipStream_t stream) {
  if (w13 != nullptr) {
    const size_t n = (size_t)m * 2 * I * H / 8;
    pack_w13_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(w13, w13_t, H, I, n);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  if (w2 != nullptr) {
    const size_t n = (size_t)m * H * I / 8;
    pack_w2_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(w2, w2_t, H, I, n);
  }
  return hipGetLastError();
}

}  // namespace sw
