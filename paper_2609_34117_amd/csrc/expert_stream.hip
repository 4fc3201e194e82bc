// Wave-streaming expert FFN kernels for gfx950: the decode fast path of the
// MoE layer (Section 2.1: a decode step reads every distinct expert chosen
// across the batch, so the step is bound by streaming expert weights).
//
// Design:
//   - A persistent grid of one 8-wave block per compute unit.  The tiles of
//     all active experts form one list; block b owns the contiguous,
//     equal-sized range b*per .. (b+1)*per of it, which crosses at most a few
//     expert boundaries ("segments").  When some expert has more tokens than
//     one pass holds, the list is of (expert, pass, tile) work items instead,
//     so every block still gets the same number of tile passes.
//   - Per segment, the block stages the expert's token activations (gate/up:
//     x rows; down: h hi/lo rows) in LDS once, up to 32 tokens per pass.
//   - Each wave then owns whole tiles (16 weight rows over the full K) and
//     streams them as 8 KiB chunks through a kDepth-deep register pipeline:
//     the kDepth - 1 chunks ahead are always in flight.  The B operand
//     (tokens) comes from LDS, so waiting for activations never waits on
//     weights, and there is no cross-wave reduction and no barrier inside a
//     segment.  The first chunks of a segment are issued as soon as its
//     expert id is known, before the activation staging and its barriers.
//   - Every step issues the same memory operations (out-of-range offsets
//     for missing chunks and for epilogue stores on non-final chunks), so
//     the compiler's wait counts are exact and the pipeline never drains on
//     a conservative wait.
// Tiles:  gate_up: 8 gate rows + the 8 matching up rows; epilogue writes
//         h = silu(g) * u as a bf16 hi/lo pair.
//         down: 16 output rows of W2; epilogue writes y (fp32) per pair.
#include <cmath>

#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kWv = 8;            // waves per block
constexpr int kBlk = 64 * kWv;    // threads per block
constexpr int kKC = 8;            // 32-wide K steps per streamed chunk
constexpr int kNT = 32;           // tokens staged per pass
constexpr int kNBk = kNT / 16;    // MFMA column blocks per pass
constexpr int kPad = 8;           // bf16 elements of padding per staged row
constexpr int kDepth = 3;         // streamed chunks held in registers per wave
constexpr int kMaxExperts = 1024;  // pool size limit of the library

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

// s_waitcnt: every vector-memory load of this wave done (lgkmcnt and expcnt
// left alone)
constexpr int kVmcntZero = (7 << 4) | (15 << 8);

struct Segment {
  int lo, hi;  // tile range [lo, hi) inside one expert
  int a, e, cnt, base;
  int p0;      // first token of the segment's pass (weighted walk), else 0
  int w_end;   // work item after the segment (weighted walk)
  bool e_ok;   // expert id in range: its weights may be read
};

// Next segment of the block's tile range starting at tile `lo`.  With
// `all_active` (n_active == m) the active list is the identity, so the
// expert is the slot itself and active[] is not read.  The loads of the
// expert's count and offset are issued here but consumed only by
// finish_segment, so the first weight chunks can go out in between.
__device__ __forceinline__ Segment next_segment(int lo, int r_hi, int tpe, const int* active,
                                                const int* counts, const int* offsets, int m,
                                                bool all_active) {
  Segment s;
  s.lo = lo;
  s.a = lo / tpe;
  s.hi = min(r_hi, (s.a + 1) * tpe);
  const int e = all_active ? s.a : active[s.a];
  s.e_ok = e >= 0 && e < m;
  s.e = s.e_ok ? e : 0;
  s.cnt = counts[s.e];
  s.base = offsets[s.e];
  s.p0 = 0;
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

// Token passes of expert e's pairs (0 for an invalid plan entry).
__device__ __forceinline__ int expert_passes(int e, const int* counts, const int* offsets, int m,
                                             int n_pairs) {
  if (e < 0 || e >= m) return 0;
  const int c = counts[e], b = offsets[e];
  if (c <= 0 || b < 0 || c > n_pairs - b) return 0;
  return (c + kNT - 1) / kNT;
}

// Counts of experts 2t and 2t + 1 (thread t) from the plan's offsets: one
// round of independent loads (no dependent plan reads on the decode path).
struct PairCounts {
  int o0, o1, o2;
};

__device__ __forceinline__ PairCounts load_pair_counts(const int* offsets, int m) {
  // unconditional loads with indices clamped to offsets[m] (branch-free, so
  // nothing consumes them before the caller does); past m the differences
  // are 0
  const int e0 = 2 * (int)threadIdx.x;
  return PairCounts{offsets[min(e0, m)], offsets[min(e0 + 1, m)], offsets[min(e0 + 2, m)]};
}

// Whether some expert has more tokens than one pass holds (a garbage plan
// can only make this true, which takes the checked weighted walk): each
// wave posts its verdict to its own LDS slot before a barrier, and every
// thread reads the eight slots after it, so the check rides on a barrier
// the kernel has anyway.  m <= 2 * kBlk.
__device__ __forceinline__ void post_passes_verdict(const PairCounts& c, int* verdict) {
  const bool big = c.o1 - c.o0 > kNT || c.o2 - c.o1 > kNT;
  const bool any = __ballot(big) != 0;
  if ((threadIdx.x & 63) == 0) verdict[threadIdx.x >> 6] = any ? 1 : 0;
}

__device__ __forceinline__ bool read_passes_verdict(const int* verdict) {
  int v = 0;
#pragma unroll
  for (int w = 0; w < kWv; ++w) v |= verdict[w];
  return v != 0;
}

// The same with a barrier of its own.  Every thread of the block calls it.
__device__ __forceinline__ bool some_expert_needs_passes(const PairCounts& c, int* verdict) {
  post_passes_verdict(c, verdict);
  __syncthreads();
  return read_passes_verdict(verdict);
}

// Work-weighted ranges, for a batch where some expert has more than kNT
// tokens: expert slot a owns np_a * tpe work items (its tiles once per
// token pass, pass-major) from wp[a] on, wp[n_act] being the total, and
// blocks take equal contiguous runs of work.  A popular expert is then
// spread over more blocks instead of lengthening the few blocks that own
// its tiles (when every expert fits one pass, the tile ranges are already
// balanced and this is not used).  Every thread of the block calls it;
// n_act <= 2 * kBlk.
__device__ void weighted_work(int n_act, int tpe, const int* active, const int* counts,
                              const int* offsets, int m, int n_pairs, int* wp, uint32_t* scan) {
  const int a0 = 2 * (int)threadIdx.x, a1 = a0 + 1;
  const int n0 = a0 < n_act ? expert_passes(active[a0], counts, offsets, m, n_pairs) : 0;
  const int n1 = a1 < n_act ? expert_passes(active[a1], counts, offsets, m, n_pairs) : 0;
  uint32_t off, unused, total, unused_t;
  block_exclusive_scan2((uint32_t)((n0 + n1) * tpe), 0u, scan, &off, &unused, &total, &unused_t);
  if (a0 < n_act) wp[a0] = (int)off;
  if (a1 < n_act) wp[a1] = (int)off + n0 * tpe;
  if (threadIdx.x == 0) wp[n_act] = (int)total;
  __syncthreads();
}

// Segment of the weighted walk starting at work item w < w_hi: the expert
// slot holding w (the last a with wp[a] <= w, which has work), its pass,
// and the run of tiles to the end of that pass or of the block's range.
__device__ __forceinline__ Segment weighted_segment(int w, int w_hi, int n_act, const int* wp,
                                                    int tpe, const int* active,
                                                    const int* counts, const int* offsets,
                                                    int m) {
  int lo = 0, hi = n_act - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (wp[mid] <= w)
      lo = mid;
    else
      hi = mid - 1;
  }
  Segment s;
  s.a = lo;
  const int q = w - wp[lo], pass = q / tpe, tile = q - pass * tpe;
  const int run = min(tpe - tile, w_hi - w);
  s.lo = lo * tpe + tile;
  s.hi = s.lo + run;
  s.w_end = w + run;
  s.p0 = pass * kNT;
  const int e = active[lo];
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
  const uint16_t* xs;  // LDS activations [kNT][H + kPad]
  int H, I, nsteps, cpt, lane, r, kg, wave;
  int seg_lo, seg_hi, a, tpe, p0, cnt, nbn;
};

// Weight chunk q of this wave's tiles.  Row-major: lane (r, kg) reads 16 B
// of weight row r at 64-byte K steps.  Tiled: the tile's fragments are
// contiguous, so the wave reads 1 KiB per load (non-temporal: read once).
template <bool kTiled>
__device__ __forceinline__ void gu_issue(const GuWave& g, int q, int Q, u32x4 (&A)[kKC]) {
  const int j = q / g.cpt, c = q - j * g.cpt;
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
#pragma unroll
  for (int s = 0; s < kKC; ++s) {
    const int step = c * kKC + s;
    const uint32_t off = (q < Q && step < g.nsteps) ? row + (uint32_t)step * stride : kOutOfRange;
    A[s] = kTiled ? buf_ld128_stream(g.w, off) : buf_ld128(g.w, off);
  }
}

__device__ __forceinline__ void gu_compute(const GuWave& g, int q, const u32x4 (&A)[kKC],
                                           f32x4 (&acc)[kNBk]) {
  const int j = q / g.cpt, c = q - j * g.cpt;
  if (c == 0) {
#pragma unroll
    for (int nb = 0; nb < kNBk; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int nb = 0; nb < kNBk; ++nb) {
    if (nb < g.nbn) {
      const uint16_t* row = g.xs + (nb * 16 + g.r) * (g.H + kPad) + g.kg * 8;
      u32x4 B[kKC];
#pragma unroll
      for (int s = 0; s < kKC; ++s) {
        const int step = c * kKC + s;
        const bool ok = step < g.nsteps;
        const u32x4 v = *reinterpret_cast<const u32x4*>(row + (ok ? step * 32 : 0));
        B[s] = ok ? v : zero4();
      }
#pragma unroll
      for (int s = 0; s < kKC; ++s) acc[nb] = mfma_16x16x32(A[s], B[s], acc[nb]);
    }
  }
  // epilogue on the tile's last chunk: SwiGLU of the 8 (gate, up) row pairs
  // for every token column; lanes 0-31 own the results
  const bool last = c == g.cpt - 1;
  const int tile = g.seg_lo + g.wave + j * kWv;
  const int ib = tile - g.a * g.tpe;
#pragma unroll
  for (int nb = 0; nb < kNBk; ++nb) {
    uint32_t off = kOutOfRange;
    u32x2 hw = {0u, 0u}, lw = {0u, 0u};
    if (last && nb < g.nbn) {
      const f32x4 v = acc[nb];
      f32x4 u;
#pragma unroll
      for (int i = 0; i < 4; ++i) u[i] = __shfl_xor(v[i], 32);
      uint16_t hb[4], lb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float gt = v[i];
        const float hv = (gt / (1.0f + expf(-gt))) * u[i];
        hb[i] = f32_to_bf16(hv);
        lb[i] = f32_to_bf16(hv - bf16_to_f32(hb[i]));
      }
      hw = u32x2{(uint32_t)hb[0] | ((uint32_t)hb[1] << 16), (uint32_t)hb[2] | ((uint32_t)hb[3] << 16)};
      lw = u32x2{(uint32_t)lb[0] | ((uint32_t)lb[1] << 16), (uint32_t)lb[2] | ((uint32_t)lb[3] << 16)};
      const int slot = g.p0 + nb * 16 + g.r;
      if (g.lane < 32 && slot < g.cnt)
        off = ((uint32_t)slot * g.I + (uint32_t)(ib * 8 + g.kg * 4)) * 2u;
    }
    __builtin_amdgcn_raw_buffer_store_b64(hw, g.hh, off, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b64(lw, g.hl, off, 0, 0);
  }
}

// kBalance: the batch has more tokens than one pass holds, so an expert
// may need several passes and the blocks may switch to the weighted walk.
// kSpeculate: guess n_active == m and issue the first weight chunks before
// n_active arrives (a wrong guess redoes the first segment).
template <bool kTiled, bool kBalance, bool kSpeculate>
__global__ __launch_bounds__(kBlk, 1) void gate_up_wave_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w13,
    const int* __restrict__ counts, const int* __restrict__ offsets,
    const int* __restrict__ perm, const int* __restrict__ active,
    const int* __restrict__ n_active_p, uint16_t* __restrict__ h_hi,
    uint16_t* __restrict__ h_lo, int H, int I, int m, int k, int n_pairs) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[kNT * (kMaxStreamH + kPad)];
  __shared__ int pid[kNT];
  __shared__ int wp[kMaxExperts + 1];
  __shared__ uint32_t scan[34];
  __shared__ int verdict[kWv];
  const int tpe = I / 8;
  const int n_act = *n_active_p;
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
  int Q = 0;
  // weight resource of the segment's expert and its first kDepth - 1 chunks
  auto begin_segment = [&](const Segment& sg) {
    g.seg_lo = sg.lo;
    g.seg_hi = sg.hi;
    g.a = sg.a;
    g.w = make_rsrc(w13 + (size_t)sg.e * 2 * I * H, sg.e_ok ? 4u * (uint32_t)I * (uint32_t)H : 0u);
    // this wave's tiles of the segment: seg_lo + wave, + kWv, ...
    const int ntw = sg.hi - sg.lo > g.wave ? (sg.hi - sg.lo - g.wave + kWv - 1) / kWv : 0;
    Q = ntw * g.cpt;
#pragma unroll
    for (int d = 0; d < kDepth - 1; ++d) gu_issue<kTiled>(g, d, Q, A[d]);
  };

  // Speculate a fully active pool (n_active == m, the usual saturated decode
  // batch): the block's tile range and its first expert then follow from m
  // alone, so that segment's plan loads and weight chunks go out together
  // with the n_active load.  A wrong guess redoes the first segment.
  // (Without kSpeculate the first segment waits for n_active instead.)
  const PairCounts pc = kBalance ? load_pair_counts(offsets, m) : PairCounts{0, 0, 0};
  int r_lo = 0, r_hi = 0;
  Segment sg;
  if constexpr (kSpeculate) {
    block_range(m * tpe, &r_lo, &r_hi);
    sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, true);
    begin_segment(sg);
  }
  if (n_act <= 0 || n_act > m) return;  // an invalid plan: no work
  if constexpr (!kSpeculate) block_range(n_act * tpe, &r_lo, &r_hi);
  const bool all = n_act == m;
  // With kBalance, whether some expert needs several token passes is
  // decided once, by the first barrier of the block's first pass (so that
  // pass's pair-id loads are already out); a block without such a barrier
  // decides it here.  With several passes the block switches to its range
  // of the weighted walk.
  bool checked = !kBalance, weighted = false;
  int w_hi = 0;
  auto go_weighted = [&]() {
    weighted = true;
    weighted_work(n_act, tpe, active, counts, offsets, m, n_pairs, wp, scan);
    block_range(wp[n_act], &r_lo, &w_hi);
    if (r_lo >= w_hi) return false;
    sg = weighted_segment(r_lo, w_hi, n_act, wp, tpe, active, counts, offsets, m);
    begin_segment(sg);
    return true;
  };
  if constexpr (!kBalance) {
    if (!all) {
      block_range(n_act * tpe, &r_lo, &r_hi);
      if (r_lo >= r_hi) return;
      sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, false);
      begin_segment(sg);
    } else if (r_lo >= r_hi) {
      return;
    }
  } else {
    if (kSpeculate && !all) block_range(n_act * tpe, &r_lo, &r_hi);
    if (r_lo < r_hi && (!kSpeculate || !all)) {
      sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, all);
      begin_segment(sg);
    }
    if (r_lo >= r_hi) {
      checked = true;
      if (!some_expert_needs_passes(pc, verdict) || !go_weighted()) return;
    }
  }

  for (;;) {
    finish_segment(sg, n_pairs);
    if (!checked && sg.cnt == 0) {  // no pass (hence no barrier) in this segment
      checked = true;
      if (some_expert_needs_passes(pc, verdict)) {
        if (!go_weighted()) return;
        continue;
      }
    }
    g.cnt = sg.cnt;
    const uint32_t hbytes = 2u * (uint32_t)sg.cnt * (uint32_t)I;
    g.hh = make_rsrc(h_hi + (size_t)sg.base * I, hbytes);
    g.hl = make_rsrc(h_lo + (size_t)sg.base * I, hbytes);
    // one pass per segment on the weighted walk, every pass otherwise
    const int p_end = weighted ? min(sg.cnt, sg.p0 + kNT) : sg.cnt;
    bool restart = false;
    for (int p0 = sg.p0; p0 < p_end; p0 += kNT) {
      if (p0 > sg.p0) {
#pragma unroll
        for (int d = 0; d < kDepth - 1; ++d) gu_issue<kTiled>(g, d, Q, A[d]);
      }
      g.p0 = p0;
      g.nbn = (min(kNT, sg.cnt - p0) + 15) >> 4;
      // stage this pass's token rows of x in LDS (the pair ids are loaded
      // before the barrier that waits for the previous pass's readers)
      int pv = -1;
      if ((int)threadIdx.x < kNT) {
        const int slot = p0 + threadIdx.x;
        const int p = slot < sg.cnt ? perm[sg.base + slot] : -1;
        pv = (p >= 0 && p < n_pairs) ? p : -1;
      }
      if (!checked) post_passes_verdict(pc, verdict);
      __syncthreads();
      if (!checked) {
        checked = true;
        if (read_passes_verdict(verdict)) {
          restart = true;
          break;
        }
      }
      if ((int)threadIdx.x < kNT) pid[threadIdx.x] = pv;
      __syncthreads();
      // the pass's token rows of x, straight into LDS: wave w stages rows
      // w, w + kWv, ... (rows without a pair read zeros), then one wait
      for (int tok = g.wave; tok < g.nbn * 16; tok += kWv) {
        const int p = pid[tok];
        stage_row(xr, p >= 0 ? (uint32_t)(p / k) * (uint32_t)H * 2u : kOutOfRange,
                  xs + tok * (H + kPad), 2 * H, g.lane);
      }
      __builtin_amdgcn_s_waitcnt(kVmcntZero);
      __syncthreads();

      f32x4 acc[kNBk];
#pragma unroll
      for (int nb = 0; nb < kNBk; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      // chunk q lives in A[q % kDepth]; the issue for q + kDepth - 1 goes
      // out before the compute of q
      for (int q = 0; q < Q; q += kDepth) {
#pragma unroll
        for (int d = 0; d < kDepth; ++d) {
          gu_issue<kTiled>(g, q + d + kDepth - 1, Q, A[(d + kDepth - 1) % kDepth]);
          if (d == 0 || q + d < Q) gu_compute(g, q + d, A[d], acc);
        }
      }
    }
    if (restart) {
      if (!go_weighted()) return;
      continue;
    }
    if (weighted) {
      if (sg.w_end >= w_hi) break;
      sg = weighted_segment(sg.w_end, w_hi, n_act, wp, tpe, active, counts, offsets, m);
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
  const uint16_t* hs;  // LDS h hi rows [kNT][I + kPad], then the lo rows
  const int* pid;      // LDS pair ids of the pass
  int H, I, nsteps, cpt, lane, r, kg, wave;
  int seg_lo, a, tpe, nbn;
};

template <bool kTiled>
__device__ __forceinline__ void dn_issue(const DnWave& g, int q, int Q, u32x4 (&A)[kKC]) {
  const int j = q / g.cpt, c = q - j * g.cpt;
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
#pragma unroll
  for (int s = 0; s < kKC; ++s) {
    const int step = c * kKC + s;
    const bool ok = q < Q && step < g.nsteps && o < g.H;
    const uint32_t off = ok ? row + (uint32_t)step * stride : kOutOfRange;
    A[s] = kTiled ? buf_ld128_stream(g.w, off) : buf_ld128(g.w, off);
  }
}

__device__ __forceinline__ void dn_compute(const DnWave& g, int q, const u32x4 (&A)[kKC],
                                           f32x4 (&acc)[kNBk]) {
  const int j = q / g.cpt, c = q - j * g.cpt;
  if (c == 0) {
#pragma unroll
    for (int nb = 0; nb < kNBk; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int lo_rows = kNT * (g.I + kPad);
#pragma unroll
  for (int nb = 0; nb < kNBk; ++nb) {
    if (nb < g.nbn) {
      const uint16_t* row = g.hs + (nb * 16 + g.r) * (g.I + kPad) + g.kg * 8;
#pragma unroll
      for (int s = 0; s < kKC; ++s) {
        const int step = c * kKC + s;
        const bool ok = step < g.nsteps;
        const int col = ok ? step * 32 : 0;
        const u32x4 bh = *reinterpret_cast<const u32x4*>(row + col);
        const u32x4 bl = *reinterpret_cast<const u32x4*>(row + lo_rows + col);
        acc[nb] = mfma_16x16x32(A[s], ok ? bh : zero4(), acc[nb]);
        acc[nb] = mfma_16x16x32(A[s], ok ? bl : zero4(), acc[nb]);
      }
    }
  }
  const bool last = c == g.cpt - 1;
  const int tile = g.seg_lo + g.wave + j * kWv;
  const int o = (tile - g.a * g.tpe) * 16 + g.kg * 4;
#pragma unroll
  for (int nb = 0; nb < kNBk; ++nb) {
    uint32_t off = kOutOfRange;
    if (last && nb < g.nbn) {
      const int p = g.pid[nb * 16 + g.r];
      if (p >= 0 && o < g.H) off = ((uint32_t)p * g.H + (uint32_t)o) * 4u;
    }
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[nb]), g.y, off, 0, 0);
  }
}

template <bool kTiled, bool kBalance, bool kSpeculate>
__global__ __launch_bounds__(kBlk, 1) void down_wave_kernel(
    const uint16_t* __restrict__ h_hi, const uint16_t* __restrict__ h_lo,
    const uint16_t* __restrict__ w2, const int* __restrict__ counts,
    const int* __restrict__ offsets, const int* __restrict__ perm,
    const int* __restrict__ active, const int* __restrict__ n_active_p, float* __restrict__ y,
    int H, int I, int m, int n_pairs) {
  __shared__ __attribute__((aligned(16))) uint16_t hs[2 * kNT * (kMaxStreamI + kPad)];
  __shared__ int pid[kNT];
  __shared__ int wp[kMaxExperts + 1];
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
  const int lo_rows = kNT * (I + kPad);
  const uint32_t hbytes = 2u * (uint32_t)n_pairs * (uint32_t)I;
  const auto hhr = make_rsrc(h_hi, hbytes);
  const auto hlr = make_rsrc(h_lo, hbytes);

  u32x4 A[kDepth][kKC];
  int Q = 0;
  auto begin_segment = [&](const Segment& sg) {
    g.seg_lo = sg.lo;
    g.a = sg.a;
    g.w = make_rsrc(w2 + (size_t)sg.e * H * I, sg.e_ok ? 2u * (uint32_t)H * (uint32_t)I : 0u);
    const int ntw = sg.hi - sg.lo > g.wave ? (sg.hi - sg.lo - g.wave + kWv - 1) / kWv : 0;
    Q = ntw * g.cpt;
#pragma unroll
    for (int d = 0; d < kDepth - 1; ++d) dn_issue<kTiled>(g, d, Q, A[d]);
  };

  // Speculate a fully active pool, as in gate_up_wave_kernel.
  // (Without kSpeculate the first segment waits for n_active instead.)
  const PairCounts pc = kBalance ? load_pair_counts(offsets, m) : PairCounts{0, 0, 0};
  int r_lo = 0, r_hi = 0;
  Segment sg;
  if constexpr (kSpeculate) {
    block_range(m * tpe, &r_lo, &r_hi);
    sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, true);
    begin_segment(sg);
  }
  if (n_act <= 0 || n_act > m) return;  // an invalid plan: no work
  if constexpr (!kSpeculate) block_range(n_act * tpe, &r_lo, &r_hi);
  const bool all = n_act == m;
  // With kBalance, whether some expert needs several token passes is
  // decided once, by the first barrier of the block's first pass (so that
  // pass's pair-id loads are already out); a block without such a barrier
  // decides it here.  With several passes the block switches to its range
  // of the weighted walk.
  bool checked = !kBalance, weighted = false;
  int w_hi = 0;
  auto go_weighted = [&]() {
    weighted = true;
    weighted_work(n_act, tpe, active, counts, offsets, m, n_pairs, wp, scan);
    block_range(wp[n_act], &r_lo, &w_hi);
    if (r_lo >= w_hi) return false;
    sg = weighted_segment(r_lo, w_hi, n_act, wp, tpe, active, counts, offsets, m);
    begin_segment(sg);
    return true;
  };
  if constexpr (!kBalance) {
    if (!all) {
      block_range(n_act * tpe, &r_lo, &r_hi);
      if (r_lo >= r_hi) return;
      sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, false);
      begin_segment(sg);
    } else if (r_lo >= r_hi) {
      return;
    }
  } else {
    if (kSpeculate && !all) block_range(n_act * tpe, &r_lo, &r_hi);
    if (r_lo < r_hi && (!kSpeculate || !all)) {
      sg = next_segment(r_lo, r_hi, tpe, active, counts, offsets, m, all);
      begin_segment(sg);
    }
    if (r_lo >= r_hi) {
      checked = true;
      if (!some_expert_needs_passes(pc, verdict) || !go_weighted()) return;
    }
  }

  for (;;) {
    finish_segment(sg, n_pairs);
    if (!checked && sg.cnt == 0) {  // no pass (hence no barrier) in this segment
      checked = true;
      if (some_expert_needs_passes(pc, verdict)) {
        if (!go_weighted()) return;
        continue;
      }
    }
    const int p_end = weighted ? min(sg.cnt, sg.p0 + kNT) : sg.cnt;
    bool restart = false;
    for (int p0 = sg.p0; p0 < p_end; p0 += kNT) {
      if (p0 > sg.p0) {
#pragma unroll
        for (int d = 0; d < kDepth - 1; ++d) dn_issue<kTiled>(g, d, Q, A[d]);
      }
      g.nbn = (min(kNT, sg.cnt - p0) + 15) >> 4;
      // the pass's pair ids (for the y rows) and its h rows, which are
      // contiguous in dispatch-slot order
      int pv = -1;
      if ((int)threadIdx.x < kNT) {
        const int slot = p0 + threadIdx.x;
        const int p = slot < sg.cnt ? perm[sg.base + slot] : -1;
        pv = (p >= 0 && p < n_pairs) ? p : -1;
      }
      if (!checked) post_passes_verdict(pc, verdict);
      __syncthreads();  // the previous pass's readers of hs and pid are done
      if (!checked) {
        checked = true;
        if (read_passes_verdict(verdict)) {
          restart = true;
          break;
        }
      }
      if ((int)threadIdx.x < kNT) pid[threadIdx.x] = pv;
      // the pass's h rows (hi, then lo), straight into LDS: wave w stages
      // rows w, w + kWv, ... of both halves, then one wait
      for (int tok = g.wave; tok < g.nbn * 16; tok += kWv) {
        const int slot = p0 + tok;
        const uint32_t src =
            slot < sg.cnt ? (uint32_t)(sg.base + slot) * (uint32_t)I * 2u : kOutOfRange;
        stage_row(hhr, src, hs + tok * (I + kPad), 2 * I, g.lane);
        stage_row(hlr, src, hs + lo_rows + tok * (I + kPad), 2 * I, g.lane);
      }
      __builtin_amdgcn_s_waitcnt(kVmcntZero);
      __syncthreads();

      f32x4 acc[kNBk];
#pragma unroll
      for (int nb = 0; nb < kNBk; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int q = 0; q < Q; q += kDepth) {
#pragma unroll
        for (int d = 0; d < kDepth; ++d) {
          dn_issue<kTiled>(g, q + d + kDepth - 1, Q, A[(d + kDepth - 1) % kDepth]);
          if (d == 0 || q + d < Q) dn_compute(g, q + d, A[d], acc);
        }
      }
    }
    if (restart) {
      if (!go_weighted()) return;
      continue;
    }
    if (weighted) {
      if (sg.w_end >= w_hi) break;
      sg = weighted_segment(sg.w_end, w_hi, n_act, wp, tpe, active, counts, offsets, m);
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

// Variant of a launch.  An expert receives at most one pair per token of a
// routed batch, so a batch of T tokens gives an expert at most ceil(T / kNT)
// passes; the weighted walk (and the check that selects it, which costs a
// little on every launch) is compiled in once that bound exceeds two, where
// one popular expert could otherwise make a few blocks take three or more
// times as long as the rest.  Guessing a fully active pool pays when the
// expected number of idle experts, m (1 - k/m)^T, is well below one.
struct WaveMode {
  bool balance, speculate;
};

WaveMode wave_mode(int T, int m, int k) {
  WaveMode md;
  md.balance = T > 2 * kNT;
  const double idle = m * std::pow(1.0 - (double)k / m, (double)T);
  md.speculate = !md.balance || idle < 0.25;
  return md;
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
  const WaveMode md = wave_mode(T, m, k);
#define SW_GU(TI, BA, SP)                                                                      \
  gate_up_wave_kernel<TI, BA, SP><<<stream_grid(), kBlk, 0, stream>>>(                          \
      x, w13, counts, offsets, perm, active, n_active, h_hi, h_lo, H, I, m, k, T * k)
  if (!md.balance) {
    if (tiled) SW_GU(true, false, true); else SW_GU(false, false, true);
  } else if (md.speculate) {
    if (tiled) SW_GU(true, true, true); else SW_GU(false, true, true);
  } else {
    if (tiled) SW_GU(true, true, false); else SW_GU(false, true, false);
  }
#undef SW_GU
  return hipGetLastError();
}

hipError_t launch_down_wave(int T, const uint16_t* w2, bool tiled, const int* counts,
                            const int* offsets, const int* perm, const int* active,
                            const int* n_active, int H, int I, int m, int k, const uint16_t* h_hi,
                            const uint16_t* h_lo, float* y, hipStream_t stream) {
  const WaveMode md = wave_mode(T, m, k);
#define SW_DN(TI, BA, SP)                                                                      \
  down_wave_kernel<TI, BA, SP><<<stream_grid(), kBlk, 0, stream>>>(                             \
      h_hi, h_lo, w2, counts, offsets, perm, active, n_active, y, H, I, m, T * k)
  if (!md.balance) {
    if (tiled) SW_DN(true, false, true); else SW_DN(false, false, true);
  } else if (md.speculate) {
    if (tiled) SW_DN(true, true, true); else SW_DN(false, true, true);
  } else {
    if (tiled) SW_DN(true, true, false); else SW_DN(false, true, false);
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
