// Expert FFN kernels for prefill-sized batches on gfx950 (Section 2.1: with
// many tokens per expert the layer reuses each weight across those tokens,
// so the step turns from weight streaming toward MFMA work).
//
// The decode kernels keep an expert's tokens in LDS over the whole
// contraction and stream each 16-row tile once per 32-token pass; with
// ~128 tokens per expert that would re-stream every weight four times.
// Here the loop order is inverted:
//   - a unit is (active expert, group of 16 row tiles), two tiles per wave;
//     a persistent grid of one 8-wave block per compute unit walks the units,
//     each XCD taking a contiguous run of every round's units (an expert's
//     units then share one L2 for its gathered activations);
//   - a pass covers up to 160 of the expert's tokens (10 MFMA column
//     blocks), so a unit streams its weights once per pass, normally once;
//   - the contraction runs in chunks of K: the activations of the pass are
//     staged chunk by chunk through a double-buffered LDS ring (the loads of
//     chunk c + 1 go out before chunk c is computed and land in LDS after),
//     while the weight chunks stream through a register pipeline (two
//     chunks deep for gate/up, three for down) in the same fragment-major
//     layout as the decode kernels;
//   - every B fragment read from LDS feeds the MFMAs of both of the wave's
//     tiles, halving LDS traffic per MFMA.
// Each output accumulates over K in the same order as the decode kernels.
#include <type_traits>

#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kWv = 8;                 // waves per block
constexpr int kBlk = 64 * kWv;         // threads per block
constexpr int kTpw = 2;                // 16-row tiles per wave per unit
constexpr int kTpu = kWv * kTpw;       // tiles per unit
constexpr int kNB = 10;                // 16-token column blocks per pass
constexpr int kNT = 16 * kNB;          // tokens per pass
constexpr int kPad = 8;                // bf16 padding per staged row
constexpr int kRowsPad = kNT + 32;     // staged rows: the pass's, then a trash area that
                                       // takes the idle slots of a partial staging round

// gate/up: chunk = 2 K steps (64 columns of x), 3 chunks of weights in flight
constexpr int kGuKs = 2;
constexpr int kGuKc = 32 * kGuKs;
// Pipeline depth D: D chunks of weights held in registers per wave and D
// ring slots of staged activations in LDS, so D - 1 chunks of each are in
// flight ahead of the one computed.  The code takes 2 or 4; 2 measured
// faster for both kernels (about 4% for gate/up, 14% for down at the
// 4096-token prefill shape).
constexpr int kDepth = 2;
constexpr int kSegRows = 8;            // staged rows per 1 KiB direct-to-LDS load of a wave
static_assert(kGuKc * 2 * kSegRows == 1024, "one wave load fills kSegRows rows");
// down: chunk = 2 K steps (64 columns of h hi and of h lo), 3 in flight;
// the staged h goes through the same kind of ring as gate/up's x
constexpr int kDnKs = 2;
constexpr int kDnKc = 32 * kDnKs;
static_assert(kDnKc == kGuKc, "one segment geometry for both staged operands");

// Unit u -> (active slot a, tile group grp); the expert and its pair range,
// validated against the plan.
struct Unit {
  int e, cnt, base, grp;
  bool ok;
};

__device__ __forceinline__ Unit unit_of(int u, int gpe, const int* active, const int* counts,
                                        const int* offsets, int m, int n_pairs) {
  Unit s;
  const int a = u / gpe;
  s.grp = u - a * gpe;
  const int e = active[a];
  s.ok = e >= 0 && e < m;
  s.e = s.ok ? e : 0;
  s.cnt = s.ok ? counts[s.e] : 0;
  s.base = s.ok ? offsets[s.e] : 0;
  s.ok = s.ok && s.cnt > 0 && s.base >= 0 && s.cnt <= n_pairs - s.base;
  return s;
}

// Slot of block b in each round of gridDim.x units.  Blocks are dispatched
// round-robin over the eight XCDs (block b runs on XCD b % 8); giving each
// XCD a contiguous run of the round's units puts the units of one expert
// (consecutive in the list) on one XCD at the same time, so they share that
// XCD's L2 for the expert's gathered activations.
__device__ __forceinline__ int unit_slot() {
  const int b = blockIdx.x, g = gridDim.x;
  return (g & 7) ? b : (b & 7) * (g >> 3) + (b >> 3);
}

// Rows of one pass into LDS: the pair id of dispatch slot p0 + i divided by
// `div` (k: the token), -1 past the expert's count and in the trash rows.
__device__ __forceinline__ void load_pass_rows(const int* perm, int base, int p0, int cnt,
                                               int n_pairs, int div, int* rows) {
  if ((int)threadIdx.x < kRowsPad) {
    const int slot = p0 + threadIdx.x;
    const int p = (int)threadIdx.x < kNT && slot < cnt ? perm[base + slot] : -1;
    rows[threadIdx.x] = (p >= 0 && p < n_pairs) ? p / div : -1;
  }
}

// Column blocks computed by a pass of nbn blocks: every MFMA loop of a pass
// runs over a compile-time count (no per-block branch between an LDS read
// and its MFMAs); blocks past the pass's tokens multiply zero rows.
template <typename F>
__device__ __forceinline__ void with_blocks(int nbn, F&& f) {
  if (nbn <= 4)
    f(std::integral_constant<int, 4>{});
  else if (nbn <= 8)
    f(std::integral_constant<int, 8>{});
  else
    f(std::integral_constant<int, kNB>{});
}

// ---------------------------------------------------------------------------
// gate/up + SwiGLU

// Weight chunk c of the wave's tiles: kGuKs fragments of 1 KiB per tile.
template <bool kTiled>
__device__ __forceinline__ void gu_issue(__amdgpu_buffer_rsrc_t w, const int (&ib)[kTpw],
                                         int c, int nchunks, int H, int I, int lane,
                                         u32x4 (&A)[kTpw][kGuKs]) {
  const int r = lane & 15, kg = lane >> 4;
#pragma unroll
  for (int t = 0; t < kTpw; ++t) {
    uint32_t row, stride;
    if (kTiled) {
      row = (uint32_t)ib[t] * 32u * H + (uint32_t)lane * 16u;
      stride = 1024u;
    } else {
      const int wrow = r < 8 ? ib[t] * 8 + r : I + ib[t] * 8 + (r - 8);
      row = (uint32_t)wrow * H * 2u + kg * 16u;
      stride = 64u;
    }
    const bool ok = c < nchunks && ib[t] >= 0;
#pragma unroll
    for (int s = 0; s < kGuKs; ++s) {
      const uint32_t off = ok ? row + (uint32_t)(c * kGuKs + s) * stride : kOutOfRange;
      A[t][s] = kTiled ? buf_ld128_stream(w, off) : buf_ld128(w, off);
    }
  }
}

// x of a pass of NBK column blocks goes straight from memory to LDS
// (buffer loads with the LDS bit: lane l of a wave writes bytes 16 l .. +15
// of a 1 KiB segment).  A segment holds kSegRows rows of the chunk's 64
// columns, unpadded; the 16-byte pieces of row R sit in XOR-swizzled slots,
// slot = piece ^ x_swizzle(R), so that the MFMA operand reads (16 rows, one
// piece each, per 16 lanes) hit distinct banks.  Segments run over the
// pass's rows and then, for a partial last round of the waves, the trash
// rows.
__device__ __forceinline__ int x_swizzle(int row) { return (row & 7) ^ ((row >> 3) & 1); }

template <int NBK>
constexpr int gu_segs() {  // direct-to-LDS loads per wave per chunk
  constexpr int kSegs = (NBK * 16 / kSegRows + kWv - 1) / kWv;
  static_assert(kSegs * kWv * kSegRows <= kRowsPad, "trash rows hold the idle segments");
  return kSegs;
}

// s_waitcnt immediates: at most n vector-memory loads outstanding (expcnt
// and lgkmcnt left alone), and the same with every LDS access done
constexpr int vmcnt_at_most(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int vmcnt_at_most_lds_done(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

template <bool kTiled, int D, int NBK>
__device__ __forceinline__ void gu_pass(__amdgpu_buffer_rsrc_t w, __amdgpu_buffer_rsrc_t xr,
                                        const int (&ib)[kTpw], const int* tok,
                                        uint16_t* __restrict__ x0, uint16_t* __restrict__ x1,
                                        uint16_t* __restrict__ x2, uint16_t* __restrict__ x3,
                                        __amdgpu_buffer_rsrc_t hh, __amdgpu_buffer_rsrc_t hl,
                                        int p0, int cnt, int H, int I, int nchunks, int lane,
                                        int wave) {
  // the ring slots as distinct restrict pointers: the compiler then knows
  // that the loads into one slot do not write the slot being read, and does
  // not wait for them before the reads
  static_assert(D == 2 || D == 4, "two or four ring slots");
  constexpr int kAhead = D - 1;
  auto slot = [&](int k) { return k == 0 ? x0 : k == 1 ? x1 : k == 2 ? x2 : x3; };
  constexpr int kSegs = gu_segs<NBK>();
  constexpr int kWloads = kTpw * kGuKs;  // weight loads per wave per chunk
  const int r = lane & 15, kg = lane >> 4;
  // source byte offset of this lane's piece of each segment in chunk 0; a
  // row without a pair reads out of range in every chunk (at most H * 2
  // bytes are added to 2^31, still past the resource)
  uint32_t soff[kSegs];
#pragma unroll
  for (int j = 0; j < kSegs; ++j) {
    const int row = (wave + j * kWv) * kSegRows + (lane >> 3);
    const int piece = (lane & 7) ^ x_swizzle(row);
    const int t = tok[row];
    soff[j] = t >= 0 ? ((uint32_t)t * H + (uint32_t)piece * 8u) * 2u : kOutOfRange;
  }
  auto stage = [&](int c, int k) {  // chunk c into ring slot k = c % D
    uint16_t* buf = slot(k);
#pragma unroll
    for (int j = 0; j < kSegs; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          xr, (__attribute__((address_space(3))) void*)(buf + (wave + j * kWv) * kSegRows * kGuKc),
          16, soff[j] + (uint32_t)c * kGuKc * 2u, 0, 0, 0);
  };
  // this lane's operand slot in a staged row, per K step (row & 15 = r)
  int bslot[kGuKs];
#pragma unroll
  for (int st = 0; st < kGuKs; ++st) bslot[st] = ((st * 4 + kg) ^ x_swizzle(r)) * 8;

  // prologue: x chunks 0 .. D - 2, then weight chunks 0 .. D - 2
#pragma unroll
  for (int c = 0; c < kAhead; ++c) stage(c, c);
  __builtin_amdgcn_sched_barrier(0);  // the load order the waits below count on
  u32x4 A[D][kTpw][kGuKs];
#pragma unroll
  for (int d = 0; d < kAhead; ++d) {  // in chunk order: the waits assume it
    gu_issue<kTiled>(w, ib, d, nchunks, H, I, lane, A[d]);
    __builtin_amdgcn_sched_barrier(0);
  }
  f32x4 acc[kTpw][NBK];
#pragma unroll
  for (int t = 0; t < kTpw; ++t)
#pragma unroll
    for (int nb = 0; nb < NBK; ++nb) acc[t][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Each chunk issues x chunk c + D - 1 and weight chunk c + D - 1,
  // unconditionally (nchunks is a multiple of D; past the end the
  // loads read out of range or land in ring slots never read again), so the
  // count of loads issued after x chunk c is known: the wait below lets
  // exactly those stay outstanding.  The compiler does not track the LDS
  // writes of these loads, hence the explicit wait and a plain barrier
  // (a __syncthreads fence would wait for every load, weights included).
  // (the prologue leaves the same count ahead of chunk 0 as a chunk body
  // leaves ahead of chunk c + D - 1, and the ring slot of chunk c is d)
  constexpr int kAfter = (kAhead - 1) * (kSegs + kWloads) + kWloads;
  for (int c0 = 0; c0 < nchunks; c0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int c = c0 + d;
      // this wave's part of chunk c landed and its reads of chunk c - 1 are done
      __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(kAfter));
      __builtin_amdgcn_s_barrier();  // so for every wave: chunk c - 1's slot is free
      stage(c + kAhead, (d + kAhead) % D);  // c0 is a multiple of D
      __builtin_amdgcn_sched_barrier(0);  // x loads first, then the weights (the count)
      gu_issue<kTiled>(w, ib, c + kAhead, nchunks, H, I, lane, A[(d + kAhead) % D]);
      // the loads stay ahead of the chunk's MFMAs (the scheduler would sink
      // them to their first use to shorten register lifetimes)
      __builtin_amdgcn_sched_barrier(0);
      const uint16_t* buf = slot(d);
#pragma unroll
      for (int st = 0; st < kGuKs; ++st) {
#pragma unroll
        for (int nb = 0; nb < NBK; ++nb) {
          const u32x4 b =
              *reinterpret_cast<const u32x4*>(buf + (nb * 16 + r) * kGuKc + bslot[st]);
#pragma unroll
          for (int t = 0; t < kTpw; ++t) acc[t][nb] = mfma_16x16x32(A[d][t][st], b, acc[t][nb]);
        }
      }
    }
  }
  // the x loads past the last chunk write ring slots that the next pass
  // stages into: they land before this pass ends
  __builtin_amdgcn_s_waitcnt(vmcnt_at_most(0));

  // SwiGLU of each tile's 8 (gate, up) row pairs, two column blocks (a, b)
  // at a time so that every lane finishes an output: lanes 0-31 hold a's
  // gates and lanes 32-63 a's ups (likewise for b); one exchange across the
  // halves hands lanes 0-31 a's ups and lanes 32-63 b's gates.  The
  // arithmetic per output is unchanged.
  static_assert(NBK % 2 == 0, "column blocks in pairs");
  const int half = lane >> 5, kgx = (lane >> 4) & 1;
#pragma unroll
  for (int t = 0; t < kTpw; ++t) {
#pragma unroll
    for (int nb = 0; nb < NBK; nb += 2) {
      f32x4 g4, u4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float a = acc[t][nb][i], b = acc[t][nb + 1][i];
        const float y = __shfl_xor(half ? a : b, 32);  // lanes < 32: a's up; else b's gate
        g4[i] = half ? y : a;
        u4[i] = half ? b : y;
      }
      float hv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) hv[i] = swiglu(g4[i], u4[i]);
      u32x2 hw, lw;
      split_bf16x4(hv, hw, lw);
      const int slot = p0 + (nb + half) * 16 + r;
      uint32_t off = kOutOfRange;
      if (ib[t] >= 0 && slot < cnt) off = ((uint32_t)slot * I + (uint32_t)(ib[t] * 8 + kgx * 4)) * 2u;
      __builtin_amdgcn_raw_buffer_store_b64(hw, hh, off, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b64(lw, hl, off, 0, 0);
    }
  }
}

template <bool kTiled, int D>
__global__ __launch_bounds__(kBlk, 1) void gate_up_prefill_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w13,
    const int* __restrict__ counts, const int* __restrict__ offsets,
    const int* __restrict__ perm, const int* __restrict__ active,
    const int* __restrict__ n_active_p, uint16_t* __restrict__ h_hi,
    uint16_t* __restrict__ h_lo, int H, int I, int m, int k, int n_pairs) {
  __shared__ __attribute__((aligned(1024))) uint16_t xs0[kRowsPad * kGuKc];
  __shared__ __attribute__((aligned(1024))) uint16_t xs1[kRowsPad * kGuKc];
  __shared__ __attribute__((aligned(1024))) uint16_t xs2[kRowsPad * kGuKc];
  __shared__ __attribute__((aligned(1024))) uint16_t xs3[kRowsPad * kGuKc];
  __shared__ int tok[kRowsPad];
  const int n_act = *n_active_p;
  if (n_act <= 0 || n_act > m) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int tpe = I / 8;                      // tiles per expert
  const int gpe = (tpe + kTpu - 1) / kTpu;    // units per expert
  const int nchunks = H / kGuKc;
  const auto xr = make_rsrc(x, 2u * (uint32_t)(n_pairs / k) * (uint32_t)H);

  for (int u = unit_slot(); u < n_act * gpe; u += gridDim.x) {
    const Unit s = unit_of(u, gpe, active, counts, offsets, m, n_pairs);
    if (!s.ok) continue;  // block-uniform
    const auto w = make_rsrc(w13 + (size_t)s.e * 2 * I * H, 4u * (uint32_t)I * (uint32_t)H);
    const uint32_t hbytes = 2u * (uint32_t)s.cnt * (uint32_t)I;
    const auto hh = make_rsrc(h_hi + (size_t)s.base * I, hbytes);
    const auto hl = make_rsrc(h_lo + (size_t)s.base * I, hbytes);
    int ib[kTpw];
#pragma unroll
    for (int t = 0; t < kTpw; ++t) {
      const int tile = s.grp * kTpu + wave * kTpw + t;
      ib[t] = tile < tpe ? tile : -1;
    }

    for (int p0 = 0; p0 < s.cnt; p0 += kNT) {
      const int nbn = (min(kNT, s.cnt - p0) + 15) >> 4;
      __syncthreads();  // the previous pass's readers of tok and xs are done
      load_pass_rows(perm, s.base, p0, s.cnt, n_pairs, k, tok);
      __syncthreads();
      with_blocks(nbn, [&](auto nbk) {
        gu_pass<kTiled, D, decltype(nbk)::value>(w, xr, ib, tok, xs0, xs1, xs2, xs3, hh, hl, p0,
                                              s.cnt, H, I, nchunks, lane, wave);
      });
    }
  }
}

// ---------------------------------------------------------------------------
// down projection

template <bool kTiled>
__device__ __forceinline__ void dn_issue(__amdgpu_buffer_rsrc_t w, const int (&ob)[kTpw], int c,
                                         int nchunks, int H, int I, int lane,
                                         u32x4 (&A)[kTpw][kDnKs]) {
  const int r = lane & 15, kg = lane >> 4;
#pragma unroll
  for (int t = 0; t < kTpw; ++t) {
    uint32_t row, stride;
    if (kTiled) {
      row = (uint32_t)ob[t] * 32u * I + (uint32_t)lane * 16u;
      stride = 1024u;
    } else {
      row = (uint32_t)(ob[t] * 16 + r) * I * 2u + kg * 16u;
      stride = 64u;
    }
    const bool ok = c < nchunks && ob[t] >= 0;
#pragma unroll
    for (int s = 0; s < kDnKs; ++s) {
      const uint32_t off = ok ? row + (uint32_t)(c * kDnKs + s) * stride : kOutOfRange;
      A[t][s] = kTiled ? buf_ld128_stream(w, off) : buf_ld128(w, off);
    }
  }
}

// h of a pass of NBK column blocks goes straight to LDS like gate/up's x:
// per ring slot the hi rows, then the lo rows, each kNT rows of the chunk's
// 64 columns in swizzled 1 KiB segments.  The rows are the expert's dispatch
// slots base + p0 + row, contiguous, so no pair id is needed to stage them.
template <int NBK>
constexpr int dn_segs() {  // direct-to-LDS loads per wave per chunk (both halves)
  static_assert(2 * NBK * 16 / kSegRows % kWv == 0, "whole rounds of segments");
  return 2 * NBK * 16 / kSegRows / kWv;
}

template <bool kTiled, int D, int NBK>
__device__ __forceinline__ void dn_pass(__amdgpu_buffer_rsrc_t w, __amdgpu_buffer_rsrc_t hhr,
                                        __amdgpu_buffer_rsrc_t hlr, const int (&ob)[kTpw],
                                        const int* __restrict__ perm, int n_pairs,
                                        uint16_t* __restrict__ s0, uint16_t* __restrict__ s1,
                                        uint16_t* __restrict__ s2, uint16_t* __restrict__ s3,
                                        __amdgpu_buffer_rsrc_t yr, int base, int p0, int cnt,
                                        int H, int I, int nchunks, int lane, int wave) {
  static_assert(D == 2 || D == 4, "two or four ring slots");
  constexpr int kAhead = D - 1;
  auto slot = [&](int k) { return k == 0 ? s0 : k == 1 ? s1 : k == 2 ? s2 : s3; };
  constexpr int kSegs = dn_segs<NBK>(), kSegsHalf = NBK * 16 / kSegRows;
  constexpr int kWloads = kTpw * kDnKs;
  const int r = lane & 15, kg = lane >> 4;
  // the pair (y row) of each of this lane's output columns, for the
  // epilogue; loaded now, before the staging loads that the waits count
  int pid[NBK];
#pragma unroll
  for (int nb = 0; nb < NBK; ++nb) {
    const int sl = p0 + nb * 16 + r;
    const int p = sl < cnt ? perm[base + sl] : -1;
    pid[nb] = p >= 0 && p < n_pairs ? p : -1;
  }
  // source offset of this lane's piece of each segment in chunk 0 (out of
  // range past the expert's count), its half and its LDS segment
  uint32_t soff[kSegs];
#pragma unroll
  for (int j = 0; j < kSegs; ++j) {
    const int g = wave + j * kWv;                    // wave-uniform
    const int gh = g < kSegsHalf ? g : g - kSegsHalf;
    const int row = gh * kSegRows + (lane >> 3);
    const int piece = (lane & 7) ^ x_swizzle(row);
    soff[j] = p0 + row < cnt
                  ? ((uint32_t)(base + p0 + row) * I + (uint32_t)piece * 8u) * 2u
                  : kOutOfRange;
  }
  auto stage = [&](int c, int k) {  // chunk c into ring slot k = c % D
    uint16_t* buf = slot(k);
#pragma unroll
    for (int j = 0; j < kSegs; ++j) {
      const int g = wave + j * kWv;
      const bool lo = g >= kSegsHalf;
      const int gh = lo ? g - kSegsHalf : g;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          lo ? hlr : hhr,
          (__attribute__((address_space(3))) void*)(buf + ((lo ? kNT : 0) + gh * kSegRows) * kDnKc),
          16, soff[j] + (uint32_t)c * kDnKc * 2u, 0, 0, 0);
    }
  };
  int bslot[kDnKs];
#pragma unroll
  for (int st = 0; st < kDnKs; ++st) bslot[st] = ((st * 4 + kg) ^ x_swizzle(r)) * 8;

#pragma unroll
  for (int c = 0; c < kAhead; ++c) stage(c, c);
  __builtin_amdgcn_sched_barrier(0);  // the load order the waits below count on
  u32x4 A[D][kTpw][kDnKs];
#pragma unroll
  for (int d = 0; d < kAhead; ++d) {  // in chunk order: the waits assume it
    dn_issue<kTiled>(w, ob, d, nchunks, H, I, lane, A[d]);
    __builtin_amdgcn_sched_barrier(0);
  }
  f32x4 acc[kTpw][NBK];
#pragma unroll
  for (int t = 0; t < kTpw; ++t)
#pragma unroll
    for (int nb = 0; nb < NBK; ++nb) acc[t][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // nchunks is a multiple of D; the waits work as for gate/up
  constexpr int kAfter = (kAhead - 1) * (kSegs + kWloads) + kWloads;
  for (int c0 = 0; c0 < nchunks; c0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int c = c0 + d;
      __builtin_amdgcn_s_waitcnt(vmcnt_at_most_lds_done(kAfter));
      __builtin_amdgcn_s_barrier();
      stage(c + kAhead, (d + kAhead) % D);
      __builtin_amdgcn_sched_barrier(0);
      dn_issue<kTiled>(w, ob, c + kAhead, nchunks, H, I, lane, A[(d + kAhead) % D]);
      __builtin_amdgcn_sched_barrier(0);  // loads ahead of the chunk's MFMAs
      const uint16_t* buf = slot(d);
#pragma unroll
      for (int st = 0; st < kDnKs; ++st) {
#pragma unroll
        for (int nb = 0; nb < NBK; ++nb) {
          const uint16_t* row = buf + (nb * 16 + r) * kDnKc + bslot[st];
          const u32x4 bh = *reinterpret_cast<const u32x4*>(row);
          const u32x4 bl = *reinterpret_cast<const u32x4*>(row + kNT * kDnKc);
#pragma unroll
          for (int t = 0; t < kTpw; ++t) {
            acc[t][nb] = mfma_16x16x32(A[d][t][st], bh, acc[t][nb]);
            acc[t][nb] = mfma_16x16x32(A[d][t][st], bl, acc[t][nb]);
          }
        }
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_at_most(0));  // the loads past the end landed

  // y rows of the pass's pairs: lane (r, kg) holds output rows
  // ob * 16 + 4 kg .. + 3 of pair pid[nb]
#pragma unroll
  for (int t = 0; t < kTpw; ++t) {
#pragma unroll
    for (int nb = 0; nb < NBK; ++nb) {
      const int o = ob[t] * 16 + kg * 4;
      uint32_t off = kOutOfRange;
      if (ob[t] >= 0 && pid[nb] >= 0) off = ((uint32_t)pid[nb] * H + (uint32_t)o) * 4u;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[t][nb]), yr, off, 0,
                                             0);
    }
  }
}

template <bool kTiled, int D>
__global__ __launch_bounds__(kBlk, 1) void down_prefill_kernel(
    const uint16_t* __restrict__ h_hi, const uint16_t* __restrict__ h_lo,
    const uint16_t* __restrict__ w2, const int* __restrict__ counts,
    const int* __restrict__ offsets, const int* __restrict__ perm,
    const int* __restrict__ active, const int* __restrict__ n_active_p, float* __restrict__ y,
    int H, int I, int m, int n_pairs) {
  // the h ring: four slots of hi rows then lo rows
  __shared__ __attribute__((aligned(1024))) uint16_t hs0[2 * kNT * kDnKc];
  __shared__ __attribute__((aligned(1024))) uint16_t hs1[2 * kNT * kDnKc];
  __shared__ __attribute__((aligned(1024))) uint16_t hs2[2 * kNT * kDnKc];
  __shared__ __attribute__((aligned(1024))) uint16_t hs3[2 * kNT * kDnKc];
  const int n_act = *n_active_p;
  if (n_act <= 0 || n_act > m) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int tpe = H / 16;
  const int gpe = (tpe + kTpu - 1) / kTpu;
  const int nchunks = I / kDnKc;
  const auto yr = make_rsrc(y, 4u * (uint32_t)n_pairs * (uint32_t)H);
  const uint32_t hbytes = 2u * (uint32_t)n_pairs * (uint32_t)I;
  const auto hhr = make_rsrc(h_hi, hbytes);
  const auto hlr = make_rsrc(h_lo, hbytes);

  for (int u = unit_slot(); u < n_act * gpe; u += gridDim.x) {
    const Unit s = unit_of(u, gpe, active, counts, offsets, m, n_pairs);
    if (!s.ok) continue;
    const auto w = make_rsrc(w2 + (size_t)s.e * H * I, 2u * (uint32_t)H * (uint32_t)I);
    int ob[kTpw];
#pragma unroll
    for (int t = 0; t < kTpw; ++t) {
      const int tile = s.grp * kTpu + wave * kTpw + t;
      ob[t] = tile < tpe ? tile : -1;
    }

    for (int p0 = 0; p0 < s.cnt; p0 += kNT) {
      const int nbn = (min(kNT, s.cnt - p0) + 15) >> 4;
      __syncthreads();  // the previous pass's reads of the ring are done
      with_blocks(nbn, [&](auto nbk) {
        dn_pass<kTiled, D, decltype(nbk)::value>(w, hhr, hlr, ob, perm, n_pairs, hs0, hs1, hs2,
                                                 hs3, yr, s.base, p0, s.cnt, H, I, nchunks, lane,
                                                 wave);
      });
    }
  }
}

int prefill_grid() {
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    cus = 256;
  return cus;
}

}  // namespace

bool prefill_supported(int T, int H, int I, int m, int k) {
  // 16 or more pairs per expert on average over a pool large enough to
  // spread its units over the chip, K in whole rounds of the pipelines (H
  // and I multiples of 128), and 32-bit offsets.  From 16 pairs an expert
  // on, its 160-token passes beat the decode kernels' 32-token ones
  // (measured on the 256-expert layer at H 2048, I 512: batch 256 over 64
  // kept experts 146 -> 100 us a step, gate/up at 5.5 instead of 3.1 TB/s;
  // batch 128 over 64 and batch 256 over 128, 4-6 us faster); at 8 a
  // decode step is faster on the decode kernels.
  return m >= 16 && (int64_t)T * k >= (int64_t)16 * m && H % (kDepth * kGuKc) == 0 &&
         I % (kDepth * kDnKc) == 0 &&
         H <= 32768 && 4 * (int64_t)T * k * H < ((int64_t)1 << 31);
}

hipError_t launch_gate_up_prefill(const uint16_t* x, int T, const uint16_t* w13, bool tiled,
                                  const int* counts, const int* offsets, const int* perm,
                                  const int* active, const int* n_active, int H, int I, int m,
                                  int k, uint16_t* h_hi, uint16_t* h_lo, hipStream_t stream) {
  if (tiled)
    gate_up_prefill_kernel<true, kDepth><<<prefill_grid(), kBlk, 0, stream>>>(
        x, w13, counts, offsets, perm, active, n_active, h_hi, h_lo, H, I, m, k, T * k);
  else
    gate_up_prefill_kernel<false, kDepth><<<prefill_grid(), kBlk, 0, stream>>>(
        x, w13, counts, offsets, perm, active, n_active, h_hi, h_lo, H, I, m, k, T * k);
  return hipGetLastError();
}

hipError_t launch_down_prefill(int T, const uint16_t* w2, bool tiled, const int* counts,
                               const int* offsets, const int* perm, const int* active,
                               const int* n_active, int H, int I, int m, int k,
                               const uint16_t* h_hi, const uint16_t* h_lo, float* y,
                               hipStream_t stream) {
  if (tiled)
    down_prefill_kernel<true, kDepth><<<prefill_grid(), kBlk, 0, stream>>>(
        h_hi, h_lo, w2, counts, offsets, perm, active, n_active, y, H, I, m, T * k);
  else
    down_prefill_kernel<false, kDepth><<<prefill_grid(), kBlk, 0, stream>>>(
        h_hi, h_lo, w2, counts, offsets, perm, active, n_active, y, H, I, m, T * k);
  return hipGetLastError();
}

}  // namespace sw
