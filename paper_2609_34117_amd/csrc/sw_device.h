// Device helpers shared by the gfx950 kernels of libslimwise.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

// 128-bit global load of 8 bf16 (16-byte aligned).
__device__ __forceinline__ u32x4 ld128(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// 128-bit streaming load: data read once per call (expert weights), so
// mark it non-temporal and keep L2 for activations.
__device__ __forceinline__ u32x4 ld128_stream(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Buffer resources: a 128-bit descriptor (base, byte size) with hardware
// range checking.  A load whose byte offset lies outside the buffer returns
// zeros and a store there is dropped, so per-lane predicates become an
// out-of-range offset instead of a branch.
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;  // gfx9-family descriptor word 3
constexpr int kGlc = 1, kNonTemporal = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

__device__ __forceinline__ u32x4 buf_ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// Streaming variant for data read once per call (expert weights).
__device__ __forceinline__ u32x4 buf_ld128_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal);
}

__device__ __forceinline__ uint32_t buf_ld32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}

// D = A(16x32) * B(32x16) + C on the bf16 matrix cores, fp32 accumulate.
// Lane l supplies A row (l % 16), B column (l % 16), and the 8-wide k-group
// (l / 16) of both; D row 4*(l/16)+i, column l%16 lands in D[i].
__device__ __forceinline__ f32x4 mfma_16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16 with round-to-nearest-even (NaN stays NaN, quieted): gfx950's
// conversion instruction, which rounds exactly like adding 0x7fff plus the
// kept lsb to the bits and truncating (checked bit for bit against that
// formula on 2^24 inputs: every exponent, the halfway cases, denormals,
// infinities and NaN payloads).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// Two fp32 values rounded to bf16 in one instruction, a in the low half.
__device__ __forceinline__ uint32_t bf16x2_of(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// SiLU(g) * u in fp32: the expert FFN's activation (the experts of Section
// 2.1 read as SwiGLU FFNs, gate rows first in W13), silu(g) = g / (1 + e^-g).  exp(-g)
// is the hardware base-2 exponential of -g log2(e), with the rounding error
// of that product put back to first order (an FMA residual, times ln 2);
// 1 / (1 + exp(-g)) is the hardware reciprocal.  A few ulp from the exact
// value, for a third of the instructions of expf and an IEEE division.  g is
// clamped to [-88, 88] inside the exponential only: beyond, 1 + exp(-g) is
// either 1 or so large that the product is below 1e-36.  Contraction is off
// and the FMAs are explicit, so every kernel that inlines this (and the
// split below) rounds the same way: the paths agree bit for bit.
__device__ __forceinline__ float swiglu(float g, float u) {
#pragma clang fp contract(off)
  constexpr float kL2e = 1.44269502162933349609375f;  // log2(e) rounded to fp32
  constexpr float kL2eLo = 1.9259629911266175e-08f;   // log2(e) - kL2e
  constexpr float kLn2 = 0.693147180559945309f;
  const float gc = __builtin_amdgcn_fmed3f(g, -88.0f, 88.0f);
  const float t = -gc * kL2e;
  const float r = fmaf(-gc, kL2eLo, fmaf(-gc, kL2e, -t));  // -gc log2(e) - t
  const float den = fmaf(__builtin_amdgcn_exp2f(t), fmaf(r, kLn2, 1.0f), 1.0f);
  return g * __builtin_amdgcn_rcpf(den) * u;
}

// Four fp32 values as bf16 pairs v = hi + lo (hi = v rounded to nearest
// even, lo = the remainder, exact in fp32, rounded likewise), packed two a
// word in order.
__device__ __forceinline__ void split_bf16x4(const float (&v)[4], u32x2& hi, u32x2& lo) {
#pragma clang fp contract(off)
  hi = u32x2{bf16x2_of(v[0], v[1]), bf16x2_of(v[2], v[3])};
  const float h0 = __uint_as_float(hi[0] << 16), h1 = __uint_as_float(hi[0] & 0xffff0000u);
  const float h2 = __uint_as_float(hi[1] << 16), h3 = __uint_as_float(hi[1] & 0xffff0000u);
  lo = u32x2{bf16x2_of(v[0] - h0, v[1] - h1), bf16x2_of(v[2] - h2, v[3] - h3)};
}

// Monotone map from fp32 to uint32 (a < b  <=>  key(a) < key(b) for
// non-NaN values; -0 and +0 share a key).
__device__ __forceinline__ uint32_t f32_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float f32_from_order_key(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m);
  const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Wave-wide reductions with DPP lane moves: swaps within quads, mirrors
// within 8- and 16-lane rows, then the row broadcasts of lanes 15 and 31;
// lane 63 ends with the total, which is returned to every lane.  Each step
// is one cross-lane ALU move, far cheaper than an LDS-crossbar shuffle.
namespace dpp {
constexpr int kXor1 = 0xb1;         // quad_perm [1,0,3,2]
constexpr int kXor2 = 0x4e;         // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141;  // row_half_mirror
constexpr int kMirror = 0x140;      // row_mirror
constexpr int kBcast15 = 0x142;     // row_bcast:15
constexpr int kBcast31 = 0x143;     // row_bcast:31
}  // namespace dpp

template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t identity, uint32_t v) {
  return __builtin_amdgcn_update_dpp(identity, v, CTRL, ROW_MASK, 0xf, false);
}

template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v, uint32_t identity, Op op) {
  v = op(v, dpp_mov<dpp::kXor1>(identity, v));
  v = op(v, dpp_mov<dpp::kXor2>(identity, v));
  v = op(v, dpp_mov<dpp::kHalfMirror>(identity, v));
  v = op(v, dpp_mov<dpp::kMirror>(identity, v));
  v = op(v, dpp_mov<dpp::kBcast15, 0xa>(identity, v));
  v = op(v, dpp_mov<dpp::kBcast31, 0xc>(identity, v));
  return __builtin_amdgcn_readlane(v, 63);
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  return wave_reduce_u32(v, 0u, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  return wave_reduce_u32(v, 0xffffffffu, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
}

__device__ __forceinline__ float wave_sum_f32(float v) {
  const uint32_t r = wave_reduce_u32(__float_as_uint(v), 0u, [](uint32_t a, uint32_t b) {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  });
  return __uint_as_float(r);
}

// Inclusive prefix sum over the 64 lanes with DPP: Hillis-Steele shifts
// inside each 16-lane row, then the row broadcasts carry row totals upward.
__device__ __forceinline__ uint32_t wave_inclusive_scan_u32(uint32_t v) {
  v += dpp_mov<0x111>(0u, v);  // row_shr:1
  v += dpp_mov<0x112>(0u, v);  // row_shr:2
  v += dpp_mov<0x114>(0u, v);  // row_shr:4
  v += dpp_mov<0x118>(0u, v);  // row_shr:8
  v += dpp_mov<dpp::kBcast15, 0xa>(0u, v);
  v += dpp_mov<dpp::kBcast31, 0xc>(0u, v);
  return v;
}

// Work-tile mapping for memory-streaming grids.  Blocks are dispatched
// round-robin over the eight XCDs (block b runs on XCD b % 8); each XCD is
// given one contiguous range of the `valid` tiles, so tiles that read the
// same activations share one XCD's L2.  Returns -1 for surplus blocks.
__device__ __forceinline__ int xcd_tile(int bid, int valid) {
  const int xcd = bid & 7, j = bid >> 3;
  const int per = (valid + 7) >> 3;
  const int tile = xcd * per + j;
  return (j < per && tile < valid) ? tile : -1;
}

// Exclusive prefix sums of two values over a block of blockDim.x (a
// multiple of 64, <= 1024) threads.  `scratch` holds >= 34 uint32 of LDS.
// Returns the prefixes in *pa / *pb and the block totals in *ta / *tb.
// Must be called by every thread of the block.
__device__ __forceinline__ void block_exclusive_scan2(uint32_t a, uint32_t b, uint32_t* scratch,
                                                      uint32_t* pa, uint32_t* pb, uint32_t* ta,
                                                      uint32_t* tb) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const uint32_t ia = wave_inclusive_scan_u32(a), ib = wave_inclusive_scan_u32(b);
  if (lane == 63) {
    scratch[wave] = ia;
    scratch[16 + wave] = ib;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t ra = 0, rb = 0;
    for (int w = 0; w < nwaves; ++w) {
      const uint32_t ca = scratch[w], cb = scratch[16 + w];
      scratch[w] = ra;
      scratch[16 + w] = rb;
      ra += ca;
      rb += cb;
    }
    scratch[32] = ra;
    scratch[33] = rb;
  }
  __syncthreads();
  *pa = scratch[wave] + ia - a;
  *pb = scratch[16 + wave] + ib - b;
  *ta = scratch[32];
  *tb = scratch[33];
  __syncthreads();
}

}  // namespace sw
