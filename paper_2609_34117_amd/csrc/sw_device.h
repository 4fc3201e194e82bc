// Device helpers shared by the gfx950 kernels of libslimwise.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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

// fp32 -> bf16 with round-to-nearest-even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
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

// Exclusive prefix sum over a block of blockDim.x (<= 1024) threads.
// `scratch` holds >= 17 ints of LDS.  Returns the prefix of v and writes the
// block total to *total.  Must be called by every thread of the block.
__device__ __forceinline__ int block_exclusive_scan(int v, int* scratch, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = (blockDim.x + 63) >> 6;
  int incl = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(incl, d);
    if (lane >= d) incl += o;
  }
  if (lane == 63) scratch[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < nwaves; ++w) {
      const int c = scratch[w];
      scratch[w] = run;
      run += c;
    }
    scratch[16] = run;
  }
  __syncthreads();
  const int excl = scratch[wave] + incl - v;
  *total = scratch[16];
  __syncthreads();
  return excl;
}

}  // namespace sw
