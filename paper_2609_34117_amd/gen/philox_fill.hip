// Device draws of synthetic expert weights: Philox4x64-10 (Salmon et al.,
// SC 2011) as a counter-based stream, summed to an Irwin-Hall normal and
// rounded to bf16.  The layout of the stream is documented in swgen.h.
#include <hip/hip_runtime.h>

#include "swgen.h"

namespace {

// Philox4x64 round constants of the published definition: the two
// multipliers and the two key increments (Weyl sequence).
constexpr uint64_t kMul0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kMul1 = 0xCA5A826395121157ull;
constexpr uint64_t kWeyl0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kWeyl1 = 0xBB67AE8584CAA73Bull;
constexpr int kIrwinHallMean = 393210;  // 12 * 65535 / 2
constexpr int kPerThread = 8;           // elements per thread (one 16-byte store)

struct Block4 {
  uint64_t v[4];
};

__device__ __forceinline__ Block4 philox4x64_10(uint64_t c0, uint64_t k0, uint64_t k1) {
  uint64_t c[4] = {c0, 0ull, 0ull, 0ull};
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += kWeyl0;
      k1 += kWeyl1;
    }
    const uint64_t lo0 = kMul0 * c[0], hi0 = __umul64hi(kMul0, c[0]);
    const uint64_t lo1 = kMul1 * c[2], hi1 = __umul64hi(kMul1, c[2]);
    const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
  return Block4{{c[0], c[1], c[2], c[3]}};
}

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ uint16_t element(uint64_t i, uint64_t k0, uint64_t k1, float scale) {
  const Block4 b = philox4x64_10(i + 1ull, k0, k1);
  int s = 0;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int h = 0; h < 4; ++h) s += static_cast<int>((b.v[w] >> (16 * h)) & 0xFFFFull);
  return bf16_rne(static_cast<float>(s - kIrwinHallMean) * scale);
}

__global__ __launch_bounds__(256) void philox_normal_bf16_kernel(uint16_t* __restrict__ dst,
                                                                 uint64_t n, uint64_t k0,
                                                                 uint64_t k1, uint64_t start,
                                                                 float scale) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x * kPerThread;
  for (uint64_t base = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * kPerThread; base < n;
       base += stride) {
    uint16_t v[kPerThread];
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) v[j] = element(start + base + j, k0, k1, scale);
    if (base + kPerThread <= n && (reinterpret_cast<uintptr_t>(dst + base) & 15u) == 0) {
      uint4 w;
      w.x = v[0] | ((uint32_t)v[1] << 16);
      w.y = v[2] | ((uint32_t)v[3] << 16);
      w.z = v[4] | ((uint32_t)v[5] << 16);
      w.w = v[6] | ((uint32_t)v[7] << 16);
      *reinterpret_cast<uint4*>(dst + base) = w;
    } else {
      for (int j = 0; j < kPerThread && base + j < n; ++j) dst[base + j] = v[j];
    }
  }
}

}  // namespace

extern "C" int swg_philox_normal_bf16(uint16_t* dst, uint64_t n, uint64_t key0, uint64_t key1,
                                      uint64_t start, float std_dev, void* stream) {
  if (n == 0) return 0;
  if (dst == nullptr) return 1;
  // std / 65536 is exact (a power-of-two division of an fp32 value)
  const float scale = std_dev / 65536.0f;
  const uint64_t threads = (n + kPerThread - 1) / kPerThread;
  const unsigned blocks = (unsigned)std::min<uint64_t>((threads + 255) / 256, 65536ull);
  (void)hipGetLastError();
  philox_normal_bf16_kernel<<<blocks, 256, 0, static_cast<hipStream_t>(stream)>>>(
      dst, n, key0, key1, start, scale);
  return (int)hipGetLastError();
}
