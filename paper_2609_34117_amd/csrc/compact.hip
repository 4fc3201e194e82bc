// Pruned-decoder construction on gfx950 (Section 3.1: keep the top m' experts
// of a layer by importance; the pruned checkpoint holds only those experts
// and their router entries).  Offline: run once per layer, not per step.
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kSelectThreads = 1024;
constexpr int kMaxPool = 1024;

// Rank of expert e = number of experts ordered before it by (importance
// desc, id asc); the ranks are a permutation, so exactly n_keep experts get
// rank < n_keep.  Kept ids are then compacted in ascending order.
__global__ __launch_bounds__(kSelectThreads) void prune_select_kernel(
    const float* __restrict__ importance, int m, int n_keep, int32_t* __restrict__ kept,
    int32_t* __restrict__ remap, uint8_t* __restrict__ keep_mask) {
  __shared__ uint32_t key[kMaxPool];
  __shared__ uint32_t scan_scratch[34];
  const int e = threadIdx.x;
  if (e < m) key[e] = f32_order_key(importance[e]);
  __syncthreads();
  int keep = 0;
  if (e < m) {
    const uint32_t ke = key[e];
    int rank = 0;
    for (int j = 0; j < m; ++j) {
      const uint32_t kj = key[j];
      rank += (kj > ke || (kj == ke && j < e)) ? 1 : 0;
    }
    keep = rank < n_keep ? 1 : 0;
  }
  uint32_t pos, unused_p, total, unused_t;
  block_exclusive_scan2((uint32_t)keep, 0u, scan_scratch, &pos, &unused_p, &total, &unused_t);
  if (e < m) {
    keep_mask[e] = static_cast<uint8_t>(keep);
    remap[e] = keep ? pos : -1;
    if (keep) kept[pos] = e;
  }
}

// Copies `bytes` per expert from src[kept[c]] to dst[c] with 128-bit moves.
// Block (c, chunk); every per-expert block size is a multiple of 16 bytes.
__global__ __launch_bounds__(256) void gather_rows_kernel(const int32_t* __restrict__ kept,
                                                         const char* __restrict__ src,
                                                         char* __restrict__ dst,
                                                         size_t bytes) {
  const int c = blockIdx.y;
  const size_t e = (size_t)kept[c];
  const u32x4* s = reinterpret_cast<const u32x4*>(src + e * bytes);
  u32x4* d = reinterpret_cast<u32x4*>(dst + (size_t)c * bytes);
  const size_t n = bytes / 16;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
    d[i] = s[i];
}

__global__ __launch_bounds__(256) void gather_scalars_kernel(const int32_t* __restrict__ kept,
                                                            int n_keep,
                                                            const float* __restrict__ src,
                                                            float* __restrict__ dst) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c < n_keep) dst[c] = src[kept[c]];
}

hipError_t gather(const int32_t* kept, int n_keep, const void* src, void* dst, size_t bytes,
                  hipStream_t stream) {
  const size_t vecs = bytes / 16;
  const unsigned gx = (unsigned)std::min<size_t>((vecs + 255) / 256, 64);
  dim3 grid(gx, n_keep);
  gather_rows_kernel<<<grid, 256, 0, stream>>>(kept, static_cast<const char*>(src),
                                               static_cast<char*>(dst), bytes);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_prune_select(const float* importance, int m, int n_keep, int32_t* kept,
                               int32_t* remap, uint8_t* keep_mask, hipStream_t stream) {
  prune_select_kernel<<<1, kSelectThreads, 0, stream>>>(importance, m, n_keep, kept, remap,
                                                        keep_mask);
  return hipGetLastError();
}

hipError_t launch_compact_gather(const int32_t* kept, int n_keep, int H, int I,
                                 const uint16_t* w13, const uint16_t* w2, const float* wr,
                                 const float* bias, uint16_t* w13_c, uint16_t* w2_c, float* wr_c,
                                 float* bias_c, hipStream_t stream) {
  hipError_t err = hipSuccess;
  if (w13_c) err = gather(kept, n_keep, w13, w13_c, (size_t)2 * I * H * sizeof(uint16_t), stream);
  if (err == hipSuccess && w2_c)
    err = gather(kept, n_keep, w2, w2_c, (size_t)H * I * sizeof(uint16_t), stream);
  if (err == hipSuccess && wr_c)
    err = gather(kept, n_keep, wr, wr_c, (size_t)H * sizeof(float), stream);
  if (err == hipSuccess && bias_c) {
    gather_scalars_kernel<<<(n_keep + 255) / 256, 256, 0, stream>>>(kept, n_keep, bias, bias_c);
    err = hipGetLastError();
  }
  return err;
}

}  // namespace sw
