// Dispatch plan of a decode step on gfx950 (Section 2.1: the step reads the
// union of the experts selected across the batch).  One 1024-thread block
// builds the histogram, its exclusive scan, the active-expert list and the
// stable permutation that groups pairs by expert.
#include "dispatch_block.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kDispatchThreads = 1024;
constexpr int kDispatchWaves = kDispatchThreads / kWave;
constexpr int kMaxPool = 1024;

__global__ __launch_bounds__(kDispatchThreads) void dispatch_kernel(
    const int* __restrict__ ids, int n_pairs, int m, int* __restrict__ counts,
    int* __restrict__ offsets, int* __restrict__ perm, int* __restrict__ active,
    int* __restrict__ n_active) {
  __shared__ int cursor[kMaxPool];
  __shared__ int wave_base[kDispatchWaves * kMaxPool];
  __shared__ uint8_t wave_cnt[kDispatchWaves * kMaxPool];
  __shared__ uint32_t scan_scratch[34];
  __shared__ int bad;
  const DispatchLds lds{cursor, wave_base, wave_cnt, scan_scratch, &bad};
  dispatch_block(ids, n_pairs, m, lds, counts, offsets, perm, active, n_active);
}

}  // namespace

hipError_t launch_dispatch(const int* topk_ids, int n_pairs, int m, int* counts, int* offsets,
                           int* perm, int* active, int* n_active, hipStream_t stream) {
  dispatch_kernel<<<1, kDispatchThreads, 0, stream>>>(topk_ids, n_pairs, m, counts, offsets, perm,
                                                      active, n_active);
  return hipGetLastError();
}

}  // namespace sw
