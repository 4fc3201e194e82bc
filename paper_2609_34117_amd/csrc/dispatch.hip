// Dispatch plan of a decode step on gfx950 (Section 2.1: the step reads the
// union of the experts selected across the batch).  One 1024-thread block
// builds the histogram, its exclusive scan, the active-expert list and the
// stable permutation that groups pairs by expert.
#include "sw_device.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kDispatchThreads = 1024;
constexpr int kDispatchWaves = kDispatchThreads / kWave;
constexpr int kMaxPool = 1024;

// Lanes of the wave whose `key` equals this lane's (only lanes with `valid`
// take part): one ballot per key bit.
__device__ __forceinline__ uint64_t match_peers(int key, bool valid, int nbits) {
  uint64_t peers = __ballot(valid);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (key >> b) & 1;
    const uint64_t ones = __ballot(valid && bit);
    peers &= bit ? ones : ~ones;
  }
  return peers;
}

__global__ __launch_bounds__(kDispatchThreads) void dispatch_kernel(
    const int* __restrict__ ids, int n_pairs, int m, int* __restrict__ counts,
    int* __restrict__ offsets, int* __restrict__ perm, int* __restrict__ active,
    int* __restrict__ n_active) {
  __shared__ int cursor[kMaxPool];                        // running output position per expert
  __shared__ int wave_base[kDispatchWaves * kMaxPool];    // [wave][e]: this chunk's run start
  __shared__ uint8_t wave_cnt[kDispatchWaves * kMaxPool]; // [wave][e]: this chunk's run length
  __shared__ uint32_t scan_scratch[34];
  __shared__ int bad;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) bad = 0;
  if (tid < m) cursor[tid] = 0;
  for (int i = tid; i < kDispatchWaves * m; i += kDispatchThreads) wave_cnt[i] = 0;
  __syncthreads();

  // histogram (integer LDS atomics: order-independent) and id validation
  for (int p = tid; p < n_pairs; p += kDispatchThreads) {
    const int e = ids[p];
    if (e < 0 || e >= m)
      atomicOr(&bad, 1);
    else
      atomicAdd(&cursor[e], 1);
  }
  __syncthreads();

  if (bad) {
    for (int e = tid; e <= m; e += kDispatchThreads) {
      if (e < m) counts[e] = 0;
      offsets[e] = 0;
    }
    for (int p = tid; p < n_pairs; p += kDispatchThreads) perm[p] = p;
    if (tid == 0) *n_active = -1;
    return;
  }

  // offsets = exclusive scan of counts; active = ascending compaction of
  // the experts with a nonzero count (one fused two-value block scan)
  const uint32_t c = tid < m ? (uint32_t)cursor[tid] : 0u;
  uint32_t off, apos, total, n_act;
  block_exclusive_scan2(c, c > 0 ? 1u : 0u, scan_scratch, &off, &apos, &total, &n_act);
  if (tid < m) {
    counts[tid] = (int)c;
    offsets[tid] = (int)off;
    cursor[tid] = (int)off;
    if (c > 0) active[apos] = tid;
  }
  if (tid == 0) {
    offsets[m] = (int)total;
    *n_active = (int)n_act;
  }
  __syncthreads();

  // stable scatter, 1024 pairs per chunk in pair order: within a wave a
  // pair's rank among equal ids comes from a ballot match; across waves the
  // per-expert runs are placed in wave order by a column scan.
  int nbits = 0;
  while ((1 << nbits) < m) ++nbits;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int c0 = 0; c0 < n_pairs; c0 += kDispatchThreads) {
    const int p = c0 + tid;
    const bool valid = p < n_pairs;
    const int e = valid ? ids[p] : 0;
    const uint64_t peers = match_peers(e, valid, nbits);
    const int rank = __popcll(peers & lt_mask);
    if (valid && rank == 0) wave_cnt[wave * m + e] = static_cast<uint8_t>(__popcll(peers));
    __syncthreads();
    if (tid < m) {
      int run = cursor[tid];
      for (int w = 0; w < kDispatchWaves; ++w) {
        wave_base[w * m + tid] = run;
        run += wave_cnt[w * m + tid];
        wave_cnt[w * m + tid] = 0;
      }
      cursor[tid] = run;
    }
    __syncthreads();
    if (valid) perm[wave_base[wave * m + e] + rank] = p;
  }
}

}  // namespace

hipError_t launch_dispatch(const int* topk_ids, int n_pairs, int m, int* counts, int* offsets,
                           int* perm, int* active, int* n_active, hipStream_t stream) {
  dispatch_kernel<<<1, kDispatchThreads, 0, stream>>>(topk_ids, n_pairs, m, counts, offsets, perm,
                                                      active, n_active);
  return hipGetLastError();
}

}  // namespace sw
