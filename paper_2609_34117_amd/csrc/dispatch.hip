// Dispatch plan of a decode step on gfx950 (Section 2.1: the step reads the
// union of the experts selected across the batch): the histogram of the
// selected expert ids, its exclusive scan, the active-expert list and the
// stable permutation that groups pairs by expert.
//
// Up to kSingleBlockPairs pairs, one block builds everything (1024 threads,
// or 512 for at most 512 pairs over at most 512 experts).
// Larger batches (prefill) split the pairs into 1024-pair chunks, one block
// each, in two launches:
//   1. per-chunk histograms (and id validation);
//   2. every chunk's block adds the histograms up per expert, scans the
//      totals (block 0 writes counts / offsets / active from them), and
//      scatters its pairs in pair order from offsets[e] plus the counts of e
//      in the earlier chunks.
// The result is identical to the single block's: chunk c's pairs of expert e
// land after those of chunks 0 .. c-1, each chunk in pair order.
#include "dispatch_block.h"
#include "sw_launch.h"

namespace sw {
namespace {

constexpr int kDispatchThreads = 1024;
constexpr int kDispatchWaves = kDispatchThreads / kWave;
constexpr int kMaxPool = 1024;
constexpr int kSingleBlockPairs = 2048;

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

// Scratch of the chunked dispatch (inside the caller's workspace).
struct ChunkScratch {
  int* hist;  // [n_chunks][m] per-chunk histograms
  int* bad;   // [n_chunks] invalid id seen in the chunk
};

int n_chunks_of(int n_pairs) { return (n_pairs + kDispatchThreads - 1) / kDispatchThreads; }

ChunkScratch carve_chunks(void* ws, int n_pairs, int m) {
  char* p = static_cast<char*>(ws);
  ChunkScratch s;
  s.hist = reinterpret_cast<int*>(p);
  p += align_up((size_t)n_chunks_of(n_pairs) * m * 4, 256);
  s.bad = reinterpret_cast<int*>(p);
  return s;
}

__global__ __launch_bounds__(kDispatchThreads) void dispatch_count_kernel(
    const int* __restrict__ ids, int n_pairs, int m, int* __restrict__ hist_out,
    int* __restrict__ bad_out) {
  __shared__ int hist[kMaxPool];
  __shared__ int bad;
  const int tid = threadIdx.x;
  if (tid == 0) bad = 0;
  for (int e = tid; e < m; e += kDispatchThreads) hist[e] = 0;
  __syncthreads();
  const int p = blockIdx.x * kDispatchThreads + tid;
  if (p < n_pairs) {
    const int e = ids[p];
    if (e < 0 || e >= m)
      atomicOr(&bad, 1);
    else
      atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  for (int e = tid; e < m; e += kDispatchThreads) hist_out[(size_t)blockIdx.x * m + e] = hist[e];
  if (tid == 0) bad_out[blockIdx.x] = bad;
}

// Chunk b = blockIdx.x: expert e's total over all chunks and over the chunks
// before b (thread e, eight loads in flight at a time), the block scan of
// the totals, and the stable scatter of the chunk from offsets[e] plus the
// earlier chunks' count.  Block 0 also writes counts, offsets, active and
// n_active.
__global__ __launch_bounds__(kDispatchThreads) void dispatch_scatter_kernel(
    const int* __restrict__ ids, int n_pairs, int m, int n_chunks, const int* __restrict__ hist,
    const int* __restrict__ bad_in, int* __restrict__ counts, int* __restrict__ offsets,
    int* __restrict__ perm, int* __restrict__ active, int* __restrict__ n_active) {
  __shared__ int cursor[kMaxPool];
  __shared__ int wave_base[kDispatchWaves * kMaxPool];
  __shared__ uint8_t wave_cnt[kDispatchWaves * kMaxPool];
  __shared__ uint32_t scan_scratch[34];
  const int tid = threadIdx.x, b = blockIdx.x, c0 = b * kDispatchThreads;
  int any_bad = 0;
  for (int c = tid; c < n_chunks; c += kDispatchThreads) any_bad |= bad_in[c];
  if (__syncthreads_or(any_bad)) {  // an invalid id: perm is the identity
    if (c0 + tid < n_pairs) perm[c0 + tid] = c0 + tid;
    if (b == 0) {
      for (int e = tid; e <= m; e += kDispatchThreads) {
        if (e < m) counts[e] = 0;
        offsets[e] = 0;
      }
      if (tid == 0) *n_active = -1;
    }
    return;
  }
  uint32_t total = 0, before = 0;
  if (tid < m) {
    const int* col = hist + tid;
    int ch = 0;
    for (; ch + 8 <= n_chunks; ch += 8) {
      int v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = col[(size_t)(ch + j) * m];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        total += (uint32_t)v[j];
        before += ch + j < b ? (uint32_t)v[j] : 0u;
      }
    }
    for (; ch < n_chunks; ++ch) {
      const uint32_t v = (uint32_t)col[(size_t)ch * m];
      total += v;
      before += ch < b ? v : 0u;
    }
  }
  uint32_t off, apos, sum, n_act;
  block_exclusive_scan2(total, total > 0 ? 1u : 0u, scan_scratch, &off, &apos, &sum, &n_act);
  if (tid < m) cursor[tid] = (int)(off + before);
  for (int i = tid; i < kDispatchWaves * m; i += kDispatchThreads) wave_cnt[i] = 0;
  if (b == 0) {
    if (tid < m) {
      counts[tid] = (int)total;
      offsets[tid] = (int)off;
      if (total > 0) active[apos] = tid;
    }
    if (tid == 0) {
      offsets[m] = (int)sum;
      *n_active = (int)n_act;
    }
  }
  __syncthreads();
  const DispatchLds lds{cursor, wave_base, wave_cnt, nullptr, nullptr};
  scatter_chunk(ids, c0, n_pairs, m, id_bits(m), lds, perm);
}

}  // namespace

size_t dispatch_workspace_bytes(int n_pairs, int m) {
  if (n_pairs <= kSingleBlockPairs) return 0;
  const int nc = n_chunks_of(n_pairs);
  return align_up((size_t)nc * m * 4, 256) + align_up((size_t)nc * 4, 256);
}

hipError_t launch_dispatch(const int* topk_ids, int n_pairs, int m, int* counts, int* offsets,
                           int* perm, int* active, int* n_active, hipStream_t stream,
                           void* workspace) {
  if (workspace == nullptr || n_pairs <= kSingleBlockPairs) {
    // half the block when one 512-pair chunk and the expert scan fit in it
    // (0.5 us a batch-64 step faster: the plan's barriers and LDS clearing
    // cover half the waves)
    const int threads = (n_pairs <= 512 && m <= 512) ? 512 : kDispatchThreads;
    dispatch_kernel<<<1, threads, 0, stream>>>(topk_ids, n_pairs, m, counts, offsets, perm, active,
                                               n_active);
    return hipGetLastError();
  }
  const int nc = n_chunks_of(n_pairs);
  const ChunkScratch s = carve_chunks(workspace, n_pairs, m);
  dispatch_count_kernel<<<nc, kDispatchThreads, 0, stream>>>(topk_ids, n_pairs, m, s.hist, s.bad);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  dispatch_scatter_kernel<<<nc, kDispatchThreads, 0, stream>>>(
      topk_ids, n_pairs, m, nc, s.hist, s.bad, counts, offsets, perm, active, n_active);
  return hipGetLastError();
}

}  // namespace sw
