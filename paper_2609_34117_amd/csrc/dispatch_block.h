// Block-level dispatch plan (Section 2.1, Eq. 1: the step reads the union of
// the experts selected across the batch).  From the n_pairs expert ids of a
// batch (pair p = t * k + j), one block of up to 1024 threads builds:
//   counts[e]   pairs per expert,
//   offsets[e]  exclusive prefix sum of counts (offsets[m] = n_pairs),
//   perm        pair indices grouped by expert, ascending within an expert,
//   active      experts with a nonzero count, ascending; n_active of them.
// Any id outside [0, m) flags the batch: counts and offsets are zeroed, perm
// is the identity and n_active = -1.
#pragma once

#include "sw_device.h"

namespace sw {

// LDS of one dispatch_block call, provided by the calling kernel.
struct DispatchLds {
  int* cursor;          // [m] running output position per expert
  int* wave_base;       // [waves * m] start of this chunk's run, per wave and expert
  uint8_t* wave_cnt;    // [waves * m] length of that run
  uint32_t* scan;       // [34] block-scan scratch
  int* bad;             // [1] invalid-id flag
};

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

// Bits needed for an expert id below m.
__device__ __forceinline__ int id_bits(int m) {
  int nbits = 0;
  while ((1 << nbits) < m) ++nbits;
  return nbits;
}

// Stable scatter of the pairs c0 .. c0 + blockDim.x - 1 (those below
// n_pairs) into perm: s.cursor[e] holds the first free slot of expert e and
// is advanced past this chunk's pairs.  Within a wave a pair's rank among
// equal ids comes from a ballot match; across waves the per-expert runs are
// placed in wave order by a column scan over the waves that hold pairs.
// Every thread of the block calls it (it contains barriers); s.wave_cnt must
// be zero on entry and is left zero.
__device__ __forceinline__ void scatter_chunk(const int* ids, int c0, int n_pairs, int m,
                                              int nbits, const DispatchLds& s,
                                              int* __restrict__ perm) {
  const int tid = threadIdx.x, nthr = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int nwaves = nthr >> 6;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  const int p = c0 + tid;
  const bool valid = p < n_pairs;
  const int e = valid ? ids[p] : 0;
  const uint64_t peers = match_peers(e, valid, nbits);
  const int rank = __popcll(peers & lt_mask);
  if (valid && rank == 0) s.wave_cnt[wave * m + e] = static_cast<uint8_t>(__popcll(peers));
  __syncthreads();
  const int used = min(nwaves, (n_pairs - c0 + 63) >> 6);
  for (int ee = tid; ee < m; ee += nthr) {
    int run = s.cursor[ee];
    for (int w = 0; w < used; ++w) {
      s.wave_base[w * m + ee] = run;
      run += s.wave_cnt[w * m + ee];
      s.wave_cnt[w * m + ee] = 0;
    }
    s.cursor[ee] = run;
  }
  __syncthreads();
  if (valid) perm[s.wave_base[wave * m + e] + rank] = p;
}

// Must be called by every thread of the block.  `ids` may live in global
// memory or in LDS (written before a barrier that precedes the call).
__device__ __forceinline__ void dispatch_block(const int* ids, int n_pairs, int m,
                                               const DispatchLds& s, int* __restrict__ counts,
                                               int* __restrict__ offsets, int* __restrict__ perm,
                                               int* __restrict__ active,
                                               int* __restrict__ n_active) {
  const int tid = threadIdx.x, nthr = blockDim.x, nwaves = nthr >> 6;
  if (tid == 0) *s.bad = 0;
  for (int e = tid; e < m; e += nthr) s.cursor[e] = 0;
  for (int i = tid; i < nwaves * m; i += nthr) s.wave_cnt[i] = 0;
  __syncthreads();

  // histogram (integer LDS atomics: order-independent) and id validation
  for (int p = tid; p < n_pairs; p += nthr) {
    const int e = ids[p];
    if (e < 0 || e >= m)
      atomicOr(s.bad, 1);
    else
      atomicAdd(&s.cursor[e], 1);
  }
  __syncthreads();

  if (*s.bad) {
    for (int e = tid; e <= m; e += nthr) {
      if (e < m) counts[e] = 0;
      offsets[e] = 0;
    }
    for (int p = tid; p < n_pairs; p += nthr) perm[p] = p;
    if (tid == 0) *n_active = -1;
    return;
  }

  // offsets = exclusive scan of counts; active = ascending compaction of the
  // experts with a nonzero count (one fused two-value block scan; m <= nthr)
  const uint32_t c = tid < m ? (uint32_t)s.cursor[tid] : 0u;
  uint32_t off, apos, total, n_act;
  block_exclusive_scan2(c, c > 0 ? 1u : 0u, s.scan, &off, &apos, &total, &n_act);
  if (tid < m) {
    counts[tid] = (int)c;
    offsets[tid] = (int)off;
    s.cursor[tid] = (int)off;
    if (c > 0) active[apos] = tid;
  }
  if (tid == 0) {
    offsets[m] = (int)total;
    *n_active = (int)n_act;
  }
  __syncthreads();

  // stable scatter, nthr pairs per chunk in pair order
  const int nbits = id_bits(m);
  for (int c0 = 0; c0 < n_pairs; c0 += nthr) scatter_chunk(ids, c0, n_pairs, m, nbits, s, perm);
}

}  // namespace sw
