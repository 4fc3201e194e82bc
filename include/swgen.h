/*
 * swgen.h -- device draws of synthetic inputs (libswgen.so).
 *
 * Not part of the MoE layer: a fill routine for expert pools too large to
 * draw on the host and upload (the 40-layer, 60 GiB skewed stack).  It
 * implements the counter-based stream the host side also implements, so
 * the host can redraw any element range of a device-drawn tensor to check
 * results against.
 *
 * Element i of a tensor takes the Philox4x64-10 block (Salmon, Moraes,
 * Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011)
 * of counter (i + 1, 0, 0, 0) under the 128-bit key (key0, key1).  The
 * twelve 16-bit halves of the block's first three 64-bit words (low half
 * first) are summed, S, and the element is
 *     bf16_rne( float32(S - 393210) * float32(std / 65536) )
 * -- a sum of 12 uniform integers (Irwin-Hall) scaled to ~N(0, std), cut
 * at +-6 std.
 */
#pragma once

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Writes elements start .. start + n - 1 of the tensor with key (key0, key1)
 * to dst[0 .. n-1] (device pointer, bf16 bits, 2-byte aligned), enqueued on
 * `stream` (a hipStream_t; NULL = the default stream).  The caller owns dst.
 * Returns 0, or a HIP error code (1 for a NULL dst with n > 0).
 */
int swg_philox_normal_bf16(uint16_t* dst, uint64_t n, uint64_t key0, uint64_t key1,
                           uint64_t start, float std_dev, void* stream);

#ifdef __cplusplus
}
#endif
