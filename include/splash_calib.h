/* libsplash_calib: measurement helpers used by the benchmark to report the
 * chip's achievable peaks next to the spec-sheet ones, and to flush the
 * caches between cold timed steps.  Not part of the attention path.
 *
 * All pointers are device pointers owned by the caller; every call only
 * enqueues one kernel on `stream` (a hipStream_t, NULL for the default
 * stream) and never synchronises.  Return: 0 on success, -1 for a bad
 * argument (NULL pointer, count below 1, pointer not 16-byte aligned), -5 if
 * the launch failed.
 */
#ifndef SPLASH_CALIB_H
#define SPLASH_CALIB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` (a multiple of 16) of `buf` once with `blocks` workgroups of
 * 256 threads (grid-stride, non-temporal 16-byte loads, four in flight per
 * lane).  `sink` receives one 32-bit word per thread: blocks * 1024 bytes.
 * Used for the streaming-read peak and as a clean cache flush (no dirty
 * lines are left behind). */
int splash_calib_stream_read(const void* buf, size_t bytes, void* sink, int32_t blocks, void* stream);

/* Bytes of operand data splash_calib_mfma_loop reads: 8 bf16x8 fragments per
 * thread. */
size_t splash_calib_mfma_ops_bytes(int32_t blocks);

/* `iters` rounds of 16 v_mfma_f32_32x32x16_bf16 per wave in four independent
 * accumulation chains, operands from `ops` (splash_calib_mfma_ops_bytes
 * bytes, bf16).  `sink`: one float per thread (blocks * 1024 bytes). */
int splash_calib_mfma_loop(const void* ops, int32_t iters, void* sink, int32_t blocks, void* stream);

/* Flops of one splash_calib_mfma_loop launch. */
double splash_calib_mfma_flops(int32_t blocks, int32_t iters);

#ifdef __cplusplus
}
#endif

#endif /* SPLASH_CALIB_H */
