/*
 * dartree_calib.h - calibration kernels of libdartree.
 *
 * Three kernels with a known amount of work that give the achievable
 * ceilings the construction kernels are measured against (on MI355X the spec
 * figures are 8 TB/s of HBM3E and 2.5 PFLOP/s of dense bf16 MFMA):
 *   - a streaming read (the access pattern of the vocabulary projection,
 *     which reads every row of U once per depth),
 *   - a plain device-to-device copy (also the known-size reference that
 *     converts hardware byte counters into bytes),
 *   - a register-only loop of bf16 matrix-core instructions on pseudo-random
 *     operands (the sustained matrix-core rate depends on the operand bits:
 *     power limits the clock, and random operands draw the most).
 * Two more price the ways kernels of one round can hand data to each other:
 * the boundary between consecutive launches, and a grid-wide barrier inside
 * one launch (the alternative of a single persistent kernel per round).
 * They compute nothing of the method.  Conventions as in dartree.h: caller-
 * owned device memory, work enqueued on `stream`, arguments validated before
 * anything is enqueued (DARTREE_ERR_INVALID_ARG otherwise).
 */
#ifndef DARTREE_CALIB_H
#define DARTREE_CALIB_H

#include "dartree.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Number of floats `sink` must hold for dartree_calib_read and
 * dartree_calib_mfma (one partial result per workgroup). */
#define DARTREE_CALIB_SINK_FLOATS 4096

/* Reads `bytes` bytes at `src` once with 16-byte non-temporal loads and
 * writes one partial sum per workgroup to sink[0 .. DARTREE_CALIB_SINK_FLOATS).
 * src: device, 16-byte aligned; bytes: > 0, a multiple of 16. */
dartree_status dartree_calib_read(const void* src, size_t bytes, float* sink, hipStream_t stream);

/* dst[0 .. bytes) = src[0 .. bytes) with 16-byte loads and stores.
 * dst, src: device, 16-byte aligned, not overlapping; bytes: > 0, a multiple of 16. */
dartree_status dartree_calib_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);

/* `iters` rounds of 64 independent 16x16x32 bf16 matrix-core products (fp32
 * accumulate, an 8 x 8 grid of accumulators) in every wave of `blocks`
 * workgroups of 256 threads (one wave per SIMD at 256 workgroups).  Total work:
 *   blocks * 4 waves * iters * 64 * (2 * 16 * 16 * 32) flop.
 * Writes one value per workgroup to sink so the work is not eliminated.
 * blocks: 1 .. DARTREE_CALIB_SINK_FLOATS; iters: >= 1. */
dartree_status dartree_calib_mfma(int32_t blocks, int32_t iters, float* sink, hipStream_t stream);

/* Most barriers one dartree_calib_grid_barrier call passes. */
#define DARTREE_CALIB_MAX_BARRIERS 64

/* One kernel of `blocks` workgroups of 1024 threads that does nothing (a
 * graph of such launches prices the boundary between consecutive kernels).
 * blocks: 1 .. DARTREE_CALIB_SINK_FLOATS. */
dartree_status dartree_calib_empty(int32_t blocks, hipStream_t stream);

/* One kernel of `blocks` workgroups of 1024 threads passing `nbar` grid-wide
 * barriers: at barrier i every workgroup adds 1 to counters[i] (device-scope
 * atomic after a release fence) and polls it (relaxed loads, then an acquire
 * fence) until it reads `blocks`.  blocks: 1 .. the current device's number
 * of compute units, so that every workgroup is resident at once; nbar: 0 ..
 * DARTREE_CALIB_MAX_BARRIERS.  counters: device, nbar words the caller set to
 * zero beforehand.  A wait gives up after about 2^22 polls and sets *fail to
 * 1 (device word; left unchanged otherwise), so the kernel always ends. */
dartree_status dartree_calib_grid_barrier(int32_t blocks, int32_t nbar, uint32_t* counters, uint32_t* fail,
                                          hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DARTREE_CALIB_H */
