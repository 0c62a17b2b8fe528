/*
 * flashbev_membench.h -- memory-ceiling micro-benchmarks for MI355X (gfx950).
 *
 * Measurement tools for the roofline of the fused Sampling-VT forward
 * (include/flashbev.h).  They are not part of the operator: bench.py calls
 * them to measure, on the running GPU, the two ceilings the operator is
 * held against:
 *
 *   - the gather ceiling: wavefronts load 16-byte slices of pixel rows at
 *     pseudo-random positions in a small buffer, four taps (two rows, two
 *     columns) per sample and several cells per wavefront, the access shape
 *     of the bilinear gather-reduce (FlashBEV paper, Sec. 3.3, Alg. 2);
 *     with a buffer of a few MiB it stays in L2, with a few KiB in L1;
 *   - the HBM read ceiling: a coalesced stream of 16-byte loads over a
 *     buffer much larger than every cache;
 *   - the float atomic-add ceiling that bounds the backward's global adds.
 *
 * Both write one float per thread to `sink` (so no load is optimized away)
 * and return 0, or a negative value on bad arguments (checked before any
 * HIP call) or a failed launch.  Every address stays inside `buf`.
 */
#ifndef FLASHBEV_MEMBENCH_H
#define FLASHBEV_MEMBENCH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Gather ceiling.
 *   buf              device buffer of buf_bytes bytes, 16-byte aligned.
 *   row_bytes        bytes per pixel row (multiple of 16, at most 1024).
 *   row_pitch        pixels per image row (the lower taps are row_pitch
 *                    pixels further), at least 1.
 *   iters            samples gathered per cell (a multiple of
 *                    loads_in_flight / 4).
 *   loads_in_flight  16-byte loads a lane issues before it sums them: 8, 16
 *                    or 32 (2, 4 or 8 samples of four taps).
 *   lds_bytes        dynamic LDS per workgroup, 0..65536; it is not used,
 *                    it only limits the workgroups resident per CU (the
 *                    occupancy).
 *   workgroups       workgroups of 256 threads to launch.
 *   sink             device float array of workgroups * 256 entries.
 * First-tap rows follow a linear congruential sequence per cell, masked to
 * the largest power-of-two span that keeps all four taps inside buf.
 * Bytes moved: workgroups * 4 * cells_per_wave * iters * 4 * row_bytes,
 * where cells_per_wave = min(8, 64 / (row_bytes / 16)).
 */
int flashbev_membench_gather(const void *buf, uint64_t buf_bytes, int32_t row_bytes,
                             int32_t row_pitch, int32_t iters, int32_t loads_in_flight,
                             int32_t lds_bytes, int32_t workgroups, float *sink, void *stream);

/*
 * HBM read ceiling: reads all of buf (bytes, a multiple of 16 * 256) once
 * with 16-byte loads spread over `workgroups` workgroups of 256 threads.
 */
int flashbev_membench_stream(const void *buf, uint64_t bytes, int32_t workgroups, float *sink,
                             void *stream);

/*
 * Float atomic-add ceiling: every lane adds 1.0 with a float atomic add
 * (no return value) to `iters` pseudo-random 256-byte rows of buf (buf_floats
 * floats, at least 64, 4-byte aligned; the values change).  Operations:
 * workgroups * 256 * iters.  The backward's per-tile flush and its overflow
 * taps are bound by this rate.
 */
int flashbev_membench_atomic(float *buf, uint64_t buf_floats, int32_t iters, int32_t workgroups,
                             void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FLASHBEV_MEMBENCH_H */
