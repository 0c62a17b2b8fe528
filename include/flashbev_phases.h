/*
 * flashbev_phases.h -- phase clocks of the fused Sampling-VT forward and the
 * FlashSCA backward (measurement tool, MI355X / gfx950).
 *
 * libflashbev_phases.so is the operator library of include/flashbev.h and
 * include/flashsca.h built once more with the phase clocks of the forward and
 * of the FlashSCA backward compiled in; it is not the operator's library
 * (libflashbev.so has no clock).  In
 * it, lane 0 of every wavefront of the forward kernel records the 100 MHz
 * real-time counter (s_memrealtime) at its start, after it has staged the
 * camera matrices and heights (and the workgroup barrier), after the
 * workgroup barrier that precedes the output stores, and at its end, and
 * the counter ticks it spent in each phase of the Sec. 3.3 / Alg. 2 path:
 * projection and masking (with the culling test and, where the packed pass
 * does both at once, the bilinear set-up), set-up, padding of the sample
 * lists, the gather, and the stash of the group's results in the output
 * tile.  The operator's results are unchanged; the clock costs a few
 * instructions and registers per wavefront.
 *
 * Slots of a wavefront's 16 (unsigned 64-bit): 0 start, 1 staged, 2
 * projection, 3 set-up, 4 padding, 5 gather, 6 stash (2..6 are tick sums),
 * 7 barrier, 8 end, 9 rounds (groups of cells), 10 projection passes,
 * 11 the wavefront's HW_ID register (SIMD, CU, shader array, shader engine)
 * in bits 0..31 and its XCC_ID register (the XCD) in bits 32..63, 12 the
 * valid samples of its groups, 13..15 zero.
 */
#ifndef FLASHBEV_PHASES_H
#define FLASHBEV_PHASES_H

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Where the forward writes the clocks: device memory of at least
 * workgroups * (threads_per_workgroup / 64) * 16 unsigned 64-bit words
 * (flashbev_launch_info gives both figures), written at
 * [(workgroup * waves + wave) * 16 + slot]; NULL stops the recording.  The
 * pointer is kept in a device variable of the current device and applies
 * to every later forward launch there; the caller keeps the memory until
 * it passes NULL.  Returns 0, or -1 if the copy to the device variable
 * fails.
 */
int flashbev_phase_log(void *log);

/*
 * The same for the FlashSCA backward (include/flashsca.h, flashsca_backward;
 * the BEVFormer spatial cross-attention of Sec. 4.5): lane 0 of every
 * wavefront of its kernel sums the real-time counter over the kernel's steps.
 * Memory of at least workgroups * (threads_per_workgroup / 64) * 16 unsigned
 * 64-bit words (flashsca_backward_launch_info), written at
 * [(workgroup * waves + wave) * 16 + slot]; NULL stops the recording.
 * Slots (tick sums unless stated): 0 start (counter), 1 projection of the
 * tile's anchors and hit masks, 2 softmax statistics, output-gradient rows and
 * merge-table set-up, 3 chunk set-up and records, 4 point gradients (tap
 * loads, dot products, sums across the slot), 5 inserts into the merge table,
 * 6 the barrier after the inserts, 7 the walk of the distinct rows with their
 * float atomics, 8 the barrier after the walk, 9 emptying the table, 10
 * chunk-camera steps (count), 11 distinct rows over all steps (count), 12 the
 * tail (offset and logit gradients), 13 end (counter), 14..15 zero.  Returns
 * 0, or -1 if the copy to the device variable fails.
 */
int flashsca_phase_log(void *log);

#ifdef __cplusplus
}
#endif

#endif /* FLASHBEV_PHASES_H */
