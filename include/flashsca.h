/*
 * flashsca.h -- C ABI of FlashSCA for AMD MI355X (gfx950): BEVFormer's
 * spatial cross-attention (SCA) with the per-camera sampling points formed on
 * the fly (FlashBEV paper, Sec. 4.5, "Cross-framework applicability",
 * Table 7), forward and backward (the paper states that FlashSCA reproduces
 * the dense path's output and gradient).
 *
 * The operation.  Every BEV query q (cell (i, j) of the grid, q = i Y + j)
 * owns a pillar of Z anchors (x_i, y_j, z_k).  Projected into camera n, an
 * anchor gets normalized image coordinates (u, v); a camera is hit by the
 * query when at least one anchor is valid (positive depth, strictly inside the
 * image).  In each hit camera, head m samples its channels of each level l at
 * P points, point k around the reference point of anchor k mod Z displaced by
 * the learned offset, weighted by the softmax of the query's logits over the
 * head's L * P (level, point) pairs.  For channel c = m D + e (D = C / heads):
 *
 *   out[b,q,c] = 1/max(1, |hit|) * sum_{n hit} sum_{l,k} a[b,q,m,l,k] *
 *                bilinear(value[b,n,l][:,:,c], (u W_l + dx) - 1/2, (v H_l + dy) - 1/2)
 *
 * where (u, v) is the reference point of anchor k mod Z in camera n and
 * (dx, dy) = offsets[b,q,m,l,k].  The dense per-camera formulation
 * materializes a [N X Y, heads, L, P, 2] tensor of sampling locations; this
 * library computes each location in registers where it is used and keeps
 * nothing but the caller's inputs and output in device memory.
 *
 * Conventions fixed by this library (BEVFormer's where it has one):
 *   - anchors: (x_min + (i + 1/2) dx, y_min + (j + 1/2) dy, z_k), z_k from the
 *     caller (host array); point k belongs to anchor k mod Z, so P must be a
 *     multiple of Z;
 *   - projection: (u', v', d) = lidar2img[b,n][0:3] . (x, y, z, 1) in float32
 *     with every product and sum rounded on its own; (u, v) =
 *     (u' / max(d, eps), v' / max(d, eps)) / (img_w, img_h), IEEE divisions,
 *     eps = spec->depth_eps;
 *   - valid anchor: d > eps and 0 < u < 1 and 0 < v < 1 (open interval);
 *   - a hit camera samples the points of all its anchors, valid or not;
 *   - sampling location in level pixels: x = (u W_l + dx) - 1/2 with each
 *     step rounded to float32 (align_corners=False convention), likewise y;
 *     bilinear taps outside the level's map contribute zero;
 *   - attention: softmax over the L P logits of each (query, head), float32;
 *   - reduction: sum over hit cameras divided by max(1, hits) (spec->reduce
 *     = FLASHBEV_REDUCE_VALID_MEAN), or the plain sum (FLASHBEV_REDUCE_SUM);
 *   - accumulation in float32; the output is float32.
 *
 * Thread safety: no state; calls are asynchronous on the given stream and
 * may come from several threads.  No allocation, no printing, no abort.
 * Kernels run on the calling thread's current HIP device, which must hold
 * every buffer of the call and the stream.  A launch that needs more than
 * 64 KiB of LDS per workgroup (many points per head) first raises that
 * kernel's dynamic-LDS limit with hipFuncSetAttribute, a per-process setting
 * that is idempotent.
 */
#ifndef FLASHSCA_H
#define FLASHSCA_H

#include <stdint.h>

#include "flashbev.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Largest number of feature levels, cameras, anchors, and L * P. */
#define FLASHSCA_LMAX 8
#define FLASHSCA_NMAX 32
#define FLASHSCA_ZMAX 32
#define FLASHSCA_LPMAX 512
/* Largest head row (D times the element size) in bytes. */
#define FLASHSCA_HEAD_BYTES_MAX 1024

/* Value maps (BEVFormer's value after its value projection): device memory,
 * [B, N, S, C] in `dtype`, channel-last, S = sum_l level_h[l] level_w[l]
 * with the levels concatenated in order and each level row-major (y, x).
 * Head m owns channels [m D, (m + 1) D), D = C / heads.  Aligned to the
 * element size; one camera's S C elements must be smaller than 2 GiB.
 * img_h x img_w is the image lidar2img projects into. */
typedef struct {
    const void *data;
    int32_t dtype;                      /* flashbev_dtype */
    int32_t B, N, C, heads, L;
    int32_t level_h[FLASHSCA_LMAX];
    int32_t level_w[FLASHSCA_LMAX];
    int32_t img_h, img_w;
} flashsca_value;

/*
 * FlashSCA forward.
 *
 *   value      value maps and image size (see flashsca_value).
 *   lidar2img  device, [B, N, 4, 4] float32 row-major, 4-byte aligned (rows
 *              0..2 are used).
 *   spec       BEV grid of the queries, depth threshold, reduction mode.
 *   anchors    pillar heights (host memory, 1 <= Z <= FLASHSCA_ZMAX).
 *   P          sampling points per (head, level), a multiple of Z;
 *              L * P <= FLASHSCA_LPMAX.
 *   offsets    device, [B, X Y, heads, L, P, 2] float32 (x, y) in pixels of
 *              the point's level, 8-byte aligned (read as pairs).
 *   logits     device, [B, X Y, heads, L, P] float32 attention logits,
 *              4-byte aligned.
 *   out        device, [B, X Y, C] float32, 4-byte aligned, must not overlap
 *              any input.  Every element is written exactly once (queries
 *              no camera sees get +0.0).
 *   stream     hipStream_t; NULL means the default stream.
 *
 * Returns FLASHBEV_OK once enqueued (asynchronous completion) or a negative
 * flashbev_status; argument errors are reported before any HIP call.  An
 * empty output (B, X or Y zero) enqueues nothing.
 */
int flashsca_forward(const flashsca_value *value, const float *lidar2img,
                     const flashbev_bev_grid_spec *spec, const flashbev_z_bins *anchors,
                     int32_t P, const float *offsets, const float *logits, float *out,
                     void *stream);

/*
 * FlashSCA backward: gradients of a loss with respect to the forward's
 * learned inputs, given G = grad_out = dL/d out [B, X Y, C] float32.  With
 * alpha = 1 / max(1, hits) (1 in sum mode), every forward term
 * alpha a w value[b, n, tap, c] of a point (head m, level l, point k) in a
 * hit camera n gives
 *
 *   grad_value[b, n, tap, c]   += alpha a w G[b, q, c]
 *   d a                        += alpha w value[b, n, tap, c] G[b, q, c]
 *   grad_offsets[b, q, m, l, k] += alpha a (dw/dx, dw/dy) value[..] G[..]
 *
 * summed over taps, channels of head m and hit cameras; w is the bilinear
 * weight of the tap, whose derivative is taken on the cell the forward's
 * float32 location falls in (a location moves one pixel per pixel of
 * offset).  grad_logits is the softmax backward over the head's L * P pairs,
 * a_j (d a_j - sum_j' a_j' d a_j').  The camera matrices and anchors get no
 * gradient.  Projection, hits, taps and weights are the forward's, computed
 * the same way.
 *
 *   value, lidar2img, spec, anchors, P, offsets, logits: as in
 *                  flashsca_forward (the value maps are read).
 *   grad_out       device, [B, X Y, C] float32, 4-byte aligned.
 *   grad_value     device, [B, N, S, C] float32 (whatever the value dtype),
 *                  4-byte aligned, or NULL to skip it.  Fully overwritten (a
 *                  fill kernel zeroes it first, on the same stream); terms
 *                  on one value row are summed within a workgroup first and
 *                  the sums added with float32 atomic adds, so the rounding
 *                  order (not the terms) varies from run to run.
 *   grad_offsets   device, [B, X Y, heads, L, P, 2] float32, 8-byte aligned,
 *                  or NULL.  Every element written once (zero for queries no
 *                  camera sees).
 *   grad_logits    device, [B, X Y, heads, L, P] float32, 4-byte aligned, or
 *                  NULL.  Every element written (it holds an intermediate
 *                  until the call's kernel ends).
 *   stream         hipStream_t; NULL means the default stream.
 *
 * At least one gradient must be requested; outputs must not overlap the
 * inputs or each other.  Limits and status codes: those of
 * flashsca_forward.  Returns FLASHBEV_OK once enqueued.
 */
int flashsca_backward(const flashsca_value *value, const float *lidar2img,
                      const flashbev_bev_grid_spec *spec, const flashbev_z_bins *anchors,
                      int32_t P, const float *offsets, const float *logits,
                      const float *grad_out, float *grad_value, float *grad_offsets,
                      float *grad_logits, void *stream);

/*
 * Launch geometry of flashsca_forward for these arguments: workgroups,
 * threads per workgroup, dynamic LDS bytes per workgroup, lanes per
 * (query, head) and bytes each lane loads per tap.  Same checks as the
 * forward; device pointers are not dereferenced and may be NULL; no HIP call.
 */
int flashsca_launch_info(const flashsca_value *value, const flashbev_bev_grid_spec *spec,
                         const flashbev_z_bins *anchors, int32_t P, int64_t *workgroups,
                         int32_t *threads_per_workgroup, int32_t *lds_bytes,
                         int32_t *lanes_per_head, int32_t *lane_bytes);

/* Launch geometry of flashsca_backward (the scatter kernel; the fill kernel
 * is not counted), with the same outputs and checks as flashsca_launch_info. */
int flashsca_backward_launch_info(const flashsca_value *value,
                                  const flashbev_bev_grid_spec *spec,
                                  const flashbev_z_bins *anchors, int32_t P,
                                  int64_t *workgroups, int32_t *threads_per_workgroup,
                                  int32_t *lds_bytes, int32_t *lanes_per_head,
                                  int32_t *lane_bytes);

#ifdef __cplusplus
}
#endif

#endif /* FLASHSCA_H */
