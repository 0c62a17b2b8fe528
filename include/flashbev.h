/*
 * flashbev.h -- C ABI of the fused Sampling-VT forward for AMD MI355X (gfx950).
 *
 * The operation (FlashBEV paper, Sec. 3.1, Eq. 1): for every batch element
 * b, BEV cell (x, y) and channel c,
 *
 *   out[b,c,x,y] = sum_z ( sum_n M_n(x,y,z) f_n(x,y,z,c) ) / max(1, sum_n M_n(x,y,z))
 *
 * where M_n = 1 when the voxel centre projected through camera n's matrix
 * has positive depth and lands inside camera n's image, and f_n is the
 * bilinear sample of camera n's feature map at that pixel.  The operator is
 * evaluated in one fused pass that never materializes the camera- and
 * height-expanded B x N x C x X x Y x Z tensor (Sec. 3.3, Alg. 2); its only
 * device memory is the caller's inputs and output.
 *
 * Conventions fixed by this library where the paper leaves them open:
 *   - voxel centres: x = x_min + (i + 1/2) dx, y = y_min + (j + 1/2) dy,
 *     heights taken from z_bins (bin centres chosen by the caller);
 *   - projection: (u', v', d) = lidar2img[b,n][0:3] . (x, y, z, 1), pixel
 *     (u, v) = (u'/d, v'/d); coordinates are float32 with every product
 *     and sum rounded on its own and IEEE division;
 *   - valid iff d > depth_eps and 0 <= u < img_w and 0 <= v < img_h;
 *   - feature coordinates x_f = u * (W / img_w) - 1/2 (align_corners=False),
 *     likewise y_f; taps outside the map contribute zero but the sample still
 *     counts in the per-height denominator;
 *   - accumulation in float32 for every input type; the output is float32.
 *
 * Thread safety: calls are asynchronous on the given stream and may be
 * issued from several threads.  The library keeps no per-call state; it
 * remembers, per device and under a lock, how many workgroups of each
 * forward kernel shape fit the GPU at once (HIP's occupancy query, which
 * picks the forward's tile order and tail priorities), and the no-allocation
 * backward holds its static scratch array (below).  It never allocates device
 * or host memory, never prints and never aborts.
 *
 * Device: kernels run on the calling thread's current HIP device, which must
 * hold every buffer of the call and the stream.
 *
 * The one side effect beyond the stream: a launch that needs more than 64 KiB
 * of LDS per workgroup (the backward's tiled mode) first raises that kernel's
 * dynamic-LDS limit with hipFuncSetAttribute, a per-process setting that is
 * idempotent and safe to repeat from several threads.
 */
#ifndef FLASHBEV_H
#define FLASHBEV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FLASHBEV_ABI_VERSION 2
/* Largest number of height bins per call (heights travel as kernel
 * arguments, so they cost no device memory). */
#define FLASHBEV_ZMAX 256
/* Largest number of cameras per batch element. */
#define FLASHBEV_NMAX 64
/* Largest feature row (C times the element size) in bytes. */
#define FLASHBEV_ROW_BYTES_MAX 4096
/* Size of the library's static device scratch (flashbev_sample_vt_backward_noalloc). */
#define FLASHBEV_SCRATCH_BYTES 67108864

/* Status codes.  Every argument check runs before any HIP call. */
typedef enum {
    FLASHBEV_OK = 0,
    FLASHBEV_ERR_NULLPTR = -1,     /* a required pointer is NULL                 */
    FLASHBEV_ERR_SHAPE = -2,       /* a dimension is negative or zero where >= 1 is needed */
    FLASHBEV_ERR_DTYPE = -3,       /* unknown feature dtype                      */
    FLASHBEV_ERR_ALIGN = -4,       /* a device pointer is not element-aligned    */
    FLASHBEV_ERR_UNSUPPORTED = -5, /* beyond a documented limit (Z, N, row, 2 GiB) */
    FLASHBEV_ERR_ALIAS = -6,       /* out overlaps an input                      */
    FLASHBEV_ERR_VALUE = -7,       /* non-finite grid spec or bad reduce mode    */
    FLASHBEV_ERR_HIP = -8,         /* the kernel launch failed                   */
    FLASHBEV_ERR_SCRATCH = -9      /* needs more than FLASHBEV_SCRATCH_BYTES     */
} flashbev_status;

/* Feature element type; accumulation is float32 for all of them. */
typedef enum {
    FLASHBEV_F32 = 0,
    FLASHBEV_F16 = 1,
    FLASHBEV_BF16 = 2
} flashbev_dtype;

/* Reduction over cameras at each height (Eq. 1 uses the valid mean). */
typedef enum {
    FLASHBEV_REDUCE_VALID_MEAN = 0, /* num_z / max(1, den_z), Eq. 1 (default) */
    FLASHBEV_REDUCE_SUM = 1         /* num_z: plain masked sum over cameras   */
} flashbev_reduce;

/* Camera feature maps F_n (Sec. 3.1): device memory, channel-last and
 * contiguous, [B, N, H, W, C] in `dtype`, aligned to the element size.
 * img_h x img_w is the image that lidar2img projects into; the feature map
 * covers it with scale W / img_w horizontally and H / img_h vertically.
 * The whole tensor must be smaller than 2 GiB and C * sizeof(dtype) at most
 * FLASHBEV_ROW_BYTES_MAX.  Values must be finite. */
typedef struct {
    const void *data;
    int32_t dtype;                  /* flashbev_dtype */
    int32_t B, N, H, W, C;
    int32_t img_h, img_w;
} flashbev_features;

/* BEV grid in the ego/lidar frame: X cells along x starting at x_min with
 * pitch dx, Y cells along y starting at y_min with pitch dy; cell (i, j)
 * has centre (x_min + (i + 1/2) dx, y_min + (j + 1/2) dy).  A sample is
 * valid only if its depth exceeds depth_eps (use 1e-5). */
typedef struct {
    float x_min, dx;
    int32_t X;
    float y_min, dy;
    int32_t Y;
    float depth_eps;
    int32_t reduce;                 /* flashbev_reduce */
} flashbev_bev_grid_spec;

/* Height bins: a HOST array of Z heights in metres (0 <= Z <= FLASHBEV_ZMAX),
 * read during the call only. */
typedef struct {
    const float *z;
    int32_t Z;
} flashbev_z_bins;

/*
 * Fused Sampling-VT forward (Eq. 1; Sec. 3.3, Alg. 2).
 *
 *   features   feature maps and image size (see flashbev_features).
 *   lidar2img  device, [B, N, 4, 4] float32 row-major, 4-byte aligned; the
 *              paper's (B, N, 3, 4) projection matrices are rows 0..2 and
 *              row 3 is ignored.
 *   spec       BEV grid, depth threshold and reduction mode.
 *   z_bins     heights (host memory).
 *   out        device, [B, C, X, Y] float32, caller-allocated, 4-byte
 *              aligned, must not overlap features or lidar2img.  Every
 *              element is written exactly once (cells no camera sees get
 *              +0.0), so it needs no zeroing beforehand.
 *   stream     hipStream_t to launch on; NULL means the default stream.
 *
 * Returns FLASHBEV_OK once the work is enqueued (it completes
 * asynchronously), or a negative flashbev_status.  Argument errors are
 * reported before any HIP call; a failed launch returns FLASHBEV_ERR_HIP.
 * An empty output (B, C, X or Y zero) enqueues nothing and returns OK.
 */
int flashbev_sample_vt(const flashbev_features *features, const float *lidar2img,
                       const flashbev_bev_grid_spec *spec, const flashbev_z_bins *z_bins,
                       float *out, void *stream);

/*
 * Backward of the fused Sampling-VT operator: the gradient of Eq. 1 with
 * respect to the camera feature maps (the gradient the paper measures in
 * Sec. 4, Tables 2 and 4).  Eq. 1 is linear in the features, so the
 * gradient is the transpose of the forward's map: each valid sample
 * (b, i, j, z, n) adds w_t / max(1, den_z) * grad_out[b, c, i, j] to channel
 * c of each of its in-range bilinear taps t (divisor 1 in sum mode).  The
 * projection, mask, den_z, feature coordinates and weights are the
 * forward's, computed the same way.  The projection matrices get no
 * gradient.
 *
 *   features       shapes only: B, N, H, W, C, img_h, img_w and a valid
 *                  dtype are read; `data` is not used and may be NULL.
 *   lidar2img      device, [B, N, 4, 4] float32, as in flashbev_sample_vt.
 *   spec, z_bins   as in flashbev_sample_vt.
 *   grad_out       device, [B, C, X, Y] float32, 4-byte aligned: the
 *                  gradient of the loss with respect to `out`.
 *   grad_features  device, [B, N, H, W, C] float32 (whatever the feature
 *                  dtype), caller-allocated, 4-byte aligned, must not
 *                  overlap grad_out or lidar2img.  Fully overwritten (a
 *                  fill kernel zeroes it first, on the same stream).
 *   stream         hipStream_t; NULL means the default stream.
 *
 * The sum over samples uses float32 atomic adds, so its rounding order (not
 * its terms) varies from run to run.  Limits: those of flashbev_sample_vt,
 * plus B N H W C < 2^31.  Returns FLASHBEV_OK once enqueued or a negative
 * flashbev_status; argument errors are reported before any HIP call.
 * Nothing is enqueued when B, N, H, W or C is zero; only the fill runs
 * when X, Y or Z is zero.
 */
int flashbev_sample_vt_backward(const flashbev_features *features, const float *lidar2img,
                                const flashbev_bev_grid_spec *spec,
                                const flashbev_z_bins *z_bins, const float *grad_out,
                                float *grad_features, void *stream);

/*
 * The same gradient as flashbev_sample_vt_backward, in gather form: every
 * element of grad_features is written exactly once, with no atomics, and
 * the result is bitwise identical from run to run.  Two kernels run on
 * `stream`:
 *   1. the output gradient is transposed to cell-major rows
 *      Gt[b, i Y + j, c] = grad_out[b, c, i, j] and den_z of every
 *      (b, i, j, z) (the number of cameras whose mask M_n holds, Eq. 1) is
 *      tabulated, both in `workspace`;
 *   2. each wavefront takes a few consecutive pixels of one feature-map row
 *      of camera n (of two rows where the rows are wide: at most two pixels
 *      per row), finds the (cell, height) samples whose bilinear taps
 *      reach them (a conservative float64 region per height, then the
 *      forward's exact float32 projection, mask and floor for each
 *      candidate), and sums w_t / max(1, den_z) times their Gt rows in a
 *      fixed order.
 *
 *   features, lidar2img, spec, z_bins, grad_out, grad_features, stream
 *                  as in flashbev_sample_vt_backward.
 *   workspace      device memory of at least workspace_bytes bytes, 256-byte
 *                  aligned, owned by the caller; it must not overlap
 *                  grad_out, lidar2img or grad_features, and must not be
 *                  used by other work until the call's kernels have run.
 *                  Its contents on entry do not matter.  Layout: Gt
 *                  (float32, B X Y C), then at the next 256-byte boundary
 *                  den_z (uint8, B X Y Z).
 *   workspace_bytes  its size; flashbev_backward_workspace_size gives the
 *                  minimum.
 *
 * Errors (before any HIP call): those of flashbev_sample_vt_backward;
 * FLASHBEV_ERR_NULLPTR if workspace is NULL, FLASHBEV_ERR_ALIGN if it is not
 * 256-byte aligned, FLASHBEV_ERR_VALUE if workspace_bytes is too small,
 * FLASHBEV_ERR_ALIAS if it overlaps another buffer, and
 * FLASHBEV_ERR_UNSUPPORTED when B X Y C * 4 or B X Y Z reaches 2^31 or
 * C * 4 exceeds FLASHBEV_ROW_BYTES_MAX (flashbev_sample_vt_backward serves
 * those shapes).  Nothing is enqueued when B, N, H, W or C is zero.
 */
int flashbev_sample_vt_backward_ws(const flashbev_features *features, const float *lidar2img,
                                   const flashbev_bev_grid_spec *spec,
                                   const flashbev_z_bins *z_bins, const float *grad_out,
                                   float *grad_features, void *workspace,
                                   uint64_t workspace_bytes, void *stream);

/*
 * flashbev_sample_vt_backward_ws without a caller workspace and without any
 * allocation, for callers that cannot call hipMalloc: work captured into a
 * HIP graph, tight serving loops, harnesses that forbid allocation.  The
 * workspace is a static device array of FLASHBEV_SCRATCH_BYTES (64 MiB) that
 * the library holds on each GPU it runs on until the process ends; its
 * address on the current device is looked up once, on the first call on
 * that device.  The call makes no hipMalloc, hipFree or other allocating
 * call.
 *
 * Arguments, results and errors are those of flashbev_sample_vt_backward_ws
 * without `workspace` and `workspace_bytes`; in addition it returns
 * FLASHBEV_ERR_SCRATCH, before any HIP call, when the workspace the call
 * needs (flashbev_backward_workspace_size) exceeds FLASHBEV_SCRATCH_BYTES.
 * Every call on a GPU uses that GPU's one scratch array: calls that can
 * overlap on one GPU (on different streams, or from several threads) race
 * and must be ordered by the caller.  Nothing in the scratch needs to be
 * zero on entry; a call overwrites what it reads.
 */
int flashbev_sample_vt_backward_noalloc(const flashbev_features *features,
                                        const float *lidar2img,
                                        const flashbev_bev_grid_spec *spec,
                                        const flashbev_z_bins *z_bins, const float *grad_out,
                                        float *grad_features, void *stream);

/*
 * Workspace bytes flashbev_sample_vt_backward_ws needs for these arguments
 * (written to *bytes; a multiple of 256).  Same shape checks, no device
 * pointer needed, no HIP call; FLASHBEV_ERR_UNSUPPORTED for the shapes the
 * gather form does not serve.
 */
int flashbev_backward_workspace_size(const flashbev_features *features,
                                     const flashbev_bev_grid_spec *spec,
                                     const flashbev_z_bins *z_bins, uint64_t *bytes);

/*
 * Launch geometry of flashbev_sample_vt_backward for these arguments: the
 * scatter kernel's workgroup count (0 when only the fill runs), threads per
 * workgroup, dynamic LDS bytes per workgroup, the LDS rows (distinct feature
 * pixels) a tile can accumulate (0 when the kernel adds every term with a
 * global atomic) and the lanes per BEV cell.  Same shape checks as the
 * backward; no device pointer is needed and no HIP call is made.
 */
int flashbev_backward_launch_info(const flashbev_features *features,
                                  const flashbev_bev_grid_spec *spec,
                                  const flashbev_z_bins *z_bins, int64_t *workgroups,
                                  int32_t *threads_per_workgroup, int32_t *lds_bytes,
                                  int32_t *rows_per_tile, int32_t *lanes_per_cell);

/* Static, human-readable text for a status code (never NULL). */
const char *flashbev_status_string(int status);

/* FLASHBEV_ABI_VERSION of the built library. */
int flashbev_abi_version(void);

/*
 * Launch geometry the library would use for these arguments, for tools that
 * report per-launch figures.  On success writes the workgroup count, the
 * threads per workgroup, the dynamic LDS bytes per workgroup, the BEV cells
 * per wavefront and the lanes per cell.  Performs the same argument checks
 * as flashbev_sample_vt (pointers to device data are not dereferenced and
 * may be NULL here) and makes no HIP call.
 */
int flashbev_launch_info(const flashbev_features *features, const flashbev_bev_grid_spec *spec,
                         const flashbev_z_bins *z_bins, int64_t *workgroups,
                         int32_t *threads_per_workgroup, int32_t *lds_bytes,
                         int32_t *cells_per_wave, int32_t *lanes_per_cell);

#ifdef __cplusplus
}
#endif

#endif /* FLASHBEV_H */
