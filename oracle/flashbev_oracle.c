/*
 * CPU oracle for the fused Sampling-VT operator (FlashBEV forward).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plainly written reference
 * that the GPU library is checked against.  It shares no code, header, table
 * or helper with the GPU library, and the product path never links it: only
 * the tests, the smoke check and the bench's CPU-baseline leg load it.
 *
 * What it computes (FlashBEV paper, Sec. 3.1, Eq. 1):
 *
 *   out[b,c,x,y] = sum_z  ( sum_n M_n(x,y,z) f_n(x,y,z,c) ) / max(1, sum_n M_n(x,y,z))
 *
 * with M_n the validity mask (the projected voxel centre lies inside camera
 * n's image and has positive depth) and f_n the bilinear sample of camera n's
 * feature map at the projected pixel (Sec. 3.1, text after Eq. 1).  The loop
 * order is the one Sec. 3.3.1 describes for one output element: heights
 * outer, cameras inner, per-height numerator and denominator, then the
 * per-height valid mean added to the running sum.  Here one call handles all
 * channels of a BEV cell at once, which changes nothing in the arithmetic.
 *
 * It also computes the backward of Eq. 1 with respect to the feature maps
 * (the gradient the paper measures in Sec. 4, Tables 2 and 4): the transpose
 * of the forward's linear map, written as a scatter of each valid sample's
 * weighted output gradient onto its bilinear taps.
 *
 * Readings where the paper is silent:
 *   - coordinates follow one fixed float32 recipe: every product and sum is
 *     rounded on its own (no fused multiply-add), left to right, and the
 *     perspective divide is an IEEE float32 division.  Mask and floor
 *     decisions are integer outcomes decided by floating point, so the GPU
 *     library takes them in the same precision (the paper's FP32);
 *   - voxel centres are cell centres: x = x_min + (i + 1/2) dx;
 *   - "positive depth" is d > depth_eps, checked before the divide;
 *   - "inside the image" is the half-open box 0 <= u < img_w, 0 <= v < img_h;
 *   - pixel -> feature coordinates use the align_corners=False convention,
 *     x_f = u * (W / img_w) - 1/2 (and likewise for y);
 *   - bilinear taps outside the feature map contribute zero (zero padding),
 *     but the sample still counts in the denominator;
 *   - accumulation is float64.  The oracle also returns, per output element,
 *     the magnitude scale S = sum_z sum_n sum_taps w |F| / max(1, den), which
 *     bounds the size of any rounding error of a float32 implementation.
 *
 * Parity pins (tests/): brute-force tensorized evaluation (Alg. 1) on tiny
 * inputs, torch grid_sample for one camera and one height, constant and
 * planar feature maps, hand-placed points with known projections, and the
 * invariants of Eq. 1 (camera permutation, linearity, height additivity).
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t B, N, H, W, C;   /* features: NHWC [B, N, H, W, C]             */
    int32_t img_h, img_w;    /* image size lidar2img projects into         */
    int32_t X, Y, Z;         /* BEV grid and number of height bins         */
    float x_min, dx;         /* cell i has centre x_min + (i + 1/2) dx     */
    float y_min, dy;
    float depth_eps;         /* valid iff depth > depth_eps                */
    int32_t reduce;          /* 0: valid mean per height (Eq. 1), 1: sum   */
} oracle_problem;

typedef struct {
    int64_t valid_samples;   /* samples with M = 1                         */
    int64_t taps;            /* in-range bilinear taps over valid samples  */
} oracle_counters;

int oracle_abi_version(void) { return 1; }

/* Voxel centre of cell (i, j); Sec. 3.1 ("voxel center"), Alg. 1 step 1. */
static void voxel_centre(const oracle_problem *p, int i, int j, float *x, float *y)
{
    float fi = (float)i + 0.5f;
    float fj = (float)j + 0.5f;
    float tx = fi * p->dx;
    float ty = fj * p->dy;
    *x = p->x_min + tx;
    *y = p->y_min + ty;
}

/*
 * Project point (x, y, z) through camera matrix m (rows 0..2 of a row-major
 * 4x4 lidar2img; Alg. 1 step 2) and apply the validity mask M_n (Sec. 3.1).
 * Returns 1 when valid, with the feature-map coordinates in *xf, *yf.
 */
static int project(const oracle_problem *p, const float *m, float x, float y, float z,
                   float *xf, float *yf)
{
    float a, b, c;
    a = m[0] * x; b = m[1] * y; c = m[2] * z;
    float up = ((a + b) + c) + m[3];
    a = m[4] * x; b = m[5] * y; c = m[6] * z;
    float vp = ((a + b) + c) + m[7];
    a = m[8] * x; b = m[9] * y; c = m[10] * z;
    float d = ((a + b) + c) + m[11];
    if (!(d > p->depth_eps))          /* positive depth (also rejects NaN) */
        return 0;
    float u = up / d;
    float v = vp / d;
    if (!(u >= 0.0f && u < (float)p->img_w && v >= 0.0f && v < (float)p->img_h))
        return 0;                     /* outside the camera image */
    float sx = (float)p->W / (float)p->img_w;
    float sy = (float)p->H / (float)p->img_h;
    float tx = u * sx;
    float ty = v * sy;
    *xf = tx - 0.5f;
    *yf = ty - 0.5f;
    return 1;
}

/*
 * Bilinear taps of a sample at feature coordinates (xf, yf) (Sec. 3.1, text
 * after Eq. 1): the in-range pixels among the four neighbours and their
 * weights.  Taps outside the map are left out (zero padding).  Returns the
 * number of taps written to xt[], yt[], w[].
 */
static int bilinear_taps(const oracle_problem *p, float xf, float yf, int *xs, int *ys, double *ws)
{
    float x0f = floorf(xf), y0f = floorf(yf);
    float ax = xf - x0f, ay = yf - y0f;
    int x0 = (int)x0f, y0 = (int)y0f;
    int n = 0;
    for (int ty = 0; ty < 2; ++ty) {
        for (int tx = 0; tx < 2; ++tx) {
            int xt = x0 + tx, yt = y0 + ty;
            if (xt < 0 || xt >= p->W || yt < 0 || yt >= p->H)
                continue;
            double wx = tx ? (double)ax : 1.0 - (double)ax;
            double wy = ty ? (double)ay : 1.0 - (double)ay;
            xs[n] = xt;
            ys[n] = yt;
            ws[n] = wx * wy;
            ++n;
        }
    }
    return n;
}

/*
 * All C channels of one BEV cell (b, i, j): Eq. 1 evaluated with heights
 * outer and cameras inner.  acc and scale receive C values each; num and mag
 * are C-sized scratch arrays.
 */
static void one_cell(const oracle_problem *p, const float *feat, const float *l2i,
                     const float *zs, int b, int i, int j, double *acc, double *scale,
                     double *num, double *mag, oracle_counters *cnt)
{
    const int C = p->C;
    float x, y;
    voxel_centre(p, i, j, &x, &y);
    for (int c = 0; c < C; ++c) { acc[c] = 0.0; scale[c] = 0.0; }
    for (int k = 0; k < p->Z; ++k) {
        const float z = zs[k];
        int den = 0;
        for (int c = 0; c < C; ++c) { num[c] = 0.0; mag[c] = 0.0; }
        for (int n = 0; n < p->N; ++n) {
            const float *m = l2i + ((size_t)b * p->N + n) * 16;
            float xf, yf;
            if (!project(p, m, x, y, z, &xf, &yf))
                continue;
            /* bilinear sample f_n (Sec. 3.1), zero padding outside the map */
            int txs[4], tys[4];
            double tws[4];
            const int nt = bilinear_taps(p, xf, yf, txs, tys, tws);
            for (int t = 0; t < nt; ++t) {
                const int xt = txs[t], yt = tys[t];
                const double w = tws[t];
                const float *f = feat + ((((size_t)b * p->N + n) * p->H + yt) * p->W + xt) * C;
                for (int c = 0; c < C; ++c) {
                    num[c] += w * (double)f[c];
                    mag[c] += w * fabs((double)f[c]);
                }
                if (cnt) cnt->taps += 1;
            }
            den += 1;                 /* num_z += M f ; den_z += M */
            if (cnt) cnt->valid_samples += 1;
        }
        /* per-height valid mean (Eq. 1), or the plain sum when reduce == 1 */
        double dd = (p->reduce == 0 && den > 1) ? (double)den : 1.0;
        for (int c = 0; c < C; ++c) {
            acc[c] += num[c] / dd;
            scale[c] += mag[c] / dd;
        }
    }
}

static int check(const oracle_problem *p)
{
    if (!p) return -1;
    if (p->B < 0 || p->N < 0 || p->H < 1 || p->W < 1 || p->C < 1 || p->img_h < 1 ||
        p->img_w < 1 || p->X < 0 || p->Y < 0 || p->Z < 0)
        return -2;
    return 0;
}

/*
 * Full operator: out and scale are [B, C, X, Y] float64 (scale may be NULL).
 * feat is NHWC [B, N, H, W, C] float32 (16-bit inputs arrive as their exact
 * float32 values), lidar2img is [B, N, 4, 4] float32 row-major, zs is [Z].
 * nthreads <= 0 uses the OpenMP default.
 */
int oracle_sample_vt(const oracle_problem *p, const float *feat, const float *l2i,
                     const float *zs, double *out, double *scale, oracle_counters *counters,
                     int nthreads)
{
    int rc = check(p);
    if (rc) return rc;
    const int C = p->C;
    const int64_t rows = (int64_t)p->B * p->X;
    int64_t V = 0, T = 0;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
#pragma omp parallel reduction(+ : V, T)
    {
        double *buf = (double *)malloc(sizeof(double) * 4 * (size_t)C);
        oracle_counters cnt = {0, 0};
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < rows; ++r) {
            int b = (int)(r / p->X), i = (int)(r % p->X);
            for (int j = 0; j < p->Y; ++j) {
                one_cell(p, feat, l2i, zs, b, i, j, buf, buf + C, buf + 2 * C, buf + 3 * C, &cnt);
                for (int c = 0; c < C; ++c) {
                    size_t o = (((size_t)b * C + c) * p->X + i) * p->Y + j;
                    out[o] = buf[c];
                    if (scale) scale[o] = buf[C + c];
                }
            }
        }
        V += cnt.valid_samples;
        T += cnt.taps;
        free(buf);
    }
    if (counters) { counters->valid_samples = V; counters->taps = T; }
    return 0;
}

/*
 * Selected cells only: cells is [ncells, 3] int32 (b, i, j); out and scale
 * are [ncells, C] float64 (scale may be NULL).  Used for sampled checks of
 * workloads too large to evaluate in full.
 */
int oracle_sample_cells(const oracle_problem *p, const float *feat, const float *l2i,
                        const float *zs, const int32_t *cells, int64_t ncells, double *out,
                        double *scale, int nthreads)
{
    int rc = check(p);
    if (rc) return rc;
    const int C = p->C;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    for (int64_t q = 0; q < ncells; ++q) {
        const int32_t *cl = cells + 3 * q;
        if (cl[0] < 0 || cl[0] >= p->B || cl[1] < 0 || cl[1] >= p->X || cl[2] < 0 || cl[2] >= p->Y)
            return -3;
    }
#pragma omp parallel
    {
        double *buf = (double *)malloc(sizeof(double) * 4 * (size_t)C);
#pragma omp for schedule(dynamic, 16)
        for (int64_t q = 0; q < ncells; ++q) {
            const int32_t *cl = cells + 3 * q;
            one_cell(p, feat, l2i, zs, cl[0], cl[1], cl[2], buf, buf + C, buf + 2 * C,
                     buf + 3 * C, NULL);
            memcpy(out + q * C, buf, sizeof(double) * C);
            if (scale) memcpy(scale + q * C, buf + C, sizeof(double) * C);
        }
        free(buf);
    }
    return 0;
}

/*
 * Projection-only pass: for every (b, i, j, k, n) writes the mask M_n
 * (uint8) and, where valid, the feature-map coordinates (x_f, y_f) (NaN
 * where invalid).  Arrays are [B, X, Y, Z, N].
 */
int oracle_project(const oracle_problem *p, const float *l2i, const float *zs,
                   uint8_t *mask, float *xf, float *yf)
{
    int rc = check(p);
    if (rc) return rc;
    for (int b = 0; b < p->B; ++b)
        for (int i = 0; i < p->X; ++i)
            for (int j = 0; j < p->Y; ++j) {
                float x, y;
                voxel_centre(p, i, j, &x, &y);
                for (int k = 0; k < p->Z; ++k)
                    for (int n = 0; n < p->N; ++n) {
                        size_t o = ((((size_t)b * p->X + i) * p->Y + j) * p->Z + k) * p->N + n;
                        const float *m = l2i + ((size_t)b * p->N + n) * 16;
                        float a = NAN, c = NAN;
                        int ok = project(p, m, x, y, zs[k], &a, &c);
                        mask[o] = (uint8_t)ok;
                        xf[o] = ok ? a : NAN;
                        yf[o] = ok ? c : NAN;
                    }
            }
    return 0;
}

/*
 * Backward of Eq. 1 with respect to the camera feature maps F_n.
 *
 * Eq. 1 is linear in F: every valid sample (b, i, j, k, n) adds, for each
 * in-range bilinear tap (xt, yt) with weight w, the term
 * w / max(1, den_k) * F[b, n, yt, xt, c] to out[b, c, i, j] (den_k = number
 * of cameras valid at height k; the divisor is 1 in sum mode).  The gradient
 * of a loss with output gradient G = dL/d out is therefore the transpose of
 * that map:
 *
 *   grad_feat[b, n, yt, xt, c] = sum over those (i, j, k, tap) of
 *                                w / max(1, den_k) * G[b, c, i, j].
 *
 * It is computed as a scatter in two passes: first den_k for every
 * (b, i, j, k), then, one camera (b, n) per task, the samples of that camera
 * in the forward's order; a task writes only its own camera's slice, so the
 * tasks never write the same element.  Accumulation is float64.
 *
 *   grad_out   [B, C, X, Y] float32
 *   grad_feat  [B, N, H, W, C] float64 (fully written)
 *   scale      [B, N, H, W, C] float64, sum of |terms| (may be NULL)
 *   terms      [B, N, H, W] int32, number of (sample, tap) terms per pixel
 *              (may be NULL)
 */
int oracle_sample_vt_backward(const oracle_problem *p, const float *l2i, const float *zs,
                              const float *grad_out, double *grad_feat, double *scale,
                              int32_t *terms, int nthreads)
{
    int rc = check(p);
    if (rc) return rc;
    const int C = p->C;
    const size_t cells = (size_t)p->B * p->X * p->Y;
    const size_t pix = (size_t)p->H * p->W;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    /* pass 1: number of valid cameras per (b, i, j, k) */
    uint8_t *valid_count = (uint8_t *)malloc(cells * (size_t)(p->Z > 0 ? p->Z : 1));
    if (!valid_count) return -4;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < (int64_t)p->B * p->X; ++r) {
        const int b = (int)(r / p->X), i = (int)(r % p->X);
        for (int j = 0; j < p->Y; ++j) {
            float x, y;
            voxel_centre(p, i, j, &x, &y);
            for (int k = 0; k < p->Z; ++k) {
                int seen = 0;
                for (int n = 0; n < p->N; ++n) {
                    float xf, yf;
                    seen += project(p, l2i + ((size_t)b * p->N + n) * 16, x, y, zs[k], &xf, &yf);
                }
                valid_count[(((size_t)b * p->X + i) * p->Y + j) * p->Z + k] = (uint8_t)seen;
            }
        }
    }
    /* pass 2: scatter, one camera per task */
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t bn = 0; bn < (int64_t)p->B * p->N; ++bn) {
        const int b = (int)(bn / p->N);
        const float *m = l2i + (size_t)bn * 16;
        double *gf = grad_feat + (size_t)bn * pix * C;
        double *sf = scale ? scale + (size_t)bn * pix * C : NULL;
        int32_t *tf = terms ? terms + (size_t)bn * pix : NULL;
        memset(gf, 0, sizeof(double) * pix * C);
        if (sf) memset(sf, 0, sizeof(double) * pix * C);
        if (tf) memset(tf, 0, sizeof(int32_t) * pix);
        for (int i = 0; i < p->X; ++i)
            for (int j = 0; j < p->Y; ++j) {
                float x, y;
                voxel_centre(p, i, j, &x, &y);
                for (int k = 0; k < p->Z; ++k) {
                    float xf, yf;
                    if (!project(p, m, x, y, zs[k], &xf, &yf))
                        continue;
                    const int seen = valid_count[(((size_t)b * p->X + i) * p->Y + j) * p->Z + k];
                    const double norm = (p->reduce == 0 && seen > 1) ? 1.0 / (double)seen : 1.0;
                    int txs[4], tys[4];
                    double tws[4];
                    const int nt = bilinear_taps(p, xf, yf, txs, tys, tws);
                    for (int t = 0; t < nt; ++t) {
                        const size_t q = (size_t)tys[t] * p->W + txs[t];
                        for (int c = 0; c < C; ++c) {
                            const double g = (double)grad_out[(((size_t)b * C + c) * p->X + i) * p->Y + j];
                            const double term = tws[t] * norm * g;
                            gf[q * C + c] += term;
                            if (sf) sf[q * C + c] += fabs(term);
                        }
                        if (tf) tf[q] += 1;
                    }
                }
            }
    }
    free(valid_count);
    return 0;
}
