/*
 * CPU oracle for FlashSCA: BEVFormer's spatial cross-attention (SCA) with the
 * per-camera sampling points formed on the fly (FlashBEV paper, Sec. 4.5,
 * "Cross-framework applicability", Table 7).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plainly written reference
 * that the GPU library is checked against.  It shares no code, header, table
 * or helper with the GPU library, and the product path never links it: only
 * the tests, the smoke check and the bench's CPU-baseline leg load it.
 *
 * What it computes.  The paper applies its execution idea to the SCA of
 * BEVFormer (Li et al., ECCV 2022, Sec. 3.4): each BEV query q owns a pillar
 * of Z anchor heights above its cell; the anchors are projected into every
 * camera; a camera is "hit" when at least one anchor lands in its image; in
 * every hit camera, deformable attention samples each head's L levels at P
 * points around the anchors' reference points, weighted by a softmax over
 * the L*P (level, point) logits of that head; the result is summed over the
 * hit cameras and divided by their number.  With value V (per camera and
 * level, channels split into heads of D = C / heads), offsets dp and logits
 * s, for channel c = m D + e of head m:
 *
 *   out[b,q,c] = 1/max(1, |hit(q)|) * sum_{n in hit(q)} sum_{l,k}
 *                softmax_{l,k}(s[b,q,m,:,:])[l,k] *
 *                bilinear(V[b,n,l][:, :, c], ref_n(anchor(k)) * (W_l, H_l) + dp[b,q,m,l,k] - 1/2)
 *
 * Readings (the paper gives the idea; the semantics are BEVFormer's published SCA):
 *   - queries are the BEV cells of the Eq. 1 grid, q = i Y + j, with cell
 *     centre (x_min + (i + 1/2) dx, y_min + (j + 1/2) dy);
 *   - point k of a (head, level) belongs to anchor k mod Z (BEVFormer splits
 *     the P points of a level into P / Z groups of Z, one point per anchor);
 *   - an anchor is valid in camera n when its depth exceeds depth_eps and its
 *     normalized image coordinates (u / img_w, v / img_h) lie strictly
 *     inside (0, 1); the pixel divides by the depth clamped from below at
 *     depth_eps, so anchors behind a camera still get (far away) reference
 *     points;
 *   - a hit camera samples the points of all its anchors, valid or not;
 *   - the projection follows the float32 recipe of Eq. 1's oracle (every
 *     product and sum rounded on its own, IEEE division); the normalized
 *     coordinates are two further float32 divisions;
 *   - the sampling location in level-l pixels is x = (u_n W_l + dp_x) - 1/2,
 *     each step rounded to float32 (algebraically BEVFormer's
 *     (u_n + dp_x / W_l) W_l - 1/2 of grid_sample with align_corners=False);
 *     these float32 values decide the taps, so the GPU library takes them in
 *     the same precision;
 *   - bilinear taps outside the level's map contribute zero (zero padding);
 *   - softmax and all sums are float64.  Per output element the oracle also
 *     returns the magnitude scale S (the same sum over |terms|), and per
 *     (query, head) the number of in-range taps K, which bound the rounding
 *     error of a float32 implementation.
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

#define SCA_LMAX 8

typedef struct {
    int32_t B, N, C, heads, L, P, Z;
    int32_t level_h[SCA_LMAX], level_w[SCA_LMAX];
    int32_t img_h, img_w;
    int32_t X, Y;
    float x_min, dx, y_min, dy;
    float depth_eps;
    int32_t reduce;          /* 0: mean over hit cameras, 1: plain sum      */
} sca_problem;

typedef struct {
    int64_t hits;            /* (query, camera) pairs with a hit            */
    int64_t taps;            /* in-range bilinear taps, all heads           */
} sca_counters;

int sca_oracle_abi_version(void) { return 1; }

static int64_t sca_pixels(const sca_problem *p)
{
    int64_t s = 0;
    for (int l = 0; l < p->L; ++l) s += (int64_t)p->level_h[l] * p->level_w[l];
    return s;
}

/* BEV cell centre of query (i, j). */
static void cell_centre(const sca_problem *p, int i, int j, float *x, float *y)
{
    float fi = (float)i + 0.5f;
    float fj = (float)j + 0.5f;
    float tx = fi * p->dx;
    float ty = fj * p->dy;
    *x = p->x_min + tx;
    *y = p->y_min + ty;
}

/*
 * Reference point of anchor (x, y, z) in the camera with matrix m (rows 0..2
 * of a row-major 4x4 lidar2img): normalized image coordinates (un, vn).
 * Returns 1 when the anchor is valid (positive depth, strictly inside the
 * image), 0 otherwise; the coordinates are written either way.
 */
static int reference_point(const sca_problem *p, const float *m, float x, float y, float z,
                           float *un, float *vn)
{
    float a, b, c;
    a = m[0] * x; b = m[1] * y; c = m[2] * z;
    float up = ((a + b) + c) + m[3];
    a = m[4] * x; b = m[5] * y; c = m[6] * z;
    float vp = ((a + b) + c) + m[7];
    a = m[8] * x; b = m[9] * y; c = m[10] * z;
    float d = ((a + b) + c) + m[11];
    int in_front = d > p->depth_eps;
    float dd = in_front ? d : p->depth_eps;     /* depth clamped at depth_eps */
    float u = up / dd;
    float v = vp / dd;
    *un = u / (float)p->img_w;
    *vn = v / (float)p->img_h;
    return in_front && *un > 0.0f && *un < 1.0f && *vn > 0.0f && *vn < 1.0f;
}

/*
 * Steps 1 and 2 for query (b, i, j): reference points of every anchor in
 * every camera (un, vn [N*Z]), hit cameras (hit [N]) and the attention
 * weights, a softmax over the L*P logits of each head (attn [heads*L*P]).
 * Returns the number of hit cameras.
 */
static int prepare_query(const sca_problem *p, const float *l2i, const float *zs,
                         const float *logits, int b, int i, int j, float *un, float *vn,
                         int *hit, double *attn)
{
    const int N = p->N, Z = p->Z, H = p->heads, L = p->L, P = p->P;
    const int64_t Q = (int64_t)p->X * p->Y;
    const int64_t q = (int64_t)i * p->Y + j;
    float x, y;
    cell_centre(p, i, j, &x, &y);

    /* 1. reference points of every anchor in every camera; hit cameras */
    int count = 0;
    for (int n = 0; n < N; ++n) {
        const float *m = l2i + ((size_t)b * N + n) * 16;
        hit[n] = 0;
        for (int k = 0; k < Z; ++k)
            hit[n] |= reference_point(p, m, x, y, zs[k], &un[n * Z + k], &vn[n * Z + k]);
        count += hit[n];
    }

    /* 2. attention weights: softmax over the L*P logits of each head */
    const float *lg = logits + ((size_t)b * Q + q) * H * L * P;
    for (int h = 0; h < H; ++h) {
        const float *s = lg + (size_t)h * L * P;
        double mx = -INFINITY;
        for (int t = 0; t < L * P; ++t) mx = fmax(mx, (double)s[t]);
        double sum = 0.0;
        for (int t = 0; t < L * P; ++t) {
            attn[h * L * P + t] = exp((double)s[t] - mx);
            sum += attn[h * L * P + t];
        }
        for (int t = 0; t < L * P; ++t) attn[h * L * P + t] /= sum;
    }
    return count;
}

/* The anchor of point k: BEVFormer splits a level's P points into P / Z
 * groups of Z consecutive points, one per anchor. */
static int anchor_of_point(int k, int P, int Z)
{
    (void)P;
    return k % Z;
}

/*
 * Bilinear corners of point (h, l, k) of a query in one camera: the sampling
 * location (x, y) in level-l pixels from the anchor's reference point
 * (un, vn) and the offset o, then the four corners (x0 + tx, y0 + ty),
 * tx, ty in {0, 1}, in the order 00, 01 (right), 10 (below), 11, with their
 * weights and whether each lies inside the map (zero padding otherwise).
 * Returns 0 when no corner lies inside the map (also for a location that is
 * not finite); the fractions are written to *fx, *fy.
 */
typedef struct {
    int64_t pix[4];          /* pixel index within the camera's value, all levels */
    int in[4];               /* corner inside the level's map */
    double w[4];             /* bilinear weight */
} corners;

static int point_corners(const sca_problem *p, int l, int64_t start, float un, float vn,
                         const float *o, corners *cr, double *fx, double *fy)
{
    const int Hl = p->level_h[l], Wl = p->level_w[l];
    float sx = un * (float)Wl;
    float sy = vn * (float)Hl;
    sx = sx + o[0];
    sy = sy + o[1];
    const float xim = sx - 0.5f;
    const float yim = sy - 0.5f;
    /* no corner inside the map (also non-finite locations) */
    if (!(xim > -1.0f && xim < (float)Wl && yim > -1.0f && yim < (float)Hl))
        return 0;
    const float x0f = floorf(xim), y0f = floorf(yim);
    const double ax = (double)(xim - x0f), ay = (double)(yim - y0f);
    const int x0 = (int)x0f, y0 = (int)y0f;
    for (int ty = 0; ty < 2; ++ty)
        for (int tx = 0; tx < 2; ++tx) {
            const int c = ty * 2 + tx;
            const int xt = x0 + tx, yt = y0 + ty;
            cr->in[c] = !(xt < 0 || xt >= Wl || yt < 0 || yt >= Hl);
            cr->w[c] = (tx ? ax : 1.0 - ax) * (ty ? ay : 1.0 - ay);
            cr->pix[c] = cr->in[c] ? start + (int64_t)yt * Wl + xt : 0;
        }
    *fx = ax;
    *fy = ay;
    return 1;
}

/*
 * One query: all C channels of out[b, q, :], their scales, and the tap count
 * per head.  acc and scale hold C values; terms holds `heads` values.
 * Scratch: un, vn [N*Z] floats, hit [N] ints, attn [heads*L*P] doubles.
 */
static void one_query(const sca_problem *p, const float *value, const float *l2i,
                      const float *zs, const float *offsets, const float *logits, int b, int i,
                      int j, double *acc, double *scale, int32_t *terms, float *un, float *vn,
                      int *hit, double *attn, sca_counters *cnt)
{
    const int N = p->N, Z = p->Z, C = p->C, H = p->heads, L = p->L, P = p->P;
    const int D = C / H;
    const int64_t Q = (int64_t)p->X * p->Y;
    const int64_t q = (int64_t)i * p->Y + j;
    const int64_t S = sca_pixels(p);
    const int count = prepare_query(p, l2i, zs, logits, b, i, j, un, vn, hit, attn);

    /* 3. deformable sampling in every hit camera, summed over cameras */
    for (int c = 0; c < C; ++c) { acc[c] = 0.0; scale[c] = 0.0; }
    for (int h = 0; h < H; ++h) terms[h] = 0;
    const float *off = offsets + ((size_t)b * Q + q) * H * L * P * 2;
    for (int n = 0; n < N; ++n) {
        if (!hit[n]) continue;
        if (cnt) cnt->hits += 1;
        const float *vcam = value + ((size_t)b * N + n) * (size_t)S * C;
        for (int h = 0; h < H; ++h) {
            int64_t start = 0;
            for (int l = 0; l < L; ++l) {
                for (int k = 0; k < P; ++k) {
                    const int z = anchor_of_point(k, P, Z);
                    const float *o = off + (((size_t)h * L + l) * P + k) * 2;
                    corners cr;
                    double fx, fy;
                    if (!point_corners(p, l, start, un[n * Z + z], vn[n * Z + z], o, &cr, &fx,
                                       &fy))
                        continue;
                    const double a = attn[(h * L + l) * P + k];
                    for (int t = 0; t < 4; ++t) {
                        if (!cr.in[t]) continue;
                        const float *row = vcam + (size_t)cr.pix[t] * C + (size_t)h * D;
                        for (int e = 0; e < D; ++e) {
                            const double v = a * cr.w[t] * (double)row[e];
                            acc[h * D + e] += v;
                            scale[h * D + e] += fabs(v);
                        }
                        terms[h] += 1;
                        if (cnt) cnt->taps += 1;
                    }
                }
                start += (int64_t)p->level_h[l] * p->level_w[l];
            }
        }
    }
    /* 4. mean over the hit cameras */
    const double den = (p->reduce == 0 && count > 1) ? (double)count : 1.0;
    for (int c = 0; c < C; ++c) { acc[c] /= den; scale[c] /= den; }
}

static int check(const sca_problem *p)
{
    if (!p) return -1;
    if (p->B < 0 || p->N < 0 || p->C < 1 || p->heads < 1 || p->C % p->heads != 0 ||
        p->L < 1 || p->L > SCA_LMAX || p->P < 1 || p->Z < 1 || p->P % p->Z != 0 ||
        p->img_h < 1 || p->img_w < 1 || p->X < 0 || p->Y < 0)
        return -2;
    for (int l = 0; l < p->L; ++l)
        if (p->level_h[l] < 1 || p->level_w[l] < 1) return -2;
    return 0;
}

/*
 * Full operator.
 *   value    [B, N, S, C] float32, S = sum_l H_l W_l (levels concatenated,
 *            each row-major); 16-bit inputs arrive as their float32 values
 *   l2i      [B, N, 4, 4] float32 row-major
 *   zs       [Z] anchor heights
 *   offsets  [B, Q, heads, L, P, 2] float32 (x, y), level-pixel units
 *   logits   [B, Q, heads, L, P] float32
 *   out, scale [B, Q, C] float64 (scale may be NULL)
 *   terms    [B, Q, heads] int32 (may be NULL)
 */
int sca_oracle_forward(const sca_problem *p, const float *value, const float *l2i,
                       const float *zs, const float *offsets, const float *logits, double *out,
                       double *scale, int32_t *terms, sca_counters *counters, int nthreads)
{
    int rc = check(p);
    if (rc) return rc;
    const int C = p->C, H = p->heads;
    const int64_t Q = (int64_t)p->X * p->Y;
    const int64_t rows = (int64_t)p->B * p->X;
    int64_t hits = 0, taps = 0;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
#pragma omp parallel reduction(+ : hits, taps)
    {
        double *acc = (double *)malloc(sizeof(double) * 2 * (size_t)C);
        double *attn = (double *)malloc(sizeof(double) * (size_t)H * p->L * p->P);
        float *uv = (float *)malloc(sizeof(float) * 2 * (size_t)(p->N * p->Z + 1));
        int *hit = (int *)malloc(sizeof(int) * (size_t)(p->N + 1));
        int32_t *tm = (int32_t *)malloc(sizeof(int32_t) * (size_t)H);
        sca_counters cnt = {0, 0};
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < rows; ++r) {
            const int b = (int)(r / p->X), i = (int)(r % p->X);
            for (int j = 0; j < p->Y; ++j) {
                one_query(p, value, l2i, zs, offsets, logits, b, i, j, acc, acc + C, tm, uv,
                          uv + p->N * p->Z, hit, attn, &cnt);
                const size_t o = ((size_t)b * Q + (size_t)i * p->Y + j);
                memcpy(out + o * C, acc, sizeof(double) * C);
                if (scale) memcpy(scale + o * C, acc + C, sizeof(double) * C);
                if (terms) memcpy(terms + o * H, tm, sizeof(int32_t) * H);
            }
        }
        hits += cnt.hits;
        taps += cnt.taps;
        free(acc); free(attn); free(uv); free(hit); free(tm);
    }
    if (counters) { counters->hits = hits; counters->taps = taps; }
    return 0;
}

/*
 * Reference points and hits only: un, vn, valid are [B, Q, N, Z]; hit is
 * [B, Q, N] (uint8).  Used by the tests to select queries and to build the
 * dense comparison path.
 */
int sca_oracle_reference_points(const sca_problem *p, const float *l2i, const float *zs,
                                float *un, float *vn, uint8_t *valid, uint8_t *hit)
{
    int rc = check(p);
    if (rc) return rc;
    const int N = p->N, Z = p->Z;
    for (int b = 0; b < p->B; ++b)
        for (int i = 0; i < p->X; ++i)
            for (int j = 0; j < p->Y; ++j) {
                float x, y;
                cell_centre(p, i, j, &x, &y);
                const size_t q = ((size_t)b * p->X + i) * p->Y + j;
                for (int n = 0; n < N; ++n) {
                    int any = 0;
                    for (int k = 0; k < Z; ++k) {
                        const size_t o = (q * N + n) * Z + k;
                        int v = reference_point(p, l2i + ((size_t)b * N + n) * 16, x, y, zs[k],
                                                &un[o], &vn[o]);
                        valid[o] = (uint8_t)v;
                        any |= v;
                    }
                    hit[q * N + n] = (uint8_t)any;
                }
            }
    return 0;
}

/*
 * Backward of the FlashSCA forward with respect to its learned inputs: the
 * value maps, the sampling offsets and the attention logits (the camera
 * matrices and anchors get no gradient).  With G = dL/d out and
 * alpha = 1 / max(1, hits) (1 in sum mode), every term of the forward,
 * alpha a w V[tap, c] for a point (head h, level l, point k) in hit camera n,
 * gives:
 *
 *   d value[b, n, tap, c]  += alpha a w G[b, q, c]                  (scatter)
 *   d a                    += alpha w V[tap, c] G[b, q, c]
 *   d x                    += alpha a (dw / dx) V[tap, c] G[b, q, c]
 *
 * where x, y is the sampling location in level pixels and w the bilinear
 * weight of the tap, (1 - ax)(1 - ay), ax (1 - ay), (1 - ax) ay or ax ay with
 * (ax, ay) the location's fractional part; a location moves one pixel per
 * pixel of offset, so d offset = (d x, d y).  Taps outside the map have value
 * zero (zero padding) and points with no corner inside the map contribute
 * nothing.  The logits' gradient is the softmax backward over the head's
 * L * P pairs: d s_j = a_j (d a_j - sum_j' a_j' d a_j').
 *
 * Outputs (float64), with magnitude scales that bound a float32
 * implementation's rounding error:
 *   grad_value [B, N, S, C], scale_value (sum of |terms|), terms_value
 *     [B, N, S, heads] (terms reaching the pixel's head slice)
 *   grad_offsets [B, Q, heads, L, P, 2], scale_offsets (sum over cameras
 *     and channels of alpha a |G| ((1 - ay)(|V01| + |V00|) + ay (|V11| + |V10|))
 *     for x, and likewise for y)
 *   grad_logits [B, Q, heads, L, P], scale_logits (a_j (S_j + sum_j' a_j' S_j')
 *     with S_j the sum of |terms| of d a_j)
 *   terms_points [B, Q, heads, L, P] int32: in-range corners of the point
 *     over the hit cameras
 * Any of the scale and terms arrays may be NULL.
 *
 * Computed in two passes: per query (offsets and logits; reads only), then
 * one camera (b, n) per task for the value scatter, which writes only that
 * camera's slice.
 */
int sca_oracle_backward(const sca_problem *p, const float *value, const float *l2i,
                        const float *zs, const float *offsets, const float *logits,
                        const float *grad_out, double *grad_value, double *scale_value,
                        int32_t *terms_value, double *grad_offsets, double *scale_offsets,
                        double *grad_logits, double *scale_logits, int32_t *terms_points,
                        int nthreads)
{
    int rc = check(p);
    if (rc) return rc;
    const int N = p->N, Z = p->Z, C = p->C, H = p->heads, L = p->L, P = p->P;
    const int D = C / H;
    const int LP = L * P;
    const int64_t Q = (int64_t)p->X * p->Y;
    const int64_t S = sca_pixels(p);
    const int64_t rows = (int64_t)p->B * p->X;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    /* pass 1: per query, gradients of the offsets and logits */
#pragma omp parallel
    {
        double *attn = (double *)malloc(sizeof(double) * (size_t)H * LP);
        double *da = (double *)malloc(sizeof(double) * (size_t)LP * 6);
        float *uv = (float *)malloc(sizeof(float) * 2 * (size_t)(N * Z + 1));
        int *hit = (int *)malloc(sizeof(int) * (size_t)(N + 1));
        int32_t *kt = (int32_t *)malloc(sizeof(int32_t) * (size_t)LP);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < rows; ++r) {
            const int b = (int)(r / p->X), i = (int)(r % p->X);
            for (int j = 0; j < p->Y; ++j) {
                float *un = uv, *vn = uv + N * Z;
                const int count = prepare_query(p, l2i, zs, logits, b, i, j, un, vn, hit, attn);
                const double alpha = (p->reduce == 0 && count > 1) ? 1.0 / (double)count : 1.0;
                const int64_t q = (int64_t)i * p->Y + j;
                const float *off = offsets + ((size_t)b * Q + q) * (size_t)H * LP * 2;
                const float *g = grad_out + ((size_t)b * Q + q) * C;
                for (int h = 0; h < H; ++h) {
                    /* da[t]: d a; da[LP + t], da[2LP + t]: d x, d y (before alpha a);
                     * da[3LP..]: their scales */
                    for (int t = 0; t < 6 * LP; ++t) da[t] = 0.0;
                    for (int t = 0; t < LP; ++t) kt[t] = 0;
                    for (int n = 0; n < N; ++n) {
                        if (!hit[n]) continue;
                        const float *vcam = value + ((size_t)b * N + n) * (size_t)S * C;
                        int64_t start = 0;
                        for (int l = 0; l < L; ++l) {
                            for (int k = 0; k < P; ++k) {
                                const int z = anchor_of_point(k, P, Z);
                                const int t = l * P + k;
                                corners cr;
                                double ax, ay;
                                if (!point_corners(p, l, start, un[n * Z + z], vn[n * Z + z],
                                                   off + (((size_t)h * L + l) * P + k) * 2, &cr,
                                                   &ax, &ay))
                                    continue;
                                for (int c4 = 0; c4 < 4; ++c4) kt[t] += cr.in[c4];
                                for (int e = 0; e < D; ++e) {
                                    double v[4];
                                    for (int c4 = 0; c4 < 4; ++c4)
                                        v[c4] = cr.in[c4]
                                            ? (double)vcam[(size_t)cr.pix[c4] * C + (size_t)h * D + e]
                                            : 0.0;
                                    const double ge = (double)g[h * D + e];
                                    double smp = 0.0, mag = 0.0;
                                    for (int c4 = 0; c4 < 4; ++c4) {
                                        smp += cr.w[c4] * v[c4];
                                        mag += cr.w[c4] * fabs(v[c4]);
                                    }
                                    da[t] += ge * smp;
                                    da[3 * LP + t] += fabs(ge) * mag;
                                    /* corners: 0 = (x0, y0), 1 = (x0 + 1, y0), 2 = (x0, y0 + 1), 3 */
                                    da[LP + t] += ge * ((1.0 - ay) * (v[1] - v[0]) + ay * (v[3] - v[2]));
                                    da[4 * LP + t] += fabs(ge) * ((1.0 - ay) * (fabs(v[1]) + fabs(v[0]))
                                                                  + ay * (fabs(v[3]) + fabs(v[2])));
                                    da[2 * LP + t] += ge * ((1.0 - ax) * (v[2] - v[0]) + ax * (v[3] - v[1]));
                                    da[5 * LP + t] += fabs(ge) * ((1.0 - ax) * (fabs(v[2]) + fabs(v[0]))
                                                                  + ax * (fabs(v[3]) + fabs(v[1])));
                                }
                            }
                            start += (int64_t)p->level_h[l] * p->level_w[l];
                        }
                    }
                    /* softmax backward over the head's L*P pairs */
                    const double *a = attn + (size_t)h * LP;
                    double dot = 0.0, sdot = 0.0;
                    for (int t = 0; t < LP; ++t) {
                        dot += a[t] * alpha * da[t];
                        sdot += a[t] * alpha * da[3 * LP + t];
                    }
                    const size_t o = (((size_t)b * Q + q) * H + h) * LP;
                    for (int t = 0; t < LP; ++t) {
                        grad_logits[o + t] = a[t] * (alpha * da[t] - dot);
                        if (scale_logits) scale_logits[o + t] = a[t] * (alpha * da[3 * LP + t] + sdot);
                        grad_offsets[(o + t) * 2 + 0] = alpha * a[t] * da[LP + t];
                        grad_offsets[(o + t) * 2 + 1] = alpha * a[t] * da[2 * LP + t];
                        if (scale_offsets) {
                            scale_offsets[(o + t) * 2 + 0] = alpha * a[t] * da[4 * LP + t];
                            scale_offsets[(o + t) * 2 + 1] = alpha * a[t] * da[5 * LP + t];
                        }
                        if (terms_points) terms_points[o + t] = kt[t];
                    }
                }
            }
        }
        free(attn); free(da); free(uv); free(hit); free(kt);
    }
    /* pass 2: value scatter, one camera (b, n) per task */
#pragma omp parallel
    {
        double *attn = (double *)malloc(sizeof(double) * (size_t)H * LP);
        float *uv = (float *)malloc(sizeof(float) * 2 * (size_t)(N * Z + 1));
        int *hit = (int *)malloc(sizeof(int) * (size_t)(N + 1));
#pragma omp for schedule(dynamic, 1)
        for (int64_t bn = 0; bn < (int64_t)p->B * N; ++bn) {
            const int b = (int)(bn / N), n = (int)(bn % N);
            double *gv = grad_value + (size_t)bn * S * C;
            double *sv = scale_value ? scale_value + (size_t)bn * S * C : NULL;
            int32_t *tv = terms_value ? terms_value + (size_t)bn * S * H : NULL;
            memset(gv, 0, sizeof(double) * (size_t)S * C);
            if (sv) memset(sv, 0, sizeof(double) * (size_t)S * C);
            if (tv) memset(tv, 0, sizeof(int32_t) * (size_t)S * H);
            for (int i = 0; i < p->X; ++i)
                for (int j = 0; j < p->Y; ++j) {
                    float *un = uv, *vn = uv + N * Z;
                    const int count = prepare_query(p, l2i, zs, logits, b, i, j, un, vn, hit, attn);
                    if (!hit[n]) continue;
                    const double alpha = (p->reduce == 0 && count > 1) ? 1.0 / (double)count : 1.0;
                    const int64_t q = (int64_t)i * p->Y + j;
                    const float *off = offsets + ((size_t)b * Q + q) * (size_t)H * LP * 2;
                    const float *g = grad_out + ((size_t)b * Q + q) * C;
                    for (int h = 0; h < H; ++h) {
                        int64_t start = 0;
                        for (int l = 0; l < L; ++l) {
                            for (int k = 0; k < P; ++k) {
                                const int z = anchor_of_point(k, P, Z);
                                corners cr;
                                double ax, ay;
                                if (!point_corners(p, l, start, un[n * Z + z], vn[n * Z + z],
                                                   off + (((size_t)h * L + l) * P + k) * 2, &cr,
                                                   &ax, &ay))
                                    continue;
                                const double wa = alpha * attn[(size_t)h * LP + l * P + k];
                                for (int c4 = 0; c4 < 4; ++c4) {
                                    if (!cr.in[c4]) continue;
                                    double *dst = gv + (size_t)cr.pix[c4] * C + (size_t)h * D;
                                    for (int e = 0; e < D; ++e) {
                                        const double term = wa * cr.w[c4] * (double)g[h * D + e];
                                        dst[e] += term;
                                        if (sv) sv[(size_t)cr.pix[c4] * C + (size_t)h * D + e] += fabs(term);
                                    }
                                    if (tv) tv[(size_t)cr.pix[c4] * H + h] += 1;
                                }
                            }
                            start += (int64_t)p->level_h[l] * p->level_w[l];
                        }
                    }
                }
        }
        free(attn); free(uv); free(hit);
    }
    return 0;
}
