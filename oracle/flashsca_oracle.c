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
 * Readings (each one is also listed in the design doc):
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
                const int Hl = p->level_h[l], Wl = p->level_w[l];
                for (int k = 0; k < P; ++k) {
                    const int z = k % Z;                 /* the point's anchor */
                    const float *o = off + (((size_t)h * L + l) * P + k) * 2;
                    float sx = un[n * Z + z] * (float)Wl;
                    float sy = vn[n * Z + z] * (float)Hl;
                    sx = sx + o[0];
                    sy = sy + o[1];
                    const float xim = sx - 0.5f;
                    const float yim = sy - 0.5f;
                    /* no corner inside the map (also non-finite locations) */
                    if (!(xim > -1.0f && xim < (float)Wl && yim > -1.0f && yim < (float)Hl))
                        continue;
                    const float x0f = floorf(xim), y0f = floorf(yim);
                    const double ax = (double)(xim - x0f), ay = (double)(yim - y0f);
                    const int x0 = (int)x0f, y0 = (int)y0f;
                    const double a = attn[(h * L + l) * P + k];
                    for (int ty = 0; ty < 2; ++ty)
                        for (int tx = 0; tx < 2; ++tx) {
                            const int xt = x0 + tx, yt = y0 + ty;
                            if (xt < 0 || xt >= Wl || yt < 0 || yt >= Hl) continue;
                            const double w = (tx ? ax : 1.0 - ax) * (ty ? ay : 1.0 - ay);
                            const float *row = vcam + (size_t)(start + (int64_t)yt * Wl + xt) * C
                                               + (size_t)h * D;
                            for (int e = 0; e < D; ++e) {
                                const double t = a * w * (double)row[e];
                                acc[h * D + e] += t;
                                scale[h * D + e] += fabs(t);
                            }
                            terms[h] += 1;
                            if (cnt) cnt->taps += 1;
                        }
                }
                start += (int64_t)Hl * Wl;
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
