// FlashSCA forward for gfx950: BEVFormer's spatial cross-attention with the
// per-camera sampling points formed on the fly (FlashBEV paper, Sec. 4.5,
// Table 7), behind the C ABI declared in include/flashsca.h.
//
// Execution design (MI355X-first):
//   * Work items are (query, head) pairs, "slots".  A slot owns `lph` lanes
//     (a power of two); lane `sub` of a slot holds one LW-byte slice of the
//     head's D channels, so every bilinear tap of the head is one coalesced
//     run of D * elem bytes across the slot's lanes.  A wavefront holds
//     64 / lph slots; a workgroup a tile of consecutive pairs of one batch
//     element.
//   * Phase 1 (workgroup): every (query, camera) pair of the tile projects the
//     query's Z anchors (float32 recipe, IEEE divisions), records the
//     normalized reference points in LDS and sets the camera's bit in the
//     query's hit mask (LDS atomic OR).
//   * Phase 2 (slot): softmax over the head's L * P logits, read once per
//     query (not once per camera); the attention weights, already multiplied
//     by 1 / max(1, hits), go to the slot's LDS area.
//   * Phase 3 (slot, per hit camera): in chunks of lph points, lane `sub`
//     sets up point c + sub (anchor k mod Z, location (u W_l + dx) - 1/2,
//     floor, four tap offsets and weights a * w) and publishes them in LDS;
//     then all lanes of the slot gather the chunk's lph * 4 taps with raw
//     buffer loads and accumulate their channels in float32.  A tap outside
//     the map gets an offset past the end of the camera's buffer, so its load
//     returns zero without a memory access.
//   * Each output element is written once; no atomics on global memory, no
//     workspace, one launch.
// Coordinates follow the float32 recipe of the conventions in flashsca.h, so
// mask and floor decisions match the CPU oracle bit for bit: the file is
// compiled with -ffp-contract=off and uses IEEE division.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include "flashbev.h"
#include "flashsca.h"
#include "hip_common.h"

namespace {

constexpr int kScaWave = 64;
constexpr int kScaWavesMax = 4;
constexpr int kScaThreads = kScaWave * kScaWavesMax;
constexpr int kScaXcds = 8;      // MI355X: workgroups are dispatched to 8 XCDs round-robin
constexpr int kScaBlock = 32;    // queries are visited in blocks of 32 x 32 BEV cells
// Offset of a tap that is not loaded: one camera's value is smaller than
// 2 GiB and a lane adds less than 1 KiB, so the load is past the buffer's end
// and returns zero without touching memory.
constexpr uint32_t kScaNoTap = 0x80000000u;
constexpr uint64_t kScaCamBytesMax = 0x7FFFFFFFull;
constexpr uint32_t kScaLdsBudget = 64u * 1024u;
// a chunk record: 4 tap offsets then 4 weights (8 dwords) per lane, and a
// 4-dword pad per slot so that the slots' broadcast reads hit different banks
constexpr int kTapDwords = 8;
constexpr int kSlotPad = 4;

struct ScaParams {
    const void *value;
    const float *l2i;
    const float *offsets;
    const float *logits;
    float *out;
    uint64_t cam_bytes;     // bytes of one camera's value maps (S C elem)
    uint32_t row_bytes;     // C * elem
    uint32_t head_bytes;    // D * elem
    int32_t B, N, C, heads, D, L, P, Z, LP;
    int32_t X, Y, Q;
    int32_t lph;            // lanes per slot (power of two)
    int32_t lph_shift;      // log2(lph)
    int32_t spw;            // slots per wavefront
    int32_t tile_pairs;     // (query, head) pairs per workgroup
    int32_t tiles_per_b;
    int32_t stripe;         // consecutive tiles an XCD takes in turn (about one block)
    int32_t nq_max;         // queries a tile can touch
    int32_t slot_stride;    // dwords per slot in the chunk-record area
    float img_w, img_h;
    float x_min, dx, y_min, dy, depth_eps;
    int32_t reduce;
    float rcp_p, rcp_z;     // float32 1 / P and 1 / Z for div_small
    float level_wf[FLASHSCA_LMAX], level_hf[FLASHSCA_LMAX];
    int32_t level_w[FLASHSCA_LMAX], level_h[FLASHSCA_LMAX];
    uint32_t level_start[FLASHSCA_LMAX];   // first pixel of each level
    // LDS layout (byte offsets)
    uint32_t lds_mat, lds_lvl, lds_z, lds_ref, lds_hit, lds_att, lds_tap;
    float z[FLASHSCA_ZMAX];
};

// LDS: camera matrices [N][12]; level table [5][LMAX]; anchors [Z];
// reference points [nq_max][N][Z] float2; hit masks [nq_max]; attention
// weights [waves][spw][LP]; chunk records [waves][spw][slot_stride].
struct ScaLds {
    uint32_t mat, lvl, z, ref, hit, att, tap, total;
};

__host__ inline uint32_t sca_align16(uint32_t v) { return (v + 15u) & ~15u; }

__host__ ScaLds sca_lds_layout(int N, int Z, int nq_max, int waves, int spw, int LP,
                               int slot_stride)
{
    ScaLds s;
    uint32_t o = 0;
    s.mat = o; o = sca_align16(o + (uint32_t)N * 12u * 4u);
    s.lvl = o; o = sca_align16(o + 5u * FLASHSCA_LMAX * 4u);
    s.z = o; o = sca_align16(o + (uint32_t)Z * 4u);
    s.ref = o; o = sca_align16(o + (uint32_t)nq_max * N * Z * 8u);
    s.hit = o; o = sca_align16(o + (uint32_t)nq_max * 4u);
    s.att = o; o = sca_align16(o + (uint32_t)waves * spw * LP * 4u);
    s.tap = o; o = sca_align16(o + (uint32_t)waves * spw * slot_stride * 4u);
    s.total = o;
    return s;
}

// Cell (i, j) of the query of rank r in the blocked visiting order: the grid
// is cut into bands of kScaBlock rows; a band into blocks of kScaBlock
// columns (the last band and block may be narrower); blocks follow each other
// along the band, and a block's cells are row-major.  A bijection of
// [0, X Y) onto the cells.
__device__ __forceinline__ void query_of(int r, int X, int Y, int &i, int &j)
{
    const int band_cells = kScaBlock * Y;
    const int R = r / band_cells;
    const int s = r - R * band_cells;
    const int h = min(kScaBlock, X - R * kScaBlock);
    const int c = s / (h * kScaBlock);
    const int t = s - c * h * kScaBlock;
    const int w = min(kScaBlock, Y - c * kScaBlock);
    const int ti = t / w;
    i = R * kScaBlock + ti;
    j = c * kScaBlock + (t - ti * w);
}

template <int DT, int LW>
__global__ void __launch_bounds__(kScaThreads)
sca_fwd(const ScaParams p)
{
    constexpr int ES = ElemSize<DT>::value;
    constexpr int EPV = LW / ES;   // elements per lane slice
    extern __shared__ __align__(16) unsigned char smem[];
    float *s_mat = reinterpret_cast<float *>(smem + p.lds_mat);
    float *s_lwf = reinterpret_cast<float *>(smem + p.lds_lvl);
    float *s_lhf = s_lwf + FLASHSCA_LMAX;
    int32_t *s_lw = reinterpret_cast<int32_t *>(s_lhf + FLASHSCA_LMAX);
    int32_t *s_lh = s_lw + FLASHSCA_LMAX;
    uint32_t *s_lst = reinterpret_cast<uint32_t *>(s_lh + FLASHSCA_LMAX);
    float *s_z = reinterpret_cast<float *>(smem + p.lds_z);
    float2 *s_ref = reinterpret_cast<float2 *>(smem + p.lds_ref);
    uint32_t *s_hit = reinterpret_cast<uint32_t *>(smem + p.lds_hit);
    float *s_att = reinterpret_cast<float *>(smem + p.lds_att);
    uint32_t *s_tap = reinterpret_cast<uint32_t *>(smem + p.lds_tap);

    const int tid = threadIdx.x;
    const int nthreads = blockDim.x;
    const int wave = tid / kScaWave;
    const int lane = tid % kScaWave;
    const int N = p.N, Z = p.Z;

    // XCD-aware tile order.  Queries are visited block by block (see
    // query_of), so consecutive tiles cover a compact patch of the BEV whose
    // samples land on overlapping pixels.  The k-th workgroup on XCD x takes
    // tile (k / S) * 8S + x * S + k % S with S = p.stripe (about one block):
    // an XCD works through whole blocks, its resident workgroups share their
    // pixels in its L2, and the blocks of the 8 XCDs interleave over the
    // grid (a like mix of heavy and light regions).  The tail that does not
    // fill 8 stripes is split the same way with shorter stripes.
    const int g = blockIdx.x;
    const int S8 = kScaXcds * p.stripe;
    const int full = (int)(gridDim.x / S8) * S8;
    int tile = g;
    if (g < full) {
        const int xcd = g % kScaXcds, k = g / kScaXcds;
        tile = (k / p.stripe) * S8 + xcd * p.stripe + k % p.stripe;
    } else {
        const int rem = (int)gridDim.x - full;
        const int s2 = rem / kScaXcds;
        if (g - full < s2 * kScaXcds) {
            const int xcd = (g - full) % kScaXcds, k = (g - full) / kScaXcds;
            tile = full + xcd * s2 + k;
        }
    }
    const int b = tile / p.tiles_per_b;
    const int64_t pair0 = (int64_t)(tile - b * p.tiles_per_b) * p.tile_pairs;
    const int r_first = (int)(pair0 / p.heads);   // first query rank of the tile
    const int64_t pairs_b = (int64_t)p.Q * p.heads;

    for (int t = tid; t < N * 12; t += nthreads) {
        const int n = t / 12, r = t - n * 12;
        s_mat[t] = p.l2i[((size_t)b * N + n) * 16 + r];
    }
    if (tid < FLASHSCA_LMAX) {
        s_lwf[tid] = p.level_wf[tid];
        s_lhf[tid] = p.level_hf[tid];
        s_lw[tid] = p.level_w[tid];
        s_lh[tid] = p.level_h[tid];
        s_lst[tid] = p.level_start[tid];
    }
    for (int t = tid; t < Z; t += nthreads) s_z[t] = p.z[t];
    for (int t = tid; t < p.nq_max; t += nthreads) s_hit[t] = 0u;
    __syncthreads();

    // ---- phase 1: reference points of the tile's queries in every camera
    for (int t = tid; t < p.nq_max * N; t += nthreads) {
        const int qi = t / N, n = t - qi * N;
        const int rank = r_first + qi;
        if (rank >= p.Q) continue;
        int i, j;
        query_of(rank, p.X, p.Y, i, j);
        const float x = p.x_min + ((float)i + 0.5f) * p.dx;
        const float y = p.y_min + ((float)j + 0.5f) * p.dy;
        const float *m = s_mat + n * 12;
        bool any = false;
        for (int k = 0; k < Z; ++k) {
            const float z = s_z[k];
            // (u', v', d) = P[b,n] (x, y, z, 1), left to right, no contraction
            const float up = ((m[0] * x + m[1] * y) + m[2] * z) + m[3];
            const float vp = ((m[4] * x + m[5] * y) + m[6] * z) + m[7];
            const float d = ((m[8] * x + m[9] * y) + m[10] * z) + m[11];
            const bool in_front = d > p.depth_eps;
            const float dd = in_front ? d : p.depth_eps;
            const float un = (up / dd) / p.img_w;
            const float vn = (vp / dd) / p.img_h;
            s_ref[(qi * N + n) * Z + k] = make_float2(un, vn);
            any |= in_front && un > 0.0f && un < 1.0f && vn > 0.0f && vn < 1.0f;
        }
        if (any) atomicOr(&s_hit[qi], 1u << n);
    }
    __syncthreads();

    // ---- phase 2: the slot's softmax over (level, point)
    const int lph = p.lph;
    const int sub = lane & (lph - 1);
    const int slot = lane >> p.lph_shift;
    const int64_t pair = pair0 + (int64_t)wave * p.spw + slot;
    const bool active = pair < pairs_b;
    const int rank = active ? (int)(pair / p.heads) : r_first;
    const int mh = active ? (int)(pair - (int64_t)rank * p.heads) : 0;
    const int qi = rank - r_first;
    int qx, qy;
    query_of(rank, p.X, p.Y, qx, qy);
    const int q = qx * p.Y + qy;             // the query's index in offsets, logits, out
    const uint32_t hits = active ? s_hit[qi] : 0u;
    const int count = __popc(hits);
    const float inv = (p.reduce == FLASHBEV_REDUCE_VALID_MEAN && count > 1) ? 1.0f / (float)count
                                                                             : 1.0f;
    const int LP = p.LP;
    float *att = s_att + (size_t)(wave * p.spw + slot) * LP;
    const size_t pt0 = (((size_t)b * p.Q + q) * p.heads + mh) * (size_t)LP;
    if (hits) {
        float mx = -INFINITY;
        for (int j = sub; j < LP; j += lph) mx = fmaxf(mx, p.logits[pt0 + j]);
        for (int s = lph >> 1; s >= 1; s >>= 1) mx = fmaxf(mx, __shfl_xor(mx, s));
        float sum = 0.0f;
        for (int j = sub; j < LP; j += lph) {
            const float e = expf(p.logits[pt0 + j] - mx);
            att[j] = e;
            sum += e;
        }
        for (int s = lph >> 1; s >= 1; s >>= 1) sum += __shfl_xor(sum, s);
        const float r = inv / sum;
        for (int j = sub; j < LP; j += lph) att[j] *= r;
    }   // the shuffles stay inside the slot, whose lanes all take this branch or none

    // cameras any slot of the wavefront hits (wavefront-uniform)
    uint32_t cams = 0;
    for (int n = 0; n < N; ++n)
        if (__ballot((hits >> n) & 1u)) cams |= 1u << n;

    // ---- phase 3: sampling in every hit camera
    float acc[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] = 0.0f;
    const uint32_t lane_off = (uint32_t)sub * LW;
    const uint32_t head_off = (uint32_t)mh * p.head_bytes;
    uint32_t *rec_w = s_tap + (size_t)(wave * p.spw + slot) * p.slot_stride;   // this slot
    const float2 *off2 = reinterpret_cast<const float2 *>(p.offsets);

    for (int n = 0; n < N; ++n) {
        if (!((cams >> n) & 1u)) continue;
        const bool mine = (hits >> n) & 1u;
        const char *cam_base = static_cast<const char *>(p.value) +
                               ((size_t)b * N + n) * (size_t)p.cam_bytes;
        const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char *>(cam_base), (short)0, (int)p.cam_bytes, 0x00020000);
        const float2 *ref = s_ref + (size_t)(qi * N + n) * Z;
        for (int c0 = 0; c0 < LP; c0 += lph) {
            // set-up of point j = c0 + sub of this slot
            const int j = c0 + sub;
            uint32_t o0 = kScaNoTap, o1 = kScaNoTap, o2 = kScaNoTap, o3 = kScaNoTap;
            float w0 = 0.0f, w1 = 0.0f, w2 = 0.0f, w3 = 0.0f;
            if (mine && j < LP) {
                const int l = div_small(j, p.P, p.rcp_p);
                const int k = j - l * p.P;
                const int zk = k - div_small(k, Z, p.rcp_z) * Z;   // anchor k mod Z
                const float2 r = ref[zk];
                const float2 dxy = off2[pt0 + j];
                const float Wl = s_lwf[l], Hl = s_lhf[l];
                float sx = r.x * Wl;
                float sy = r.y * Hl;
                sx = sx + dxy.x;
                sy = sy + dxy.y;
                const float xim = sx - 0.5f;
                const float yim = sy - 0.5f;
                if (xim > -1.0f && xim < Wl && yim > -1.0f && yim < Hl) {
                    const float x0f = floorf(xim), y0f = floorf(yim);
                    const float ax = xim - x0f, ay = yim - y0f;
                    const int x0 = (int)x0f, y0 = (int)y0f;
                    const int wi = s_lw[l], hi = s_lh[l];
                    const float a = att[j];
                    const float wt = a * (1.0f - ay), wb = a * ay;
                    const bool xl = x0 >= 0, xr = x0 + 1 < wi;
                    const bool yt = y0 >= 0, yb = y0 + 1 < hi;
                    const int row = (int)s_lst[l] + y0 * wi + x0;
                    const uint32_t rb = p.row_bytes;
                    if (xl && yt) { o0 = (uint32_t)row * rb + head_off; w0 = wt * (1.0f - ax); }
                    if (xr && yt) { o1 = (uint32_t)(row + 1) * rb + head_off; w1 = wt * ax; }
                    if (xl && yb) { o2 = (uint32_t)(row + wi) * rb + head_off; w2 = wb * (1.0f - ax); }
                    if (xr && yb) { o3 = (uint32_t)(row + wi + 1) * rb + head_off; w3 = wb * ax; }
                }
            }
            uint32_t *mine_rec = rec_w + sub * kTapDwords;
            *reinterpret_cast<uint4 *>(mine_rec) = make_uint4(o0, o1, o2, o3);
            *reinterpret_cast<float4 *>(mine_rec + 4) = make_float4(w0, w1, w2, w3);
            wave_lds_sync();
            // gather the chunk's points: every lane of the slot, its channels
            const int npts = (LP - c0) < lph ? (LP - c0) : lph;
#pragma unroll 4
            for (int t = 0; t < npts; ++t) {
                const uint4 o = *reinterpret_cast<const uint4 *>(rec_w + t * kTapDwords);
                const float4 w = *reinterpret_cast<const float4 *>(rec_w + t * kTapDwords + 4);
                const Raw<LW> v0 = load_vec<LW>(rsrc, o.x + lane_off, 0);
                const Raw<LW> v1 = load_vec<LW>(rsrc, o.y + lane_off, 0);
                const Raw<LW> v2 = load_vec<LW>(rsrc, o.z + lane_off, 0);
                const Raw<LW> v3 = load_vec<LW>(rsrc, o.w + lane_off, 0);
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    float s = acc[e];
                    s = fmaf(w.x, elem<DT, LW>(v0, e), s);
                    s = fmaf(w.y, elem<DT, LW>(v1, e), s);
                    s = fmaf(w.z, elem<DT, LW>(v2, e), s);
                    s = fmaf(w.w, elem<DT, LW>(v3, e), s);
                    acc[e] = s;
                }
            }
            wave_lds_sync();
        }
    }

    // ---- store: each lane its slice of the head's channels
    if (active) {
        float *o = p.out + ((size_t)b * p.Q + q) * (size_t)p.C + (size_t)mh * p.D;
        const int e0 = sub * EPV;
#pragma unroll
        for (int e = 0; e < EPV; ++e)
            if (e0 + e < p.D) o[e0 + e] = acc[e];
    }
}

using ScaKernelFn = void (*)(const ScaParams);

template <int DT>
ScaKernelFn pick_sca_lw(int lw)
{
    switch (lw) {
    case 16: return sca_fwd<DT, 16>;
    case 8: return sca_fwd<DT, 8>;
    case 4: return sca_fwd<DT, 4>;
    default:
        if constexpr (DT == FLASHBEV_F32) return nullptr;
        else return sca_fwd<DT, 2>;
    }
}

ScaKernelFn pick_sca(int dtype, int lw)
{
    switch (dtype) {
    case FLASHBEV_F32: return pick_sca_lw<FLASHBEV_F32>(lw);
    case FLASHBEV_F16: return pick_sca_lw<FLASHBEV_F16>(lw);
    default: return pick_sca_lw<FLASHBEV_BF16>(lw);
    }
}

struct ScaPlan {
    ScaParams prm;
    int64_t workgroups;
    int threads;
    size_t lds;
    int lw;
    bool empty;
};

bool sca_finite(float v) { return v == v && v - v == 0.0f; }

bool sca_overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    if (!na || !nb) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + nb && b0 < a0 + na;
}

// All argument checks; `need_data` requires the device pointers.
int make_sca_plan(const flashsca_value *v, const float *l2i, const flashbev_bev_grid_spec *s,
                  const flashbev_z_bins *zb, int32_t P, const float *off, const float *lg,
                  const float *out, bool need_data, ScaPlan *pl)
{
    if (!v || !s || !zb) return FLASHBEV_ERR_NULLPTR;
    if (v->dtype != FLASHBEV_F32 && v->dtype != FLASHBEV_F16 && v->dtype != FLASHBEV_BF16)
        return FLASHBEV_ERR_DTYPE;
    if (v->B < 0 || v->N < 0 || v->C < 1 || v->heads < 1 || v->L < 1 || v->img_h < 1 ||
        v->img_w < 1 || s->X < 0 || s->Y < 0 || zb->Z < 1 || P < 1)
        return FLASHBEV_ERR_SHAPE;
    if (v->C % v->heads != 0 || P % zb->Z != 0) return FLASHBEV_ERR_SHAPE;
    if (v->L > FLASHSCA_LMAX) return FLASHBEV_ERR_UNSUPPORTED;
    uint64_t S = 0;
    for (int l = 0; l < v->L; ++l) {
        if (v->level_h[l] < 1 || v->level_w[l] < 1) return FLASHBEV_ERR_SHAPE;
        S += (uint64_t)v->level_h[l] * (uint64_t)v->level_w[l];
    }
    if (v->N > FLASHSCA_NMAX || zb->Z > FLASHSCA_ZMAX || (int64_t)v->L * P > FLASHSCA_LPMAX)
        return FLASHBEV_ERR_UNSUPPORTED;
    if (!zb->z) return FLASHBEV_ERR_NULLPTR;
    if (s->reduce != FLASHBEV_REDUCE_VALID_MEAN && s->reduce != FLASHBEV_REDUCE_SUM)
        return FLASHBEV_ERR_VALUE;
    if (!sca_finite(s->x_min) || !sca_finite(s->dx) || !sca_finite(s->y_min) ||
        !sca_finite(s->dy) || !sca_finite(s->depth_eps))
        return FLASHBEV_ERR_VALUE;
    const int es = (v->dtype == FLASHBEV_F32) ? 4 : 2;
    const int D = v->C / v->heads;
    const uint64_t head_bytes = (uint64_t)D * es;
    const uint64_t row = (uint64_t)v->C * es;
    if (head_bytes > FLASHSCA_HEAD_BYTES_MAX) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t cam_bytes = S * row;
    if (cam_bytes > kScaCamBytesMax) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t Q = (uint64_t)s->X * s->Y;
    if (Q > 0x7FFFFFFFull || Q * (uint64_t)v->heads > 0x7FFFFFFFull)
        return FLASHBEV_ERR_UNSUPPORTED;
    const int LP = v->L * P;
    const uint64_t out_elems = (uint64_t)v->B * Q * v->C;
    const bool empty = out_elems == 0;
    const uint64_t value_bytes = (uint64_t)v->B * v->N * cam_bytes;
    const uint64_t pts = (uint64_t)v->B * Q * v->heads * LP;
    if (need_data && !empty) {
        if (!out || !off || !lg) return FLASHBEV_ERR_NULLPTR;
        if (value_bytes > 0 && !v->data) return FLASHBEV_ERR_NULLPTR;
        if (v->N > 0 && !l2i) return FLASHBEV_ERR_NULLPTR;
        if (((uintptr_t)v->data % es) || ((uintptr_t)l2i % 4) || ((uintptr_t)out % 4) ||
            ((uintptr_t)off % 4) || ((uintptr_t)lg % 4))
            return FLASHBEV_ERR_ALIGN;
        const size_t ob = out_elems * 4;
        if (sca_overlaps(out, ob, v->data, value_bytes) ||
            sca_overlaps(out, ob, l2i, (size_t)v->B * v->N * 64) ||
            sca_overlaps(out, ob, off, pts * 8) || sca_overlaps(out, ob, lg, pts * 4))
            return FLASHBEV_ERR_ALIAS;
    }
    // the offsets travel as float2 loads
    if (need_data && !empty && ((uintptr_t)off % 8)) return FLASHBEV_ERR_ALIGN;

    // lane slice: 16 bytes where a head row has at least four of them
    // (measured on MI355X, BEVFormer-base bfloat16: 16-byte lanes, 4 per head,
    // 0.521 -> 0.484 ms against 8-byte lanes, 8 per head), else narrower;
    // always a width dividing the head row, the full row and the base address
    int lw = 16;
    while (lw > es && (uint64_t)lw * 4 > head_bytes) lw >>= 1;
    while (lw > es && ((head_bytes % lw) != 0 || (row % lw) != 0 ||
                       (((uintptr_t)v->data) % lw) != 0))
        lw >>= 1;
    const int nvec = (int)((head_bytes + lw - 1) / lw);
    int lph = 1, lph_shift = 0;
    while (lph < nvec) { lph <<= 1; ++lph_shift; }
    if (lph > kScaWave) return FLASHBEV_ERR_UNSUPPORTED;
    const int spw = kScaWave / lph;
    const int slot_stride = lph * kTapDwords + kSlotPad;

    int waves = kScaWavesMax;
    int nq_max = 0;
    ScaLds lay{};
    for (;;) {
        const int tp = waves * spw;
        nq_max = (tp - 1) / v->heads + 2;
        if ((uint64_t)nq_max > Q) nq_max = (int)(Q > 0 ? Q : 1);
        lay = sca_lds_layout(v->N, zb->Z, nq_max, waves, spw, LP, slot_stride);
        if (lay.total <= kScaLdsBudget || waves == 1) break;
        waves >>= 1;
    }
    if (lay.total > kScaLdsBudget) return FLASHBEV_ERR_UNSUPPORTED;
    const int tile_pairs = waves * spw;

    ScaParams &p = pl->prm;
    memset(&p, 0, sizeof(p));
    p.value = v->data;
    p.l2i = l2i;
    p.offsets = off;
    p.logits = lg;
    p.out = const_cast<float *>(out);
    p.cam_bytes = cam_bytes;
    p.row_bytes = (uint32_t)row;
    p.head_bytes = (uint32_t)head_bytes;
    p.B = v->B; p.N = v->N; p.C = v->C; p.heads = v->heads; p.D = D;
    p.L = v->L; p.P = P; p.Z = zb->Z; p.LP = LP;
    p.X = s->X; p.Y = s->Y; p.Q = (int32_t)Q;
    p.lph = lph;
    p.lph_shift = lph_shift;
    p.spw = spw;
    p.tile_pairs = tile_pairs;
    const uint64_t pairs_b = Q * (uint64_t)v->heads;
    p.tiles_per_b = (int32_t)((pairs_b + tile_pairs - 1) / tile_pairs);
    {
        const int64_t st = (int64_t)kScaBlock * kScaBlock * v->heads / tile_pairs;
        p.stripe = (int32_t)(st < 1 ? 1 : (st > 4096 ? 4096 : st));
    }
    p.nq_max = nq_max;
    p.slot_stride = slot_stride;
    p.img_w = (float)v->img_w;
    p.img_h = (float)v->img_h;
    p.x_min = s->x_min; p.dx = s->dx; p.y_min = s->y_min; p.dy = s->dy;
    p.depth_eps = s->depth_eps;
    p.reduce = s->reduce;
    p.rcp_p = 1.0f / (float)P;
    p.rcp_z = 1.0f / (float)zb->Z;
    uint32_t start = 0;
    for (int l = 0; l < v->L; ++l) {
        p.level_w[l] = v->level_w[l];
        p.level_h[l] = v->level_h[l];
        p.level_wf[l] = (float)v->level_w[l];
        p.level_hf[l] = (float)v->level_h[l];
        p.level_start[l] = start;
        start += (uint32_t)(v->level_h[l] * v->level_w[l]);
    }
    p.lds_mat = lay.mat;
    p.lds_lvl = lay.lvl;
    p.lds_z = lay.z;
    p.lds_ref = lay.ref;
    p.lds_hit = lay.hit;
    p.lds_att = lay.att;
    p.lds_tap = lay.tap;
    for (int k = 0; k < zb->Z; ++k) p.z[k] = zb->z[k];

    pl->workgroups = empty ? 0 : (int64_t)v->B * p.tiles_per_b;
    if (pl->workgroups > 0x7FFFFFFFll) return FLASHBEV_ERR_UNSUPPORTED;
    pl->threads = waves * kScaWave;
    pl->lds = lay.total;
    pl->lw = lw;
    pl->empty = empty;
    return FLASHBEV_OK;
}

}  // namespace

extern "C" int flashsca_launch_info(const flashsca_value *value,
                                    const flashbev_bev_grid_spec *spec,
                                    const flashbev_z_bins *anchors, int32_t P, int64_t *workgroups,
                                    int32_t *threads_per_workgroup, int32_t *lds_bytes,
                                    int32_t *lanes_per_head, int32_t *lane_bytes)
{
    ScaPlan pl;
    const int rc = make_sca_plan(value, nullptr, spec, anchors, P, nullptr, nullptr, nullptr,
                                 false, &pl);
    if (rc) return rc;
    if (workgroups) *workgroups = pl.workgroups;
    if (threads_per_workgroup) *threads_per_workgroup = pl.threads;
    if (lds_bytes) *lds_bytes = (int32_t)pl.lds;
    if (lanes_per_head) *lanes_per_head = pl.prm.lph;
    if (lane_bytes) *lane_bytes = pl.lw;
    return FLASHBEV_OK;
}

extern "C" int flashsca_forward(const flashsca_value *value, const float *lidar2img,
                                const flashbev_bev_grid_spec *spec,
                                const flashbev_z_bins *anchors, int32_t P, const float *offsets,
                                const float *logits, float *out, void *stream)
{
    ScaPlan pl;
    const int rc = make_sca_plan(value, lidar2img, spec, anchors, P, offsets, logits, out, true,
                                 &pl);
    if (rc) return rc;
    if (pl.empty) return FLASHBEV_OK;
    const ScaKernelFn fn = pick_sca(value->dtype, pl.lw);
    if (!fn) return FLASHBEV_ERR_UNSUPPORTED;
    void *args[] = {&pl.prm};
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(fn),
                                         dim3((unsigned)pl.workgroups), dim3(pl.threads), args,
                                         pl.lds, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? FLASHBEV_OK : FLASHBEV_ERR_HIP;
}
