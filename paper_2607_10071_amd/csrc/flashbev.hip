// Fused Sampling-VT forward for gfx950 (FlashBEV paper, Sec. 3.3, Alg. 2,
// evaluating Eq. 1), behind the C ABI declared in include/flashbev.h.
//
// Execution design (MI355X-first; the paper's one-thread-per-(b,x,y,c)
// mapping is not used):
//   * A wavefront owns `cpw` consecutive BEV cells of one batch element.
//     Lanes span the channels of a cell: each lane holds LW-byte vectors of
//     the channel-last feature row, so the four bilinear taps of a sample
//     are fully coalesced row loads across the lanes of a cell.
//   * Projection, masking and bilinear set-up are done once per
//     (cell, height, camera), not once per channel (the paper recomputes
//     them per channel, Sec. 3.3.3).  One pass maps the 64 lanes to
//     (height, camera) pairs of one cell; a ballot gives the per-height
//     camera count den_z and a deterministic compaction of the valid
//     samples into a per-wave LDS list.
//   * The per-height valid mean is folded into the tap weights
//     (w / max(1, den_z)), so the gather loop is one flat weighted sum over
//     the cell's valid samples held in float32 registers (Eq. 1
//     re-associated; only rounding changes).
//   * Camera matrices and heights are staged in LDS once per workgroup.
//   * Tap loads are raw buffer loads with 32-bit offsets; every address is
//     inside the feature tensor by construction (out-of-range taps get
//     weight zero on an in-range pixel), and the buffer descriptor bounds
//     them as well.
//   * Each output element is written exactly once; no atomics, no
//     workspace, one launch.
//
// Coordinates follow a fixed float32 recipe so that mask and floor
// decisions match the CPU oracle bit for bit: the file is compiled with
// -ffp-contract=off (every product and sum rounded on its own) and the
// perspective divide is IEEE division.  The gather uses explicit fmaf.
#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include "flashbev.h"

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;                 // wavefronts per workgroup
constexpr int kThreads = kWave * kWaves;  // 256
constexpr int kCpwMax = 8;                // BEV cells per wavefront (upper bound)
constexpr int kRecCap = 64;               // valid samples per (cell, projection pass)
constexpr int kUnroll = 2;                // samples gathered per loop iteration
// Offset of a tap that is not loaded: feature tensors are smaller than
// 2 GiB and the tap steps are smaller than the tensor, so this offset plus
// any step stays past the buffer (no 32-bit wrap) and the load returns zero
// without touching memory.
constexpr uint32_t kNoTap = 0x80000000u;
constexpr uint64_t kFeatBytesMax = 0x7FFFFFFFull;

struct Params {
    const void *feat;
    const float *l2i;
    float *out;
    uint32_t feat_bytes;   // buffer size for the descriptor
    int32_t B, N, H, W, C, X, Y, Z;
    int32_t XY;
    int32_t tiles_per_b;   // workgroups per batch element
    float img_w, img_h;    // image size as float
    float sx, sy;          // W / img_w, H / img_h (float32, computed once)
    float x_min, dx, y_min, dy, depth_eps;
    int32_t reduce;        // 0 valid mean, 1 sum
    uint32_t row_bytes;    // C * element size
    uint32_t step_x;       // byte step to the right-hand tap (0 if W == 1)
    uint32_t step_y;       // byte step to the lower tap (0 if H == 1)
    int32_t nvec;          // LW-byte vectors per feature row
    int32_t lpc;           // lanes per cell
    int32_t cpw;           // cells per wavefront
    int32_t zc;            // heights per projection pass
    float z[FLASHBEV_ZMAX];
};

// ---------------------------------------------------------------------------
// feature vector loads and conversion to float32
// ---------------------------------------------------------------------------
template <int DT>
struct ElemSize { static constexpr int value = (DT == FLASHBEV_F32) ? 4 : 2; };

template <int LW>
struct Raw;
template <>
struct Raw<16> { uint32_t w[4]; };
template <>
struct Raw<8> { uint32_t w[2]; };
template <>
struct Raw<4> { uint32_t w[1]; };
template <>
struct Raw<2> { uint32_t w[1]; };

template <int LW>
__device__ __forceinline__ Raw<LW> load_vec(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff,
                                            uint32_t soff)
{
    Raw<LW> r;
    if constexpr (LW == 16) {
        auto v = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff, soff, 0);
        r.w[0] = v[0]; r.w[1] = v[1]; r.w[2] = v[2]; r.w[3] = v[3];
    } else if constexpr (LW == 8) {
        auto v = __builtin_amdgcn_raw_buffer_load_b64(rsrc, voff, soff, 0);
        r.w[0] = v[0]; r.w[1] = v[1];
    } else if constexpr (LW == 4) {
        r.w[0] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, voff, soff, 0);
    } else {
        r.w[0] = __builtin_amdgcn_raw_buffer_load_b16(rsrc, voff, soff, 0);
    }
    return r;
}

// element e of a raw vector as float32 (exact for every input type)
template <int DT, int LW>
__device__ __forceinline__ float elem(const Raw<LW> &r, int e)
{
    if constexpr (DT == FLASHBEV_F32) {
        return __builtin_bit_cast(float, r.w[e]);
    } else if constexpr (DT == FLASHBEV_BF16) {
        uint32_t w = r.w[e >> 1];
        uint32_t bits = (e & 1) ? (w & 0xffff0000u) : (w << 16);
        return __builtin_bit_cast(float, bits);
    } else {
        uint32_t w = r.w[e >> 1];
        uint16_t h = (e & 1) ? (uint16_t)(w >> 16) : (uint16_t)(w & 0xffffu);
        return (float)__builtin_bit_cast(_Float16, h);
    }
}

__device__ __forceinline__ void wave_lds_sync()
{
    // LDS written by this wavefront must be visible to its later LDS reads,
    // and earlier reads must finish before the next writes.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Dynamic LDS layout of one workgroup.
struct Lds {
    float *mat;      // [N][12]   rows 0..2 of each camera matrix
    float *z;        // [Z]
    int *cnt;        // [kWaves][kCpwMax] valid samples per cell in this pass
    float4 *w;       // [kWaves][cpw][kRecCap] tap weights (den folded in)
    uint32_t *off;   // [kWaves][cpw][kRecCap] byte offset of the top-left tap
};

__host__ __device__ inline size_t lds_bytes_for(int cpw)
{
    size_t b = 0;
    b += sizeof(float) * FLASHBEV_NMAX * 12;
    b += sizeof(float) * FLASHBEV_ZMAX;
    b += sizeof(int) * kWaves * kCpwMax;
    b += sizeof(float4) * (size_t)kWaves * cpw * kRecCap;
    b += sizeof(uint32_t) * (size_t)kWaves * cpw * kRecCap;
    return b;
}

__device__ inline Lds carve(unsigned char *base, int cpw)
{
    Lds l;
    l.mat = reinterpret_cast<float *>(base);
    l.z = l.mat + FLASHBEV_NMAX * 12;
    l.cnt = reinterpret_cast<int *>(l.z + FLASHBEV_ZMAX);
    l.w = reinterpret_cast<float4 *>(l.cnt + kWaves * kCpwMax);
    l.off = reinterpret_cast<uint32_t *>(l.w + (size_t)kWaves * cpw * kRecCap);
    return l;
}

// ---------------------------------------------------------------------------
// the fused kernel
// ---------------------------------------------------------------------------
template <int DT, int LW, int VPL>
__global__ void __launch_bounds__(kThreads)
sample_vt_fwd(const Params p)
{
    constexpr int ES = ElemSize<DT>::value;
    constexpr int EPV = LW / ES;  // elements per vector
    extern __shared__ __align__(16) unsigned char smem[];
    const int cpw = p.cpw;
    Lds lds = carve(smem, cpw);

    const int tid = threadIdx.x;
    const int wave = tid / kWave;
    const int lane = tid % kWave;
    const int b = blockIdx.x / p.tiles_per_b;
    const int tile = blockIdx.x - b * p.tiles_per_b;
    const int N = p.N;

    // stage camera matrices (rows 0..2) and heights
    for (int t = tid; t < N * 12; t += kThreads) {
        int n = t / 12, r = t - n * 12;
        lds.mat[t] = p.l2i[((size_t)b * N + n) * 16 + r];
    }
    for (int t = tid; t < p.Z; t += kThreads) lds.z[t] = p.z[t];
    __syncthreads();

    const int q0 = (tile * kWaves + wave) * cpw;  // first cell of this wave

    // gather role: cell m_g, channel-vector slot `slot`
    const int L = p.lpc;
    const int m_g = lane / L;
    const int slot = lane - m_g * L;
    const bool g_active = (m_g < cpw) && (q0 + m_g < p.XY);
    const int m_lds = m_g < cpw ? m_g : 0;  // idle lanes address cell 0's list

    // projection role: height zl of the pass, camera n
    const int Nd = N > 0 ? N : 1;
    const int zl = lane / Nd;
    const int n_p = lane - zl * Nd;
    const uint64_t nmask = (N >= 64) ? ~0ull : ((1ull << N) - 1ull);
    const float *mrow = lds.mat + n_p * 12;

    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p.feat), (short)0,
                                          (int)p.feat_bytes, 0x00020000);
    const uint32_t cam_base = (uint32_t)b * (uint32_t)N;

    float acc[VPL][EPV];
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
        for (int e = 0; e < EPV; ++e) acc[v][e] = 0.0f;

    float4 *wl = lds.w + (size_t)wave * cpw * kRecCap;
    uint32_t *ol = lds.off + (size_t)wave * cpw * kRecCap;
    int *cl = lds.cnt + wave * kCpwMax;

    for (int z0 = 0; z0 < p.Z; z0 += p.zc) {
        // ---- phase 1: project (cell, height, camera), compact valid samples
        int maxcnt = 0;
        for (int m = 0; m < cpw; ++m) {
            const int q = q0 + m;
            if (q >= p.XY) {
                if (lane == 0) cl[m] = 0;
                continue;
            }
            const int i = q / p.Y;
            const int j = q - i * p.Y;
            // voxel centre (Alg. 2: "compute voxel center")
            const float x = p.x_min + ((float)i + 0.5f) * p.dx;
            const float y = p.y_min + ((float)j + 0.5f) * p.dy;
            const int zi = z0 + zl;
            bool ok = false;
            float xf = 0.0f, yf = 0.0f;
            if (N > 0 && zl < p.zc && zi < p.Z) {
                const float z = lds.z[zi];
                float a, bb, c;
                a = mrow[0] * x; bb = mrow[1] * y; c = mrow[2] * z;
                const float up = ((a + bb) + c) + mrow[3];
                a = mrow[4] * x; bb = mrow[5] * y; c = mrow[6] * z;
                const float vp = ((a + bb) + c) + mrow[7];
                a = mrow[8] * x; bb = mrow[9] * y; c = mrow[10] * z;
                const float d = ((a + bb) + c) + mrow[11];
                if (d > p.depth_eps) {
                    const float u = up / d;
                    const float v = vp / d;
                    if (u >= 0.0f && u < p.img_w && v >= 0.0f && v < p.img_h) {
                        ok = true;
                        xf = u * p.sx - 0.5f;
                        yf = v * p.sy - 0.5f;
                    }
                }
            }
            const uint64_t mask = __ballot(ok);
            if (ok) {
                const int den = __popcll((mask >> (zl * N)) & nmask);
                const float inv = (p.reduce == 0) ? 1.0f / (float)den : 1.0f;
                const float x0f = floorf(xf), y0f = floorf(yf);
                const float ax = xf - x0f, ay = yf - y0f;
                int xa = (int)x0f, ya = (int)y0f;
                float wxa = 1.0f - ax, wxb = ax;
                float wya = 1.0f - ay, wyb = ay;
                // keep both taps of each axis on in-range pixels; an
                // out-of-range tap gets weight zero (zero padding)
                if (xa < 0) {
                    xa = 0; wxa = ax; wxb = 0.0f;
                } else if (xa >= p.W - 1) {
                    if (p.W >= 2) { xa = p.W - 2; wxb = 1.0f - ax; wxa = 0.0f; }
                    else { xa = 0; wxb = 0.0f; }
                }
                if (ya < 0) {
                    ya = 0; wya = ay; wyb = 0.0f;
                } else if (ya >= p.H - 1) {
                    if (p.H >= 2) { ya = p.H - 2; wyb = 1.0f - ay; wya = 0.0f; }
                    else { ya = 0; wyb = 0.0f; }
                }
                const uint32_t pix = ((cam_base + (uint32_t)n_p) * (uint32_t)p.H + (uint32_t)ya) *
                                         (uint32_t)p.W + (uint32_t)xa;
                const int pos = __builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                const int r = m * kRecCap + pos;
                wl[r] = make_float4((wxa * wya) * inv, (wxb * wya) * inv, (wxa * wyb) * inv,
                                    (wxb * wyb) * inv);
                ol[r] = pix * p.row_bytes;
            }
            const int cnt = __popcll(mask);
            if (lane == 0) cl[m] = cnt;
            maxcnt = cnt > maxcnt ? cnt : maxcnt;
        }
        wave_lds_sync();

        // ---- phase 2: gather-reduce over the compacted samples
        const int my_cnt = g_active ? cl[m_g] : 0;
        const float4 *wv = wl + m_lds * kRecCap;
        const uint32_t *ov = ol + m_lds * kRecCap;
        // kUnroll samples per iteration so that 4*kUnroll tap loads are in
        // flight per wavefront; lanes past their cell's count load nothing
        // (offset beyond the buffer) with weight zero.
        for (int k = 0; k < maxcnt; k += kUnroll) {
            float4 w[kUnroll];
            uint32_t base[kUnroll];
            bool act[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int kk = k + u;
                const int kr = kk < kRecCap ? kk : kRecCap - 1;
                act[u] = kk < my_cnt;
                const float4 wr = wv[kr];
                const uint32_t br = ov[kr];
                w[u] = act[u] ? wr : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                base[u] = br;
            }
#pragma unroll
            for (int v = 0; v < VPL; ++v) {
                const int vi = slot + L * v;
                if (VPL == 1 || vi < p.nvec) {
                    Raw<LW> t[kUnroll][4];
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        const uint32_t vo = act[u] ? base[u] + (uint32_t)vi * LW : kNoTap;
                        t[u][0] = load_vec<LW>(rsrc, vo, 0u);
                        t[u][1] = load_vec<LW>(rsrc, vo, p.step_x);
                        t[u][2] = load_vec<LW>(rsrc, vo, p.step_y);
                        t[u][3] = load_vec<LW>(rsrc, vo, p.step_x + p.step_y);
                    }
#pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
                        for (int e = 0; e < EPV; ++e) {
                            float s = acc[v][e];
                            s = fmaf(w[u].x, elem<DT, LW>(t[u][0], e), s);
                            s = fmaf(w[u].y, elem<DT, LW>(t[u][1], e), s);
                            s = fmaf(w[u].z, elem<DT, LW>(t[u][2], e), s);
                            s = fmaf(w[u].w, elem<DT, LW>(t[u][3], e), s);
                            acc[v][e] = s;
                        }
                    }
                }
            }
        }
        wave_lds_sync();
    }

    // ---- single write of out[b, c, i, j] (Alg. 2: write once)
    if (g_active) {
        const size_t q = (size_t)(q0 + m_g);
        float *ob = p.out + (size_t)b * p.C * p.XY + q;
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
            const int vi = slot + L * v;
            if (VPL == 1 || vi < p.nvec) {
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    const int c = vi * EPV + e;
                    ob[(size_t)c * p.XY] = acc[v][e];
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// host side: validation, geometry, dispatch
// ---------------------------------------------------------------------------
using KernelFn = void (*)(const Params);

template <int DT, int LW>
KernelFn pick_vpl(int vpl)
{
    switch (vpl) {
    case 1: return sample_vt_fwd<DT, LW, 1>;
    case 2: return sample_vt_fwd<DT, LW, 2>;
    default: return sample_vt_fwd<DT, LW, 4>;
    }
}

template <int DT>
KernelFn pick_lw(int lw, int vpl)
{
    switch (lw) {
    case 16: return pick_vpl<DT, 16>(vpl);
    case 8: return pick_vpl<DT, 8>(vpl);
    case 4: return pick_vpl<DT, 4>(vpl);
    default:
        if constexpr (DT == FLASHBEV_F32) return nullptr;
        else return pick_vpl<DT, 2>(vpl);
    }
}

KernelFn pick_kernel(int dtype, int lw, int vpl)
{
    switch (dtype) {
    case FLASHBEV_F32: return pick_lw<FLASHBEV_F32>(lw, vpl);
    case FLASHBEV_F16: return pick_lw<FLASHBEV_F16>(lw, vpl);
    default: return pick_lw<FLASHBEV_BF16>(lw, vpl);
    }
}

struct Plan {
    Params prm;
    int64_t workgroups;
    size_t lds;
    int lw, vpl;
    bool empty;
};

bool finite(float v) { return v == v && v - v == 0.0f; }

bool overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    if (!na || !nb) return false;
    uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + nb && b0 < a0 + na;
}

// All argument checks; `need_data` requires the device pointers.
int make_plan(const flashbev_features *f, const float *l2i, const flashbev_bev_grid_spec *s,
              const flashbev_z_bins *zb, const float *out, bool need_data, Plan *pl)
{
    if (!f || !s || !zb) return FLASHBEV_ERR_NULLPTR;
    if (f->dtype != FLASHBEV_F32 && f->dtype != FLASHBEV_F16 && f->dtype != FLASHBEV_BF16)
        return FLASHBEV_ERR_DTYPE;
    if (f->B < 0 || f->N < 0 || f->C < 1 || f->H < 1 || f->W < 1 || f->img_h < 1 ||
        f->img_w < 1 || s->X < 0 || s->Y < 0 || zb->Z < 0)
        return FLASHBEV_ERR_SHAPE;
    if (zb->Z > FLASHBEV_ZMAX || f->N > FLASHBEV_NMAX) return FLASHBEV_ERR_UNSUPPORTED;
    if (s->reduce != FLASHBEV_REDUCE_VALID_MEAN && s->reduce != FLASHBEV_REDUCE_SUM)
        return FLASHBEV_ERR_VALUE;
    if (!finite(s->x_min) || !finite(s->dx) || !finite(s->y_min) || !finite(s->dy) ||
        !finite(s->depth_eps))
        return FLASHBEV_ERR_VALUE;
    const int es = (f->dtype == FLASHBEV_F32) ? 4 : 2;
    const uint64_t row = (uint64_t)f->C * es;
    if (row > FLASHBEV_ROW_BYTES_MAX) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t feat_bytes = (uint64_t)f->B * f->N * f->H * f->W * row;
    if (feat_bytes > kFeatBytesMax) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t XY = (uint64_t)s->X * s->Y;
    if (XY > 0x7FFFFFFFull) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t out_elems = (uint64_t)f->B * f->C * XY;
    const bool empty = out_elems == 0;
    if (zb->Z > 0 && !zb->z) return FLASHBEV_ERR_NULLPTR;
    if (need_data && !empty) {
        if (!out) return FLASHBEV_ERR_NULLPTR;
        if (feat_bytes > 0 && !f->data) return FLASHBEV_ERR_NULLPTR;
        if (f->N > 0 && !l2i) return FLASHBEV_ERR_NULLPTR;
        if (((uintptr_t)f->data % es) || ((uintptr_t)l2i % 4) || ((uintptr_t)out % 4))
            return FLASHBEV_ERR_ALIGN;
        const size_t ob = out_elems * 4;
        if (overlaps(out, ob, f->data, feat_bytes) ||
            overlaps(out, ob, l2i, (size_t)f->B * f->N * 64))
            return FLASHBEV_ERR_ALIAS;
    }

    // vector width: the widest of 16/8/4/2 bytes dividing the row and the
    // base address
    int lw = 16;
    while (lw > es && ((row % lw) != 0 || (((uintptr_t)f->data) % lw) != 0)) lw >>= 1;
    const int nvec = (int)(row / lw);
    int vpl = 1;
    while (vpl < 4 && (nvec + vpl - 1) / vpl > kWave) vpl <<= 1;
    const int lpc = (nvec + vpl - 1) / vpl;
    if (lpc > kWave) return FLASHBEV_ERR_UNSUPPORTED;
    int cpw = kWave / lpc;
    if (cpw > kCpwMax) cpw = kCpwMax;

    Params &p = pl->prm;
    memset(&p, 0, sizeof(p));
    p.feat = f->data;
    p.l2i = l2i;
    p.out = const_cast<float *>(out);
    p.feat_bytes = (uint32_t)feat_bytes;
    p.B = f->B; p.N = f->N; p.H = f->H; p.W = f->W; p.C = f->C;
    p.X = s->X; p.Y = s->Y; p.Z = zb->Z;
    p.XY = (int32_t)XY;
    const int cells_per_wg = kWaves * cpw;
    p.tiles_per_b = (int32_t)((XY + cells_per_wg - 1) / cells_per_wg);
    p.img_w = (float)f->img_w;
    p.img_h = (float)f->img_h;
    p.sx = (float)f->W / (float)f->img_w;
    p.sy = (float)f->H / (float)f->img_h;
    p.x_min = s->x_min; p.dx = s->dx; p.y_min = s->y_min; p.dy = s->dy;
    p.depth_eps = s->depth_eps;
    p.reduce = s->reduce;
    p.row_bytes = (uint32_t)row;
    p.step_x = f->W >= 2 ? (uint32_t)row : 0u;
    p.step_y = f->H >= 2 ? (uint32_t)(row * f->W) : 0u;
    p.nvec = nvec;
    p.lpc = lpc;
    p.cpw = cpw;
    int zc = f->N > 0 ? kWave / f->N : 1;
    if (zc > zb->Z && zb->Z > 0) zc = zb->Z;
    p.zc = zc < 1 ? 1 : zc;
    for (int k = 0; k < zb->Z; ++k) p.z[k] = zb->z[k];

    pl->workgroups = empty ? 0 : (int64_t)f->B * p.tiles_per_b;
    if (pl->workgroups > 0x7FFFFFFFll) return FLASHBEV_ERR_UNSUPPORTED;
    pl->lds = lds_bytes_for(cpw);
    pl->lw = lw;
    pl->vpl = vpl;
    pl->empty = empty;
    return FLASHBEV_OK;
}

}  // namespace

extern "C" {

int flashbev_abi_version(void) { return FLASHBEV_ABI_VERSION; }

const char *flashbev_status_string(int status)
{
    switch (status) {
    case FLASHBEV_OK: return "ok";
    case FLASHBEV_ERR_NULLPTR: return "a required pointer is NULL";
    case FLASHBEV_ERR_SHAPE: return "invalid dimension";
    case FLASHBEV_ERR_DTYPE: return "unknown feature dtype";
    case FLASHBEV_ERR_ALIGN: return "device pointer not element-aligned";
    case FLASHBEV_ERR_UNSUPPORTED: return "beyond a documented limit";
    case FLASHBEV_ERR_ALIAS: return "output overlaps an input";
    case FLASHBEV_ERR_VALUE: return "non-finite grid spec or bad reduce mode";
    case FLASHBEV_ERR_HIP: return "HIP kernel launch failed";
    default: return "unknown status";
    }
}

int flashbev_launch_info(const flashbev_features *features, const flashbev_bev_grid_spec *spec,
                         const flashbev_z_bins *z_bins, int64_t *workgroups,
                         int32_t *threads_per_workgroup, int32_t *lds_bytes,
                         int32_t *cells_per_wave, int32_t *lanes_per_cell)
{
    Plan pl;
    int rc = make_plan(features, nullptr, spec, z_bins, nullptr, false, &pl);
    if (rc) return rc;
    if (workgroups) *workgroups = pl.workgroups;
    if (threads_per_workgroup) *threads_per_workgroup = kThreads;
    if (lds_bytes) *lds_bytes = (int32_t)pl.lds;
    if (cells_per_wave) *cells_per_wave = pl.prm.cpw;
    if (lanes_per_cell) *lanes_per_cell = pl.prm.lpc;
    return FLASHBEV_OK;
}

int flashbev_sample_vt(const flashbev_features *features, const float *lidar2img,
                       const flashbev_bev_grid_spec *spec, const flashbev_z_bins *z_bins,
                       float *out, void *stream)
{
    Plan pl;
    int rc = make_plan(features, lidar2img, spec, z_bins, out, true, &pl);
    if (rc) return rc;
    if (pl.empty) return FLASHBEV_OK;
    KernelFn fn = pick_kernel(features->dtype, pl.lw, pl.vpl);
    if (!fn) return FLASHBEV_ERR_UNSUPPORTED;
    void *args[] = {&pl.prm};
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(fn),
                                   dim3((unsigned)pl.workgroups), dim3(kThreads), args, pl.lds,
                                   reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? FLASHBEV_OK : FLASHBEV_ERR_HIP;
}

}  // extern "C"
