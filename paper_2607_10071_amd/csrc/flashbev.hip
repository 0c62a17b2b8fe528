// Fused Sampling-VT forward for gfx950 (FlashBEV paper, Sec. 3.3, Alg. 2,
// evaluating Eq. 1), behind the C ABI declared in include/flashbev.h.
//
// Execution design (MI355X-first; the paper's one-thread-per-(b,x,y,c)
// mapping is not used):
//   * A workgroup (2 or 4 wavefronts) owns a tile of `tile_cells`
//     consecutive BEV cells (row-major over (x, y)) of one batch element.
//     Each wavefront covers `rounds` groups of `cpw` cells.  Within a group, lanes span the
//     channels of a cell: a lane holds LW-byte vectors of the channel-last
//     feature row, so the four bilinear taps of a sample are coalesced row
//     loads across the lanes of a cell.
//   * Projection, masking and bilinear set-up run once per
//     (cell, height, camera), not once per channel (the paper recomputes
//     them per channel, Sec. 3.3.3).  One pass maps the 64 lanes to
//     (height, camera) pairs of one cell; a ballot yields the per-height
//     camera count den_z and a deterministic compaction of the valid
//     samples into a per-wavefront LDS list.
//   * The per-height valid mean is folded into the tap weights
//     (w / max(1, den_z)), so the gather is one flat weighted sum over the
//     cell's valid samples in float32 registers (Eq. 1 re-associated; only
//     the rounding changes).
//   * Results go through an LDS tile [C][tile_cells] and leave as 16-byte
//     stores that cover whole runs of each channel plane of out[B,C,X,Y].
//     Each XCD takes one contiguous band of tiles (workgroups are
//     dispatched to the 8 XCDs round-robin), which keeps the
//     partial cache lines at tile edges inside one L2.
//   * Tap loads are raw buffer loads with 32-bit offsets; every address is
//     inside the feature tensor by construction (an out-of-range tap gets
//     weight zero on an in-range pixel) and the buffer descriptor bounds
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

#include <mutex>

#include "flashbev.h"
#include "hip_common.h"

namespace {

constexpr int kWave = 64;
constexpr int kWavesMax = 4;                 // wavefronts per workgroup (2 or 4)
constexpr int kThreadsMax = kWave * kWavesMax;  // 256
constexpr int kCpwMax = 8;                // cells per wavefront group (upper bound)
constexpr int kCellsPerWave = 6;          // a wavefront covers at least this many cells per tile
constexpr int kRecCap = 64;               // valid samples per (cell, projection pass), at most
constexpr int kRecStride = kRecCap + 1;   // odd stride: cells' lists start in different banks
constexpr int kUnroll = 2;                // samples gathered per loop iteration
constexpr int kXcds = 8;                  // MI355X: 8 XCDs, workgroups dispatched round-robin
constexpr int kStripe = 16;               // consecutive tiles per XCD stripe
// Forward calls that gather at most this many bytes of feature rows
// (B X Y Z C elem) take contiguous bands of tiles per XCD, larger ones
// interleaved stripes.  Measured on MI355X (bands against stripes of 16):
// rep 23.9 -> 23.5 us, half_batch 77.6 -> 74.6, the paper's reference
// setting 35.1 -> 32.8, long_range 105.6 -> 103.1, z_sweep 213.7 -> 212.0
// (re-checked since: half_batch 70.5 -> 66.8, long_range 72.7 -> 71.7,
// z_sweep 182.3 -> 180.4, the reference setting 33.1 -> 31.1, rep equal);
// but with 8x the work (Z = 64, C = 1024 or a 1600 x 1600 grid at the
// reference setting) bands lose 4% to the stripes' better balance.
constexpr uint64_t kBandsWorkMax = 1ull << 30;
// Offset of a tap that is not loaded: feature tensors are smaller than
// 2 GiB and the tap steps are smaller than the tensor, so this offset plus
// any step stays past the buffer (no 32-bit wrap) and the load returns zero
// without touching memory.
constexpr uint32_t kNoTap = 0x80000000u;
constexpr uint64_t kFeatBytesMax = 0x7FFFFFFFull;
constexpr uint32_t kLdsBudget = 64u * 1024u;   // dynamic LDS per workgroup
constexpr uint64_t kOneRoundTilesMax = 262144;  // grids up to this many one-round tiles
constexpr uint32_t kLdsBudgetBwd = 80u * 1024u;  // tiled backward: two workgroups per CU
constexpr int kBwdTileWaves = 8;                 // tiled backward: wavefronts per workgroup
constexpr int kBwdThreadsMax = kWave * kBwdTileWaves;
constexpr int kBwdTiledCMax = 512;               // tiled backward: widest rows (channels)
// a term-list entry packs (wavefront << 14) | (record index << 2) | tap
static_assert(kCpwMax * kRecStride < (1 << 12), "record index must fit 12 bits");
static_assert(kBwdTileWaves <= (1 << 18), "wavefront index must fit the entry");

struct Params {
    const void *feat;
    const float *l2i;
    float *out;
    uint32_t feat_bytes;   // buffer size for the descriptor
    int32_t B, N, H, W, C, X, Y, Z;
    int32_t XY;
    int32_t tiles_per_b;   // tiles per batch element
    int32_t tile_cells;    // cells per tile = waves * rounds * cpw
    int32_t rounds;        // cell groups per wavefront per tile
    float img_w, img_h;    // image size as float
    float sx, sy;          // W / img_w, H / img_h (float32, computed once)
    float x_min, dx, y_min, dy, depth_eps;
    int32_t reduce;        // 0 valid mean, 1 sum
    int32_t bands;         // 1: one contiguous band of tiles per XCD, 0: interleaved stripes
    int32_t tail_prio;     // 1: all workgroups resident at once; waves take issue priority
                           // from their groups' longest sample list (per-cell passes)
    uint32_t row_bytes;    // C * element size
    uint32_t step_x;       // byte step to the right-hand tap (0 if W == 1)
    uint32_t step_y;       // byte step to the lower tap (0 if H == 1)
    int32_t nvec;          // LW-byte vectors per feature row
    int32_t lpc;           // lanes per cell
    int32_t cpw;           // cells per wavefront group
    float rcp_n, rcp_lpc;  // float32 1 / max(N, 1) and 1 / lpc
    int32_t zc;            // heights per per-cell projection pass
    int32_t otile_ld;      // row pitch (floats) of the LDS output tile, odd
    int32_t rec_stride;    // records per cell list: one pass's samples, rounded up, odd
    double rcp_y;          // 1 / Y (float64), for the cell index split q = i Y + j
    double rcp_tiles;      // 1 / tiles_per_b (float64)
    int32_t store_rows;    // channel rows a full tile's store sweep covers: threads / tile_cells
    float rcp_tile;        // float32 1 / tile_cells
    uint32_t cam_bytes;    // bytes of one camera's feature map, H W C s
    uint32_t wrow_bytes;   // bytes of one feature-map row, W C s
    int32_t small24;       // 1: H, W C s and W below 2^24 (tap offsets in 24-bit multiplies)
    int32_t cull;          // packed phase: 1 to run the culling test (0: finite heights missing)
    float zlo, zhi, zabs;  // lowest and highest height, max(|zlo|, |zhi|)
    // LDS layout (byte offsets)
    uint32_t lds_z, lds_w, lds_off, lds_otile, lds_cl;
    float z[FLASHBEV_ZMAX];
};

// a / d for 0 <= a < 2^31 and 1 <= d < 2^31, with rcp = float64(1 / d): the
// float64 product is within one of the quotient, and one correction step
// each way makes it exact (in place of a 32-bit integer division sequence)
__device__ __forceinline__ int div_wide(int a, int d, double rcp)
{
    int q = (int)((double)a * rcp);
    // the remainder lies in [-d, 2d); unsigned arithmetic wraps where the
    // one-too-large product q d would pass 2^31
    const int r = (int)((uint32_t)a - (uint32_t)q * (uint32_t)d);
    q += (r >= d) ? 1 : 0;
    q -= (r < 0) ? 1 : 0;
    return q;
}

// the k lowest bits set (k in 0..64)
__device__ __forceinline__ uint64_t lowmask64(int k)
{
    return k >= 64 ? ~0ull : ((1ull << k) - 1ull);
}

// Camera culling of one BEV column (the mask M_n of Sec. 3.1 decided for
// every height at once).  Returns false only if every height z in
// [zlo, zhi] certainly fails the mask, whatever the float32 rounding of the
// projection recipe: along the column the homogeneous coordinates
// (u', v', d) are linear in z, so each failure below holds at every height
// once it holds at both ends with a margin.
//   depth:   d <= depth_eps;
//   left:    u' < 0 (then u = u'/d < 0; the magnitude guard keeps the
//            quotient away from -0, which the mask would accept);
//   right:   u' - img_w d > 0 (then u >= img_w where d > 0);
//   top and bottom: the same with v' and img_h.
// The margin, 2^-14 of the terms' magnitudes (|m0 x| + |m1 y| + |m2| zabs
// + |m3| per row, zabs = max(|zlo|, |zhi|)), exceeds the rounding of the
// recipe and of this test (a few 2^-24 of the same magnitudes) by far.  A
// non-finite value fails every comparison, so such a column is kept.
__device__ __forceinline__ bool column_may_project(const float (&mr)[12], float x, float y,
                                                   float zlo, float zhi, float zabs,
                                                   float img_w, float img_h, float eps)
{
    constexpr float k = 6.103515625e-05f;      // 2^-14
    constexpr float tiny = 7.888609052e-31f;   // 2^-100
    const float bu = mr[0] * x + mr[1] * y + mr[3];
    const float bv = mr[4] * x + mr[5] * y + mr[7];
    const float bd = mr[8] * x + mr[9] * y + mr[11];
    const float Mu = fabsf(mr[0] * x) + fabsf(mr[1] * y) + fabsf(mr[2]) * zabs + fabsf(mr[3]);
    const float Mv = fabsf(mr[4] * x) + fabsf(mr[5] * y) + fabsf(mr[6]) * zabs + fabsf(mr[7]);
    const float Md = fabsf(mr[8] * x) + fabsf(mr[9] * y) + fabsf(mr[10]) * zabs + fabsf(mr[11]);
    const float u0 = bu + mr[2] * zlo, u1 = bu + mr[2] * zhi;
    const float v0 = bv + mr[6] * zlo, v1 = bv + mr[6] * zhi;
    const float d0 = bd + mr[10] * zlo, d1 = bd + mr[10] * zhi;
    const float td = eps - k * Md;
    const bool behind = (d0 < td) & (d1 < td);
    const float tu = k * Mu, tv = k * Mv;
    const bool left = (u0 < -tu) & (u1 < -tu) & (Mu > tiny * Md);
    const bool top = (v0 < -tv) & (v1 < -tv) & (Mv > tiny * Md);
    const float tr = k * (Mu + img_w * Md), tb = k * (Mv + img_h * Md);
    const bool right = (u0 - img_w * d0 > tr) & (u1 - img_w * d1 > tr);
    const bool bottom = (v0 - img_h * d0 > tb) & (v1 - img_h * d1 > tb);
    return !(behind | left | top | right | bottom);
}

__device__ __forceinline__ float bcast(float v, int lane)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// LDS layout of one workgroup: camera matrices [N][12], heights [Z], sample
// records [waves][cpw][rs] (weights as float4, offsets as u32), and the
// output tile [C][otile_ld].  The record stride and the tile pitch are odd so
// that different cells and channels fall into different LDS banks.
struct LdsLayout {
    uint32_t z, w, off, otile, total;
};

__host__ __device__ inline uint32_t align16(uint32_t v) { return (v + 15u) & ~15u; }

__host__ __device__ inline LdsLayout lds_layout(int N, int Z, int waves, int cpw, int C,
                                                int otile_ld, int rs = kRecStride)
{
    LdsLayout l;
    uint32_t o = align16((uint32_t)N * 12u * 4u);
    l.z = o;
    o = align16(o + (uint32_t)Z * 4u);
    l.w = o;
    o = align16(o + (uint32_t)waves * cpw * rs * 16u);
    l.off = o;
    o = align16(o + (uint32_t)waves * cpw * rs * 4u);
    l.otile = o;
    o = align16(o + (uint32_t)C * otile_ld * 4u);
    l.total = o;
    return l;
}

// ---------------------------------------------------------------------------
// the fused kernel
// ---------------------------------------------------------------------------
// Wavefronts per SIMD the compiler must leave room for (VGPR budget).  The
// representative float32 workload (16-byte lanes, one vector per lane) fits
// 72 VGPRs without spilling, which keeps all of its workgroups resident at
// once (measured on MI355X: 23.7 -> 22.8 us); the other instantiations keep
// the compiler's choice.
// Phase clock of the forward, compiled in only with FLASHBEV_PHASE_CLOCK
// (the instrumented library libflashbev_phases.so; the operator's library
// has none of it).  Lane 0 of each wavefront keeps the real-time counter
// (100 MHz) at its start, after staging, after the final barrier and at its
// end, and the time it spent in each phase, and writes them to
// phase_log[(workgroup * waves + wave) * kPhaseSlots + slot] at its end.
#ifdef FLASHBEV_PHASE_CLOCK
__device__ unsigned long long *phase_log;
constexpr int kPhaseSlots = 16;
enum PhaseSlot {
    kPhStart = 0, kPhStaged = 1, kPhProject = 2, kPhSetup = 3, kPhPad = 4, kPhGather = 5,
    kPhStash = 6, kPhBarrier = 7, kPhEnd = 8, kPhRounds = 9, kPhPasses = 10, kPhHwId = 11,
    kPhSamples = 12
};
// slot 11: the wavefront's HW_ID register (SIMD, CU, shader array and engine)
// in the low 32 bits and XCC_ID (its XCD) in the high 32; slot 12: the valid
// samples of its groups
#define PH_DECL                                                              \
    unsigned long long ph_t = __builtin_amdgcn_s_memrealtime();              \
    unsigned long long ph_s[kPhaseSlots] = {};                               \
    ph_s[kPhStart] = ph_t;                                                   \
    ph_s[kPhHwId] = (unsigned)__builtin_amdgcn_s_getreg((31 << 11) | 4) |    \
                    ((unsigned long long)(unsigned)__builtin_amdgcn_s_getreg((31 << 11) | 20) << 32)
#define PH_AT(slot)                                                          \
    do {                                                                     \
        ph_t = __builtin_amdgcn_s_memrealtime();                             \
        ph_s[slot] = ph_t;                                                   \
    } while (0)
#define PH_ADD(slot)                                                         \
    do {                                                                     \
        const unsigned long long ph_n = __builtin_amdgcn_s_memrealtime();    \
        ph_s[slot] += ph_n - ph_t;                                           \
        ph_t = ph_n;                                                         \
    } while (0)
#define PH_COUNT(slot) (ph_s[slot] += 1)
#define PH_ADDV(slot, v) (ph_s[slot] += (unsigned long long)(v))
#define PH_WRITE(lane)                                                       \
    do {                                                                     \
        if (phase_log && (lane) == 0) {                                      \
            unsigned long long *ph_o = phase_log +                           \
                ((size_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave) * kPhaseSlots; \
            for (int k = 0; k < kPhaseSlots; ++k) ph_o[k] = ph_s[k];         \
        }                                                                    \
    } while (0)
#else
#define PH_DECL
#define PH_AT(slot) ((void)0)
#define PH_ADD(slot) ((void)0)
#define PH_COUNT(slot) ((void)0)
#define PH_ADDV(slot, v) ((void)0)
#define PH_WRITE(lane) ((void)0)
#endif

template <int DT, int LW, int VPL, bool CULL>
struct FwdWaves {
    static constexpr int value = (!CULL && DT == FLASHBEV_F32 && LW == 16 && VPL == 1) ? 7 : 1;
};

// CULL selects the projection phase (chosen on the host, make_plan):
//   false: per-cell passes.  The 64 lanes hold the (height, camera) pairs of
//          one cell; a dense set-up pass then serves the group's valid
//          samples.  Suits groups of few cells whose heights and cameras
//          fill a pass.
//   true:  a culling pass per group drops the cameras no cell of the group
//          can see (column_may_project), then passes pack several cells'
//          (height, visible camera) pairs and set up each valid sample
//          where it is found.  Suits groups of many cells, or heights and
//          cameras that would need several passes per cell.
template <int DT, int LW, int VPL, bool CULL>
__global__ void __launch_bounds__(kThreadsMax)
__attribute__((amdgpu_waves_per_eu(FwdWaves<DT, LW, VPL, CULL>::value, 8)))
sample_vt_fwd(const Params p)
{
    constexpr int ES = ElemSize<DT>::value;
    constexpr int EPV = LW / ES;  // elements per vector
    extern __shared__ __align__(16) unsigned char smem[];
    float *s_mat = reinterpret_cast<float *>(smem);
    float *s_z = reinterpret_cast<float *>(smem + p.lds_z);
    float4 *s_w = reinterpret_cast<float4 *>(smem + p.lds_w);
    uint32_t *s_off = reinterpret_cast<uint32_t *>(smem + p.lds_off);
    float *s_tile = reinterpret_cast<float *>(smem + p.lds_otile);

    PH_DECL;
    const int cpw = p.cpw;
    const int RS = p.rec_stride;
    const int tid = threadIdx.x;
    const int nthreads = blockDim.x;  // waves * 64
    // wavefront index as a scalar (uniform per wavefront), so that the
    // per-wavefront offsets below are scalar arithmetic
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int N = p.N;

    // XCD-aware tile order.  Workgroups go to the 8 XCDs round-robin.
    //  * Bands (p.bands, calls with little work): the k-th workgroup on XCD x
    //    takes tile x * per + k, so each XCD works through one contiguous
    //    band of the grid (per = workgroups / 8; the last few keep the
    //    dispatch order).  A band of rows is seen by about half of the ring's
    //    cameras, whose features then fit the XCD's L2.
    //  * Stripes (more work): tile (k / S) * 8S + x * S + k % S, stripes of
    //    S consecutive tiles interleaved over the grid, so that each XCD sees
    //    a like mix of heavy and light regions and the tail stays short.
    // Either way neighbouring tiles merge their partial output lines in one
    // L2.  The choice is made on the host (make_plan, forward_order).
    const int g = blockIdx.x;
    int tile = g;
    if (p.bands) {
        const int per = (int)gridDim.x / kXcds;
        if (g < per * kXcds) {
            const int xcd = g % kXcds, k = g / kXcds;
            tile = xcd * per + k;
        }
    } else {
        const int full = (int)(gridDim.x / (kXcds * kStripe)) * (kXcds * kStripe);
        if (g < full) {
            const int xcd = g % kXcds, k = g / kXcds;
            tile = (k / kStripe) * (kXcds * kStripe) + xcd * kStripe + k % kStripe;
        }
    }
    const int b = div_wide(tile, p.tiles_per_b, p.rcp_tiles);
    const int q_tile = (tile - b * p.tiles_per_b) * p.tile_cells;

    // stage camera matrices (rows 0..2) and heights; a thread's first
    // elements of both are loaded before either is stored, so the two loads
    // overlap
    {
        const int nm = N * 12;
        const bool hm = tid < nm, hz = tid < p.Z;
        const int n = tid / 12;
        const float mv = hm ? p.l2i[((size_t)b * N + n) * 16 + (tid - n * 12)] : 0.0f;
        const float zv = hz ? p.z[tid] : 0.0f;
        if (hm) s_mat[tid] = mv;
        if (hz) s_z[tid] = zv;
        for (int t = tid + nthreads; t < nm; t += nthreads) {
            const int n2 = t / 12, r = t - n2 * 12;
            s_mat[t] = p.l2i[((size_t)b * N + n2) * 16 + r];
        }
        for (int t = tid + nthreads; t < p.Z; t += nthreads) s_z[t] = p.z[t];
    }
    __syncthreads();
    PH_AT(kPhStaged);

    // culling role: cell zl of a group, camera n_p
    const int Nd = N > 0 ? N : 1;
    const int zl = div_small(lane, Nd, p.rcp_n);
    const int n_p = lane - zl * Nd;
    const uint64_t nmask = lowmask64(N);

    // gather role: cell m_g of the group, channel-vector slot `slot`
    const int L = p.lpc;
    const int m_g = div_small(lane, L, p.rcp_lpc);
    const int slot = lane - m_g * L;
    const bool in_group = m_g < cpw;
    const int m_lds = in_group ? m_g : 0;

    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p.feat), (short)0,
                                          (int)p.feat_bytes, 0x00020000);

    float4 *wl = s_w + (size_t)wave * cpw * RS;
    uint32_t *ol = s_off + (size_t)wave * cpw * RS;
    uint32_t *cl = reinterpret_cast<uint32_t *>(smem + p.lds_cl) + wave * kWave;  // visible cameras
    const int wcells = p.rounds * cpw;
    const int q_wave = q_tile + wave * wcells;

    // voxel centres of the wavefront's cells (Alg. 2: "compute voxel
    // center"), one cell per lane, broadcast with readlane below
    float xs = 0.0f, ys = 0.0f;
    if (lane < wcells && q_wave + lane < p.XY) {
        const int q = q_wave + lane;
        const int i = div_wide(q, p.Y, p.rcp_y);
        const int j = q - i * p.Y;
        xs = p.x_min + ((float)i + 0.5f) * p.dx;
        ys = p.y_min + ((float)j + 0.5f) * p.dy;
    }

    // phase 2 of one group: gather-reduce over the compacted samples of the
    // group's cells.  kUnroll samples per iteration keep 4*kUnroll tap
    // loads in flight per lane.
    auto gather = [&](float (&acc)[VPL][EPV], bool g_active, int maxpad) {
        if (g_active) {
            const float4 *wv = wl + m_lds * RS;
            const uint32_t *ov = ol + m_lds * RS;
            for (int k = 0; k < maxpad; k += kUnroll) {
                float4 w[kUnroll];
                uint32_t base[kUnroll];
                // the samples' offsets, then their weights, both read from
                // LDS before the tap loads are issued: the loads wait only
                // for the offsets, and the weights arrive while they are in
                // flight (the scheduling barrier keeps that order)
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) base[u] = ov[k + u];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) w[u] = wv[k + u];
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int v = 0; v < VPL; ++v) {
                    const int vi = slot + L * v;
                    if (VPL == 1 || vi < p.nvec) {
                        Raw<LW> t[kUnroll][4];
#pragma unroll
                        for (int u = 0; u < kUnroll; ++u) {
                            const uint32_t vo = base[u] + (uint32_t)vi * LW;
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
        }
        wave_lds_sync();
    };

    // records past a cell's count, up to the padded loop length, carry zero
    // weights and no tap
    auto pad = [&](int ncell, int cnt_lane, int maxpad) {
        for (int m = 0; m < ncell; ++m) {
            const int c = __builtin_amdgcn_readlane(cnt_lane, m);
            if (lane >= c && lane < maxpad) {
                wl[m * RS + lane] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                ol[m * RS + lane] = kNoTap;
            }
        }
        wave_lds_sync();
    };

    for (int r = 0; r < p.rounds; ++r) {
        PH_COUNT(kPhRounds);
        const int q_grp = q_wave + r * cpw;
        // cells of this group inside the grid (<= 0 past the end of the last tile)
        const int ncell = (p.XY - q_grp) < cpw ? (p.XY - q_grp) : cpw;
        const bool g_active = m_g < ncell;

        float acc[VPL][EPV];
#pragma unroll
        for (int v = 0; v < VPL; ++v)
#pragma unroll
            for (int e = 0; e < EPV; ++e) acc[v][e] = 0.0f;

        if constexpr (CULL) {
            // ---- camera culling for the group: lane (cell zl, camera n_p)
            // tests whether the camera can see the cell's column at any height;
            // cameras no cell of the group can see are left out of the
            // projection passes (their samples are all masked out anyway)
            uint64_t cmask = ncell > 0 ? nmask : 0ull;
            if (p.cull && ncell > 0) {
                bool vis = false;
                if (N > 0 && zl < ncell) {
                    const float4 *crow = reinterpret_cast<const float4 *>(s_mat) + n_p * 3;
                    const float4 ma = crow[0], mb = crow[1], mc = crow[2];
                    const float mr[12] = {ma.x, ma.y, ma.z, ma.w, mb.x, mb.y, mb.z, mb.w,
                                          mc.x, mc.y, mc.z, mc.w};
                    vis = column_may_project(mr, __shfl(xs, r * cpw + zl), __shfl(ys, r * cpw + zl),
                                             p.zlo, p.zhi, p.zabs, p.img_w, p.img_h, p.depth_eps);
                }
                const uint64_t vm = __ballot(vis);
                cmask = 0ull;
                for (int m = 0; m < ncell; ++m) cmask |= (vm >> (m * N)) & nmask;
            }
            const int Np = __popcll(cmask);
            PH_ADD(kPhProject);

            if (Np > 0) {
                // the visible cameras in ascending order
                if (lane < N && ((cmask >> lane) & 1ull))
                    cl[__popcll(cmask & lowmask64(lane))] = lane;
                wave_lds_sync();
                // pass layout: lane = (cell lm, height lz, visible camera lc),
                // camera fastest.  A pass holds zcp heights of cpp cells; when
                // all heights fit one pass, several cells share it.
                const int zcp = (kWave / Np) < p.Z ? (kWave / Np) : p.Z;
                const int P = zcp * Np;
                int cpp = 1;
                if (zcp == p.Z) {
                    cpp = kWave / P;
                    if (cpp > ncell) cpp = ncell;
                }
                const float rcp_p = __builtin_amdgcn_rcpf((float)P);
                const float rcp_np = __builtin_amdgcn_rcpf((float)Np);

                for (int z0 = 0; z0 < p.Z; z0 += zcp) {
                    // this lane's place in the pass, its camera's rows and map
                    // offset (formed per height chunk: nothing of it stays live
                    // through the gather)
                    const int lm = div_small(lane, P, rcp_p);
                    const int lr = lane - lm * P;
                    const int lz = div_small(lr, Np, rcp_np);
                    const int lc = lr - lz * Np;
                    const bool l_in = lm < cpp;
                    const int n = (int)cl[lc];
                    const float4 *prow = reinterpret_cast<const float4 *>(s_mat) + n * 3;
                    const uint32_t coff = ((uint32_t)b * (uint32_t)N + (uint32_t)n) * p.cam_bytes;
                    // lanes of this lane's (cell, height) group (den_z) and the
                    // lanes before its cell in the pass (compaction offset)
                    const uint64_t gmask = lowmask64(Np) << (lane - lc);
                    const uint64_t before_cell = lowmask64(lm * P);
                    int cnt_lane = 0, maxcnt = 0;  // lane m holds cell m's count
                    const int zi = z0 + lz;
                    const bool z_ok = l_in && zi < p.Z;
                    const float zv = z_ok ? s_z[zi] : 0.0f;
                    for (int m0 = 0; m0 < ncell; m0 += cpp) {
                        // ---- phase 1: project, mask, compact and set up every
                        // (cell, height, visible camera) sample of the pass
                        const float4 ma = prow[0], mb = prow[1], mc = prow[2];
                        const float mr[12] = {ma.x, ma.y, ma.z, ma.w, mb.x, mb.y, mb.z, mb.w,
                                              mc.x, mc.y, mc.z, mc.w};
                        const float t2u = mr[2] * zv, t2v = mr[6] * zv, t2d = mr[10] * zv;
                        const int m = m0 + lm;
                        const bool l_ok = z_ok && m < ncell;
                        const float x = __shfl(xs, r * cpw + m);
                        const float y = __shfl(ys, r * cpw + m);
                        // (u', v', d) = P[b,n] (x, y, z, 1), left to right, no contraction
                        const float up = ((mr[0] * x + mr[1] * y) + t2u) + mr[3];
                        const float vp = ((mr[4] * x + mr[5] * y) + t2v) + mr[7];
                        const float d = ((mr[8] * x + mr[9] * y) + t2d) + mr[11];
                        const float u = up / d;
                        const float v = vp / d;
                        // M_n: positive depth, inside the image (half-open box)
                        const bool ok = l_ok & (d > p.depth_eps) & (u >= 0.0f) & (u < p.img_w) &
                                        (v >= 0.0f) & (v < p.img_h);
                        const uint64_t mask = __ballot(ok);
                        if (ok) {
                            // den_z: the valid cameras of this (cell, height)
                            const int den = __popcll(mask & gmask);
                            const int pos = __builtin_amdgcn_mbcnt_hi(
                                                (uint32_t)(mask >> 32),
                                                __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u)) -
                                            __popcll(mask & before_cell);
                            // bilinear set-up: feature coordinates, tap weights
                            // with 1 / max(1, den_z) folded in, first tap's offset
                            const float inv = (p.reduce == 0) ? __builtin_amdgcn_rcpf((float)den) : 1.0f;
                            const float xf = u * p.sx - 0.5f;
                            const float yf = v * p.sy - 0.5f;
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
                            wya *= inv;
                            wyb *= inv;
                            // byte offset of the first tap: camera + row + column
                            // (24-bit multiplies where the host found the
                            // factors small enough; the offset is below 2^31)
                            const uint32_t rofs = p.small24
                                ? __umul24((uint32_t)ya, p.wrow_bytes) + __umul24((uint32_t)xa, p.row_bytes)
                                : (uint32_t)ya * p.wrow_bytes + (uint32_t)xa * p.row_bytes;
                            const int slotk = m * RS + pos;
                            wl[slotk] = make_float4(wxa * wya, wxb * wya, wxa * wyb, wxb * wyb);
                            ol[slotk] = coff + rofs;
                        }
                        // the pass's valid samples per cell
                        for (int mm = 0; mm < cpp && m0 + mm < ncell; ++mm) {
                            const int c = __popcll(mask & (lowmask64(P) << (mm * P)));
                            PH_ADDV(kPhSamples, c);
                            cnt_lane = lane == m0 + mm ? c : cnt_lane;
                            maxcnt = c > maxcnt ? c : maxcnt;
                        }
                    }
                    PH_ADD(kPhProject);
                    PH_COUNT(kPhPasses);
                    const int maxpad = (maxcnt + kUnroll - 1) / kUnroll * kUnroll;
                    pad(ncell, cnt_lane, maxpad);
                    PH_ADD(kPhPad);
                    gather(acc, g_active, maxpad);
                    PH_ADD(kPhGather);
                }
            }
        } else {
            // projection role: height zl of a pass, camera n_p; the lane's
            // camera rows stay in LDS (read once per pass)
            const bool p_role = (N > 0) && (zl < p.zc);
            const int zshift = p_role ? zl * N : 0;
            const float4 *mrow = reinterpret_cast<const float4 *>(s_mat) + (p_role ? n_p * 3 : 0);
            const uint32_t cam_off = ((uint32_t)b * (uint32_t)N + (uint32_t)(p_role ? n_p : 0)) * p.cam_bytes;
            for (int z0 = 0; z0 < p.Z; z0 += p.zc) {
                // ---- phase 1a: project every (height, camera) pair of each
                // cell, apply the mask M_n, and compact the valid samples as
                // (u, v, camera, den_z) in the cell's record list
                const int zi = z0 + zl;
                const bool l_ok = p_role && zi < p.Z;
                const float zv = l_ok ? s_z[zi] : 0.0f;
                const float4 ma = mrow[0], mb = mrow[1], mc = mrow[2];
                const float mr[12] = {ma.x, ma.y, ma.z, ma.w, mb.x, mb.y, mb.z, mb.w,
                                      mc.x, mc.y, mc.z, mc.w};
                const float t2u = mr[2] * zv, t2v = mr[6] * zv, t2d = mr[10] * zv;
                int total = 0, maxcnt = 0;
                int cnt_lane = 0, pre_lane = 0;  // lane m holds cell m's count and prefix
                for (int m = 0; m < ncell; ++m) {
                    const float x = bcast(xs, r * cpw + m);
                    const float y = bcast(ys, r * cpw + m);
                    // (u', v', d) = P[b,n] (x, y, z, 1), left to right, no contraction
                    const float up = ((mr[0] * x + mr[1] * y) + t2u) + mr[3];
                    const float vp = ((mr[4] * x + mr[5] * y) + t2v) + mr[7];
                    const float d = ((mr[8] * x + mr[9] * y) + t2d) + mr[11];
                    const float u = up / d;
                    const float v = vp / d;
                    // M_n: positive depth, inside the image (half-open box)
                    const bool ok = l_ok && (d > p.depth_eps) && (u >= 0.0f) && (u < p.img_w) &&
                                    (v >= 0.0f) && (v < p.img_h);
                    const uint64_t mask = __ballot(ok);
                    if (ok) {
                        const int den = __popcll((mask >> zshift) & nmask);
                        const int pos = __builtin_amdgcn_mbcnt_hi(
                            (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                        wl[m * RS + pos] = make_float4(u, v, __builtin_bit_cast(float, cam_off),
                                                       __builtin_bit_cast(float, den));
                    }
                    const int cnt = __popcll(mask);
                    cnt_lane = lane == m ? cnt : cnt_lane;
                    pre_lane = lane == m ? total : pre_lane;
                    total += cnt;
                    maxcnt = cnt > maxcnt ? cnt : maxcnt;
                }
                const int maxpad = (maxcnt + kUnroll - 1) / kUnroll * kUnroll;
                wave_lds_sync();
                if (p.tail_prio) {
                    // When every workgroup is resident from the start, the
                    // call ends with its heaviest wavefronts: the longest
                    // sample list sets a group's gather iterations, and the
                    // lists of cells that several cameras see at most heights
                    // (overlap zones, far range) are up to twice the median.
                    // Such wavefronts take a higher issue priority, the work
                    // left to them estimated as this group's longest list
                    // times the rounds left, so they are not left to finish
                    // alone at the end (measured on MI355X: rep 22.25 ->
                    // 21.4 us, Z = 4 15.8 -> 15.2, Z = 6 19.0 -> 17.7;
                    // thresholds between 1.05 and 2 samples per height give
                    // the same).  With several generations of workgroups the
                    // hardware balances the finish by itself and the
                    // priorities cost 1-2% (the paper's reference setting),
                    // so they stay off there.
                    const int zh = (p.Z - z0) < p.zc ? (p.Z - z0) : p.zc;
                    const int t20 = maxcnt * 20 * (p.rounds - r);
                    if (t20 >= 38 * zh) __builtin_amdgcn_s_setprio(3);
                    else if (t20 >= 32 * zh) __builtin_amdgcn_s_setprio(2);
                    else if (t20 >= 26 * zh) __builtin_amdgcn_s_setprio(1);
                    else __builtin_amdgcn_s_setprio(0);
                }
                PH_ADDV(kPhSamples, total);
                PH_ADD(kPhProject);
                PH_COUNT(kPhPasses);

                // ---- phase 1b: for all valid samples of the group at once,
                // bilinear set-up: feature coordinates, tap weights with
                // 1 / max(1, den_z) folded in, byte offset of the first tap
                for (int base = 0; base < total; base += kWave) {
                    const int idx = base + lane;
                    int m = 0, pm = 0;  // cell of sample idx and that cell's first index
                    for (int mm = 1; mm < ncell; ++mm) {
                        const int pf = __builtin_amdgcn_readlane(pre_lane, mm);
                        const bool ge = idx >= pf;
                        m = ge ? mm : m;
                        pm = ge ? pf : pm;
                    }
                    if (idx < total) {
                        const int slotk = m * RS + (idx - pm);
                        const float4 pr = wl[slotk];
                        const float u = pr.x, v = pr.y;
                        const uint32_t coff = __builtin_bit_cast(uint32_t, pr.z);
                        const int den = __builtin_bit_cast(int, pr.w);
                        const float inv = (p.reduce == 0) ? __builtin_amdgcn_rcpf((float)den) : 1.0f;
                        const float xf = u * p.sx - 0.5f;
                        const float yf = v * p.sy - 0.5f;
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
                        wya *= inv;
                        wyb *= inv;
                        // byte offset of the first tap: camera + row + column
                        // (24-bit multiplies where the host found the factors
                        // small enough; the offset itself is below 2^31)
                        const uint32_t rofs = p.small24
                            ? __umul24((uint32_t)ya, p.wrow_bytes) +
                                  __umul24((uint32_t)xa, p.row_bytes)
                            : (uint32_t)ya * p.wrow_bytes + (uint32_t)xa * p.row_bytes;
                        wl[slotk] = make_float4(wxa * wya, wxb * wya, wxa * wyb, wxb * wyb);
                        ol[slotk] = coff + rofs;
                    }
                }
                PH_ADD(kPhSetup);
                pad(ncell, cnt_lane, maxpad);
                PH_ADD(kPhPad);
                gather(acc, g_active, maxpad);
                PH_ADD(kPhGather);
            }
        }

        // stash this group's results in the output tile
        if (g_active) {
            const int col = wave * wcells + r * cpw + m_g;
#pragma unroll
            for (int v = 0; v < VPL; ++v) {
                const int vi = slot + L * v;
                if (VPL == 1 || vi < p.nvec) {
#pragma unroll
                    for (int e = 0; e < EPV; ++e)
                        s_tile[(vi * EPV + e) * p.otile_ld + col] = acc[v][e];
                }
            }
        }
        PH_ADD(kPhStash);
    }
    __syncthreads();
    PH_AT(kPhBarrier);

    // ---- single write of out[b, c, tile cells] (Alg. 2: write once):
    // consecutive threads write consecutive cells of one channel plane
    const int T = p.tile_cells;
    const int rem = p.XY - q_tile;
    const int nq = rem < T ? rem : T;
    float *ob = p.out + (size_t)b * p.C * p.XY + q_tile;
    // channel rows written per sweep (>= 1); a full tile takes the host's
    // figures, the grid's last partial tile computes its own
    const bool full = nq == T;
    const int rows = full ? p.store_rows : nthreads / nq;
    const int c0 = div_small(tid, nq, full ? p.rcp_tile : 1.0f / (float)nq);
    const int k = tid - c0 * nq;
    if (c0 < rows) {
        for (int c = c0; c < p.C; c += rows) ob[(size_t)c * p.XY + k] = s_tile[c * p.otile_ld + k];
    }
    PH_AT(kPhEnd);
    PH_WRITE(lane);
}

// ---------------------------------------------------------------------------
// backward: gradient with respect to the feature maps
// ---------------------------------------------------------------------------
// Eq. 1 is linear in the features; its gradient is the transpose of the
// forward's map: every valid sample scatters w_t / max(1, den_z) times the
// output gradient of its cell onto the C channels of each of its four taps.
// The kernel keeps the forward's projection pass and set-up pass; in place
// of the gather it adds the terms into a float32 channel-last gradient
// (zero-filled by a separate kernel first).  Lane `slot` of a cell owns
// channels slot, slot + L, slot + 2L, ..., so each add covers a contiguous
// run of a pixel row.
//
// Float atomics are the cost: MI355X retires about 2e11 float atomic adds
// per second, in LDS as in global memory, whatever the address spread, while
// integer LDS atomics run some 28 times faster.  In the tiled mode a
// workgroup owns a 2-D tile of cells, whose samples share most of their taps,
// and gives each distinct pixel of the tile an LDS row (a lock-free LDS hash
// table with integer atomics maps pixels to rows).  After each height pass it
// sorts the pass's (sample, tap) terms by row (integer counts, a prefix sum,
// a fill), and one wavefront per row sums its terms into the row with plain
// FMAs.  At the end each row goes to the gradient with one global atomic per
// channel.  Taps that find the table full go straight to global atomics.  The
// direct mode (no table) serves shapes whose rows (more than 512 channels) or
// pixel ids do not fit.
//
// Occupancy decides the tiled mode's speed (measured on MI355X: one 4-wave
// workgroup per CU runs at half the speed of two).  So a workgroup has 8
// wavefronts and 80 KiB of LDS (two per CU, 16 wavefronts), and a height
// pass covers half the heights a wavefront could project at once.  That
// keeps the per-pass records and term list small and leaves room for rows.
// The rows then need only hold the pixels of about one pass: when the rows in
// use plus those the last pass claimed exceed the tile's rows, the tile adds
// its rows to the gradient and starts again with an empty table.
constexpr uint32_t kSlotNone = 0xFFFFu;   // tap not in the tile's table
constexpr int kKeyBits = 20;              // pixel ids (plus one) per batch element < 2^20
constexpr uint32_t kKeyMask = (1u << kKeyBits) - 1u;
constexpr int kSlotMax = (1 << (32 - kKeyBits)) - 1;  // 4095 rows per tile

struct BwdParams {
    const float *l2i;
    const float *gout;       // [B, C, X, Y]
    float *gfeat;            // [B, N, H, W, C]
    int32_t B, N, H, W, C, X, Y, Z;
    int32_t XY;
    int32_t tiles_per_b;
    int32_t tile_cells;      // cells per tile = waves * rounds * cpw
    int32_t rounds;
    float img_w, img_h;
    float sx, sy;
    float x_min, dx, y_min, dy, depth_eps;
    int32_t reduce;
    uint32_t step_x;         // element step to the right-hand tap (0 if W == 1)
    uint32_t step_y;         // element step to the lower tap (0 if H == 1)
    int32_t lpc;             // lanes per cell
    int32_t cpw;             // cells per wavefront group
    float rcp_n, rcp_lpc;
    int32_t zc;
    int32_t gtile_ld;        // row pitch (floats) of the LDS output-gradient tile, odd
    int32_t rec_stride;      // records per cell list: one pass's samples, odd
    uint32_t lds_z, lds_w, lds_off, lds_gtile;
    // tiled mode
    int32_t tx, ty;          // tile rows (along x) and columns (along y)
    int32_t tiles_y;         // tiles per tile row
    float rcp_ty, rcp_c;
    int32_t cap;             // LDS rows (distinct pixels) per tile
    uint32_t tbl_mask;       // hash table entries - 1 (power of two >= 2 cap)
    uint32_t lds_slot, lds_tbl, lds_spix, lds_acc, lds_cnt;
    uint32_t lds_rcnt, lds_rbase, lds_rfill, lds_list;
    float z[FLASHBEV_ZMAX];
};

// Projection of one cell for one height pass (Alg. 2: compute the voxel
// centre, project into camera n, check validity): lanes hold (height,
// camera) pairs; valid samples are compacted into rec[] as (u, v, camera,
// den_z).  Returns the number of valid samples.
__device__ __forceinline__ int bwd_project_cell(const BwdParams &p, const float (&mr)[12], float t2u,
                                                float t2v, float t2d, float x, float y, bool l_ok,
                                                int zshift, uint64_t nmask, int n_p, float4 *rec)
{
    const float up = ((mr[0] * x + mr[1] * y) + t2u) + mr[3];
    const float vp = ((mr[4] * x + mr[5] * y) + t2v) + mr[7];
    const float d = ((mr[8] * x + mr[9] * y) + t2d) + mr[11];
    const float u = up / d;
    const float v = vp / d;
    const bool ok = l_ok && (d > p.depth_eps) && (u >= 0.0f) && (u < p.img_w) && (v >= 0.0f) &&
                    (v < p.img_h);
    const uint64_t mask = __ballot(ok);
    if (ok) {
        const int den = __popcll((mask >> zshift) & nmask);
        const int pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                  __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
        rec[pos] = make_float4(u, v, __builtin_bit_cast(float, n_p), __builtin_bit_cast(float, den));
    }
    return __popcll(mask);
}

// Bilinear set-up of one valid sample (u, v): first tap (xa, ya) and the
// four weights with 1 / max(1, den_z) folded in; out-of-range taps are moved
// onto in-range pixels with weight zero (value selects only).
__device__ __forceinline__ float4 bwd_setup(const BwdParams &p, float u, float v, int den, int &xa,
                                            int &ya)
{
    const float inv = (p.reduce == 0) ? __builtin_amdgcn_rcpf((float)den) : 1.0f;
    const float xf = u * p.sx - 0.5f;
    const float yf = v * p.sy - 0.5f;
    const float x0f = floorf(xf), y0f = floorf(yf);
    const float ax = xf - x0f, ay = yf - y0f;
    const int xi = (int)x0f, yi = (int)y0f;
    const bool xl = xi < 0, xh = !xl && xi >= p.W - 1, xw = p.W >= 2;
    const bool yl = yi < 0, yh = !yl && yi >= p.H - 1, yw = p.H >= 2;
    xa = xl ? 0 : (xh ? (xw ? p.W - 2 : 0) : xi);
    ya = yl ? 0 : (yh ? (yw ? p.H - 2 : 0) : yi);
    const float wxa = xl ? ax : ((xh && xw) ? 0.0f : 1.0f - ax);
    const float wxb = xl ? 0.0f : (xh ? (xw ? 1.0f - ax : 0.0f) : ax);
    const float wya = (yl ? ay : ((yh && yw) ? 0.0f : 1.0f - ay)) * inv;
    const float wyb = (yl ? 0.0f : (yh ? (yw ? 1.0f - ay : 0.0f) : ay)) * inv;
    return make_float4(wxa * wya, wxb * wya, wxa * wyb, wxb * wyb);
}

// Table entry of pixel q of the tile (q < 2^20 - 1): find it in the open-
// addressing table or insert it.  Entries pack (q + 1) | row << 20, with row
// kRowUnset until the pass's row assignment gives the pixel an LDS row; 0
// is empty.  The probe sequence is cut after kProbeMax entries, so a crowded
// table costs little: the call then returns kSlotNone and the caller reads
// or adds that tap in global memory instead.
constexpr uint32_t kRowUnset = (1u << (32 - kKeyBits)) - 1u;
constexpr uint32_t kProbeMax = 32;

__device__ __forceinline__ uint32_t tile_insert(uint32_t q, uint32_t *tbl, uint32_t mask)
{
    const uint32_t key = q + 1u;
    uint32_t h = (key * 0x9E3779B1u) >> 8;
    for (uint32_t probe = 0; probe < kProbeMax; ++probe) {
        h &= mask;
        uint32_t e = tbl[h];
        if (e == 0u) {
            e = atomicCAS(&tbl[h], 0u, key | (kRowUnset << kKeyBits));
            if (e == 0u) return h;
        }
        if ((e & kKeyMask) == key) return h;
        ++h;
    }
    return kSlotNone;
}

// LDS row of table entry h (kSlotNone when h is kSlotNone or the pixel got
// no row because the tile's rows ran out).
__device__ __forceinline__ uint32_t tile_row_of(const uint32_t *tbl, uint32_t h)
{
    if (h == kSlotNone) return kSlotNone;
    const uint32_t r = tbl[h] >> kKeyBits;
    return r == kRowUnset ? kSlotNone : r;
}

template <int KPL, bool TILED, bool WIDE>
__global__ void __launch_bounds__(kBwdThreadsMax)
sample_vt_bwd(const BwdParams p)
{
    extern __shared__ __align__(16) unsigned char smem[];
    float *s_mat = reinterpret_cast<float *>(smem);
    float *s_z = reinterpret_cast<float *>(smem + p.lds_z);
    float4 *s_w = reinterpret_cast<float4 *>(smem + p.lds_w);
    uint32_t *s_off = reinterpret_cast<uint32_t *>(smem + p.lds_off);
    float *s_g = reinterpret_cast<float *>(smem + p.lds_gtile);
    uint2 *s_slot = reinterpret_cast<uint2 *>(smem + p.lds_slot);
    uint32_t *s_tbl = reinterpret_cast<uint32_t *>(smem + p.lds_tbl);
    uint32_t *s_spix = reinterpret_cast<uint32_t *>(smem + p.lds_spix);
    float *s_acc = reinterpret_cast<float *>(smem + p.lds_acc);
    uint32_t *s_cnt = reinterpret_cast<uint32_t *>(smem + p.lds_cnt);  // [0] rows, [1] overflow
    uint32_t *s_rcnt = reinterpret_cast<uint32_t *>(smem + p.lds_rcnt);
    uint32_t *s_rbase = reinterpret_cast<uint32_t *>(smem + p.lds_rbase);
    uint32_t *s_rfill = reinterpret_cast<uint32_t *>(smem + p.lds_rfill);
    uint32_t *s_list = reinterpret_cast<uint32_t *>(smem + p.lds_list);

    const int cpw = p.cpw;
    const int tid = threadIdx.x;
    const int nthreads = blockDim.x;
    const int wave = tid / kWave;
    const int lane = tid % kWave;
    const int N = p.N;
    const int C = p.C;
    const int T = p.tile_cells;
    const int RS = p.rec_stride;
    const float rcp_rs = 1.0f / (float)RS;  // record index -> cell without an integer divide

    // XCD-aware tile order: the k-th workgroup on XCD x takes tile
    // (k / S) * 8S + x * S + k % S, stripes of S consecutive tiles that
    // interleave over the grid (a like mix of heavy and light tiles per XCD;
    // measured on MI355X, the forward's contiguous bands are 2-4% slower
    // here, the scatter's atomics being resolved past the L2 anyway).  A last
    // partial block of 8S tiles keeps the dispatch order.
    const int g = blockIdx.x;
    const int full = (int)(gridDim.x / (kXcds * kStripe)) * (kXcds * kStripe);
    int tile = g;
    if (g < full) {
        const int xcd = g % kXcds, k = g / kXcds;
        tile = (k / kStripe) * (kXcds * kStripe) + xcd * kStripe + k % kStripe;
    }
    const int b = tile / p.tiles_per_b;
    const int tl = tile - b * p.tiles_per_b;
    // tile origin: a run of T cells (direct) or a tx x ty block (tiled)
    int q_tile = 0, i0 = 0, j0 = 0;
    if constexpr (TILED) {
        const int ti = tl / p.tiles_y;
        i0 = ti * p.tx;
        j0 = (tl - ti * p.tiles_y) * p.ty;
    } else {
        q_tile = tl * T;
    }
    // cell t of the tile -> grid cell index (or -1 outside the grid)
    auto cell_of = [&](int t) -> int {
        if constexpr (TILED) {
            const int a = div_small(t, p.ty, p.rcp_ty);
            const int ci = i0 + a, cj = j0 + (t - a * p.ty);
            return (ci < p.X && cj < p.Y) ? ci * p.Y + cj : -1;
        } else {
            return q_tile + t < p.XY ? q_tile + t : -1;
        }
    };

    // stage camera matrices, heights and the tile's output gradient; in
    // the tiled mode also clear the pixel table, row accumulators and
    // row counter
    for (int t = tid; t < N * 12; t += nthreads) {
        const int n = t / 12, r = t - n * 12;
        s_mat[t] = p.l2i[((size_t)b * N + n) * 16 + r];
    }
    for (int t = tid; t < p.Z; t += nthreads) s_z[t] = p.z[t];
    {
        const float *gb = p.gout + (size_t)b * C * p.XY;
        const int rows = nthreads / T;  // >= 1: a tile has at most nthreads cells
        const int c0 = div_small(tid, T, 1.0f / (float)T);
        const int t = tid - c0 * T;
        const int q = cell_of(t);
        if (c0 < rows && q >= 0)
            for (int c = c0; c < C; c += rows) s_g[c * p.gtile_ld + t] = gb[(size_t)c * p.XY + q];
    }
    if constexpr (TILED) {
        for (uint32_t t = tid; t <= p.tbl_mask; t += nthreads) s_tbl[t] = 0u;
        const int nacc = p.cap * C;
        for (int t = tid; t < nacc; t += nthreads) s_acc[t] = 0.0f;
        for (int t = tid; t < p.cap; t += nthreads) s_rcnt[t] = 0u;
        if (tid == 0) { s_cnt[0] = 0u; s_cnt[1] = 0u; }
    }
    __syncthreads();

    const int Nd = N > 0 ? N : 1;
    const int zl = div_small(lane, Nd, p.rcp_n);
    const int n_p = lane - zl * Nd;
    const bool p_role = (N > 0) && (zl < p.zc);
    const int zshift = p_role ? zl * N : 0;
    const uint64_t nmask = (N >= 64) ? ~0ull : ((1ull << N) - 1ull);
    float mr[12];
#pragma unroll
    for (int k = 0; k < 12; ++k) mr[k] = p_role ? s_mat[n_p * 12 + k] : 0.0f;

    // scatter role: cell m_g of the group, channels slot + L * kk
    const int L = p.lpc;
    const int m_g = div_small(lane, L, p.rcp_lpc);
    const int slot = lane - m_g * L;
    const bool in_group = m_g < cpw;
    const int m_lds = in_group ? m_g : 0;

    float4 *wl = s_w + (size_t)wave * cpw * RS;
    uint32_t *ol = s_off + (size_t)wave * cpw * RS;
    uint2 *sl = s_slot + (size_t)wave * cpw * RS;
    const int wcells = p.rounds * cpw;
    const uint32_t cam0 = (uint32_t)b * (uint32_t)N;
    const uint32_t pix0 = cam0 * (uint32_t)p.H * (uint32_t)p.W;

    // voxel centres and validity of the wavefront's cells, one per lane
    float xs = 0.0f, ys = 0.0f;
    int cv = 0;
    if (lane < wcells) {
        const int q = cell_of(wave * wcells + lane);
        if (q >= 0) {
            const int i = q / p.Y;
            const int j = q - i * p.Y;
            cv = 1;
            xs = p.x_min + ((float)i + 0.5f) * p.dx;
            ys = p.y_min + ((float)j + 0.5f) * p.dy;
        }
    }
    const uint64_t cvmask = __ballot(cv != 0);

    for (int r = 0; r < p.rounds; ++r) {
        const int kg = r * cpw + m_lds;
        const bool g_active = in_group && ((cvmask >> kg) & 1ull);

        // this lane's share of the cell's output gradient
        float gv[KPL];
        {
            const int col = wave * wcells + kg;
#pragma unroll
            for (int kk = 0; kk < KPL; ++kk) {
                const int c = slot + L * kk;
                gv[kk] = (g_active && c < C) ? s_g[c * p.gtile_ld + col] : 0.0f;
            }
        }

        for (int z0 = 0; z0 < p.Z; z0 += p.zc) {
            // rows in use as this pass starts (the last pass ended with a barrier)
            uint32_t used0 = 0;
            if constexpr (TILED) used0 = s_cnt[0] < (uint32_t)p.cap ? s_cnt[0] : (uint32_t)p.cap;
            // ---- projection, mask and compaction (as in the forward)
            const int zi = z0 + zl;
            const bool l_ok = p_role && zi < p.Z;
            const float zv = l_ok ? s_z[zi] : 0.0f;
            const float t2u = mr[2] * zv, t2v = mr[6] * zv, t2d = mr[10] * zv;
            int total = 0;
            int cnt_lane = 0, pre_lane = 0;
            for (int m = 0; m < cpw; ++m) {
                int cnt = 0;
                if ((cvmask >> (r * cpw + m)) & 1ull)
                    cnt = bwd_project_cell(p, mr, t2u, t2v, t2d, bcast(xs, r * cpw + m),
                                           bcast(ys, r * cpw + m), l_ok, zshift, nmask, n_p,
                                           wl + m * RS);
                cnt_lane = lane == m ? cnt : cnt_lane;
                pre_lane = lane == m ? total : pre_lane;
                total += cnt;
            }
            wave_lds_sync();

            // ---- bilinear set-up, dense over the group's valid samples:
            // weights, element index of the first tap in the gradient and,
            // in the tiled mode, the LDS rows of the four taps
            for (int base = 0; base < total; base += kWave) {
                const int idx = base + lane;
                int m = 0, pm = 0;
                for (int mm = 1; mm < cpw; ++mm) {
                    const int pf = __builtin_amdgcn_readlane(pre_lane, mm);
                    const bool ge = idx >= pf;
                    m = ge ? mm : m;
                    pm = ge ? pf : pm;
                }
                if (idx < total) {
                    const int slotk = m * RS + (idx - pm);
                    const float4 pr = wl[slotk];
                    const uint32_t n = __builtin_bit_cast(uint32_t, pr.z);
                    int xa, ya;
                    wl[slotk] = bwd_setup(p, pr.x, pr.y, __builtin_bit_cast(int, pr.w), xa, ya);
                    const uint32_t q = (n * (uint32_t)p.H + (uint32_t)ya) * (uint32_t)p.W + (uint32_t)xa;
                    ol[slotk] = (pix0 + q) * (uint32_t)C;
                    if constexpr (TILED) {
                        // table entries of the four taps' pixels
                        const uint32_t dxp = p.step_x ? 1u : 0u;
                        const uint32_t dyp = p.step_y ? (uint32_t)p.W : 0u;
                        const uint32_t h0 = tile_insert(q, s_tbl, p.tbl_mask);
                        const uint32_t h1 = tile_insert(q + dxp, s_tbl, p.tbl_mask);
                        const uint32_t h2 = tile_insert(q + dyp, s_tbl, p.tbl_mask);
                        const uint32_t h3 = tile_insert(q + dxp + dyp, s_tbl, p.tbl_mask);
                        sl[slotk] = make_uint2(h0 | (h1 << 16), h2 | (h3 << 16));
                    }
                }
            }
            wave_lds_sync();

            if constexpr (TILED) {
                // ---- rows for the pixels first seen in this pass: one claim
                // per table entry, so every distinct pixel gets one row
                __syncthreads();
                for (uint32_t h = tid; h <= p.tbl_mask; h += nthreads) {
                    const uint32_t e = s_tbl[h];
                    if (e != 0u && (e >> kKeyBits) == kRowUnset) {
                        const uint32_t r = atomicAdd(&s_cnt[0], 1u);
                        if (r < (uint32_t)p.cap) {
                            s_tbl[h] = (e & kKeyMask) | (r << kKeyBits);
                            s_spix[r] = (e & kKeyMask) - 1u;
                        } else {
                            // no rows left: the pixel's taps go to global memory
                            s_cnt[1] = 1u;
                        }
                    }
                }
                __syncthreads();
                // ---- count the pass's terms per row (integer LDS atomics)
                for (int base = 0; base < total; base += kWave) {
                    const int idx = base + lane;
                    int m = 0, pm = 0;
                    for (int mm = 1; mm < cpw; ++mm) {
                        const int pf = __builtin_amdgcn_readlane(pre_lane, mm);
                        const bool ge = idx >= pf;
                        m = ge ? mm : m;
                        pm = ge ? pf : pm;
                    }
                    if (idx < total) {
                        const uint2 sh = sl[m * RS + (idx - pm)];
                        const uint32_t hh[4] = {sh.x & 0xFFFFu, sh.x >> 16, sh.y & 0xFFFFu, sh.y >> 16};
                        bool none = false;
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            const uint32_t r = tile_row_of(s_tbl, hh[t]);
                            if (r != kSlotNone) atomicAdd(&s_rcnt[r], 1u);
                            else none = true;
                        }
                        if (none) s_cnt[1] = 1u;
                    }
                }
                // ---- sort the pass's terms by row: prefix of the counts (one
                // wavefront), then each term claims a place in its row's run
                __syncthreads();
                const int nr = (int)(s_cnt[0] < (uint32_t)p.cap ? s_cnt[0] : (uint32_t)p.cap);
                if (wave == 0) {
                    const int per = (nr + kWave - 1) / kWave;
                    const int r0 = lane * per < nr ? lane * per : nr;
                    const int r1 = r0 + per < nr ? r0 + per : nr;
                    uint32_t sum = 0;
                    for (int q = r0; q < r1; ++q) sum += s_rcnt[q];
                    uint32_t incl = sum;
#pragma unroll
                    for (int d = 1; d < kWave; d <<= 1) {
                        const uint32_t t = __shfl_up(incl, d);
                        if (lane >= d) incl += t;
                    }
                    uint32_t run = incl - sum;
                    for (int q = r0; q < r1; ++q) {
                        s_rbase[q] = run;
                        s_rfill[q] = run;
                        run += s_rcnt[q];
                        s_rcnt[q] = 0u;
                    }
                    if (lane == kWave - 1) s_rbase[nr] = incl;
                }
                __syncthreads();
                for (int base = 0; base < total; base += kWave) {
                    const int idx = base + lane;
                    int m = 0, pm = 0;
                    for (int mm = 1; mm < cpw; ++mm) {
                        const int pf = __builtin_amdgcn_readlane(pre_lane, mm);
                        const bool ge = idx >= pf;
                        m = ge ? mm : m;
                        pm = ge ? pf : pm;
                    }
                    if (idx < total) {
                        const int slotk = m * RS + (idx - pm);
                        const uint2 sh = sl[slotk];
                        const uint32_t rr[4] = {tile_row_of(s_tbl, sh.x & 0xFFFFu), tile_row_of(s_tbl, sh.x >> 16),
                                                tile_row_of(s_tbl, sh.y & 0xFFFFu), tile_row_of(s_tbl, sh.y >> 16)};
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            if (rr[t] != kSlotNone) {
                                const uint32_t pos = atomicAdd(&s_rfill[rr[t]], 1u);
                                s_list[pos] = ((uint32_t)wave << 14) | ((uint32_t)slotk << 2) | (uint32_t)t;
                            }
                        }
                    }
                }
            }

            // ---- scatter: each lane adds its channels' terms to the four
            // taps; lanes of cells with fewer samples sit out.  In the tiled
            // mode only taps without an LDS row (table full) come here.
            const int mycnt = __shfl(cnt_lane, m_lds);
            if (g_active && (!TILED || s_cnt[1] != 0u)) {
                const float4 *wv = wl + m_lds * RS;
                const uint32_t *ov = ol + m_lds * RS;
                const uint2 *sv = sl + m_lds * RS;
                for (int k = 0; k < mycnt; ++k) {
                    const float4 w = wv[k];
                    const float wt[4] = {w.x, w.y, w.z, w.w};
                    const uint32_t toff[4] = {0u, p.step_x, p.step_y, p.step_x + p.step_y};
                    float *d = p.gfeat + ov[k] + slot;
                    uint32_t rw[4] = {kSlotNone, kSlotNone, kSlotNone, kSlotNone};
                    if constexpr (TILED) {
                        const uint2 sh = sv[k];
                        rw[0] = tile_row_of(s_tbl, sh.x & 0xFFFFu);
                        rw[1] = tile_row_of(s_tbl, sh.x >> 16);
                        rw[2] = tile_row_of(s_tbl, sh.y & 0xFFFFu);
                        rw[3] = tile_row_of(s_tbl, sh.y >> 16);
                    }
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        if (!TILED || rw[t] == kSlotNone) {
#pragma unroll
                            for (int kk = 0; kk < KPL; ++kk)
                                if (slot + L * kk < C)
                                    unsafeAtomicAdd(d + toff[t] + L * kk, wt[t] * gv[kk]);
                        }
                    }
                }
            }

            if constexpr (TILED) {
                // ---- one wavefront per row: sum the row's terms into it
                // (lanes over channels, the term's weight and cell uniform)
                __syncthreads();
                const int nr = (int)(s_cnt[0] < (uint32_t)p.cap ? s_cnt[0] : (uint32_t)p.cap);
                const float *s_wf = reinterpret_cast<const float *>(s_w);
                const int wstride = cpw * RS;
                const int nwaves = nthreads / kWave;
                for (int row = wave; row < nr; row += nwaves) {
                    const uint32_t e0 = s_rbase[row], n = s_rbase[row + 1] - e0;
                    for (uint32_t k0 = 0; k0 < n; k0 += kWave) {
                        const uint32_t kn = n - k0 < (uint32_t)kWave ? n - k0 : (uint32_t)kWave;
                        // lane i decodes term k0 + i: its weight and its cell's column
                        float wi = 0.0f;
                        uint32_t coli = 0;
                        if ((uint32_t)lane < kn) {
                            const uint32_t ent = s_list[e0 + k0 + lane];
                            const uint32_t we = ent >> 14, sk = (ent >> 2) & 0xFFFu, t = ent & 3u;
                            wi = s_wf[((we * wstride) + sk) * 4u + t];
                            coli = we * wcells + r * cpw + div_small((int)sk, RS, rcp_rs);
                        }
                        if constexpr (!WIDE) {
                            // channels lane and lane + 64 (C <= 128 in the tiled mode):
                            // each term's weight and column are read once for both
                            const int ca = lane, cb = lane + kWave;
                            const float *ga = s_g + (ca < C ? ca : C - 1) * p.gtile_ld;
                            const float *gb = s_g + (cb < C ? cb : C - 1) * p.gtile_ld;
                            float sa = 0.0f, sb = 0.0f;
                            if (C > kWave) {
                                for (uint32_t k = 0; k < kn; ++k) {
                                    const float w = __builtin_bit_cast(
                                        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wi), (int)k));
                                    const uint32_t col = (uint32_t)__builtin_amdgcn_readlane((int)coli, (int)k);
                                    sa = fmaf(w, ga[col], sa);
                                    sb = fmaf(w, gb[col], sb);
                                }
                            } else {
                                for (uint32_t k = 0; k < kn; ++k) {
                                    const float w = __builtin_bit_cast(
                                        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wi), (int)k));
                                    const uint32_t col = (uint32_t)__builtin_amdgcn_readlane((int)coli, (int)k);
                                    sa = fmaf(w, ga[col], sa);
                                }
                            }
                            if (ca < C) s_acc[row * C + ca] += sa;
                            if (cb < C) s_acc[row * C + cb] += sb;
                        } else {
                            // wide rows (128 < C <= kBwdTiledCMax): channel blocks
                            // b * 64 + lane for b < KPL, each term read once for all
                            float sk[KPL];
                            int gofs[KPL];
#pragma unroll
                            for (int b = 0; b < KPL; ++b) {
                                sk[b] = 0.0f;
                                const int c = b * kWave + lane;
                                gofs[b] = (c < C ? c : C - 1) * p.gtile_ld;
                            }
                            for (uint32_t k = 0; k < kn; ++k) {
                                const float w = __builtin_bit_cast(
                                    float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wi), (int)k));
                                const uint32_t col = (uint32_t)__builtin_amdgcn_readlane((int)coli, (int)k);
#pragma unroll
                                for (int b = 0; b < KPL; ++b)
                                    if (b * kWave < C) sk[b] = fmaf(w, s_g[gofs[b] + (int)col], sk[b]);
                            }
#pragma unroll
                            for (int b = 0; b < KPL; ++b) {
                                const int c = b * kWave + lane;
                                if (b * kWave < C && c < C) s_acc[row * C + c] += sk[b];
                            }
                        }
                    }
                }
                __syncthreads();
                // ---- if the next pass may not fit (it may claim as many rows
                // as this one did), add the rows to the gradient now and start
                // again with an empty table
                const uint32_t used = s_cnt[0] < (uint32_t)p.cap ? s_cnt[0] : (uint32_t)p.cap;
                if (z0 + p.zc < p.Z && used + (used - used0) > (uint32_t)p.cap) {
                    const int n_el = (int)used * C;
                    for (int t = tid; t < n_el; t += nthreads) {
                        const int row = div_small(t, C, p.rcp_c);
                        const float v = s_acc[t];
                        if (v != 0.0f)
                            unsafeAtomicAdd(p.gfeat + (size_t)(pix0 + s_spix[row]) * C + (t - row * C), v);
                        s_acc[t] = 0.0f;
                    }
                    for (uint32_t t = tid; t <= p.tbl_mask; t += nthreads) s_tbl[t] = 0u;
                    __syncthreads();
                    if (tid == 0) { s_cnt[0] = 0u; s_cnt[1] = 0u; }
                    __syncthreads();
                }
            } else {
                wave_lds_sync();
            }
        }
    }

    if constexpr (TILED) {
        // ---- one global add per channel of each distinct pixel's row
        __syncthreads();
        const uint32_t used = s_cnt[0] < (uint32_t)p.cap ? s_cnt[0] : (uint32_t)p.cap;
        const int n_el = (int)used * C;
        for (int t = tid; t < n_el; t += nthreads) {
            const int row = div_small(t, C, p.rcp_c);
            const float v = s_acc[t];
            if (v != 0.0f)
                unsafeAtomicAdd(p.gfeat + (size_t)(pix0 + s_spix[row]) * C + (t - row * C), v);
        }
    }
}

// ---------------------------------------------------------------------------
// backward, gather form: one write per gradient element, no atomics
// ---------------------------------------------------------------------------
// The gradient with respect to the features is the transpose of Eq. 1's map.
// In gather form each feature pixel (b, n, py, px) collects its own terms:
// the valid samples (cell, z) of camera n whose bilinear support holds the
// pixel, each adding w_t / max(1, den_z) times the cell's output-gradient
// row.  Two kernels on the caller's stream and workspace:
//   * sample_vt_bwd_prep: the output gradient transposed to cell-major rows
//     Gt[b, cell, C] (so a term's row is one contiguous read), and den_z of
//     every (b, cell, z) (the valid cameras of the point, Eq. 1's divisor).
//   * sample_vt_bwd_gather: a wavefront per group of cpw consecutive columns
//     of two feature-map rows (a sample's taps span two rows, so most of its
//     terms in the group share one load of its gradient row).  For each
//     height the cells that can reach the group's support lie in a convex
//     region of that height's plane,
//     bounded by five half-planes (depth above depth_eps; u and v inside
//     the group's support and the image) with slack for float32 rounding.
//     The region's rows give contiguous runs of candidate cells; each
//     candidate is re-checked with the forward's exact float32 recipe
//     (projection, mask, floor), so mask and tap decisions are the
//     forward's.  The terms go to per-column LDS lists (a row of Gt with its
//     weights for the group's two pixels of that column), and the lanes of a
//     column sum them into both pixels' registers, as the forward gathers
//     feature rows.  Each gradient row is written once; the summation order
//     is fixed, so results are bitwise identical run to run.
struct BwdGatherParams {
    const float *l2i;
    const float *gout;       // [B, C, X, Y]
    float *gfeat;            // [B, N, H, W, C]
    float *gt;               // workspace: [B, X Y, C]
    uint8_t *den;            // workspace: [B, X Y, Z]
    uint32_t gt_bytes;       // bytes of gt (buffer size for the descriptor)
    int32_t B, N, H, W, C, X, Y, Z;
    int32_t XY;
    float img_w, img_h;
    float sx, sy;
    float x_min, dx, y_min, dy, depth_eps;
    int32_t reduce;
    double dx_d, dy_d, x_min_d, y_min_d;  // float64 copies for the regions
    double isx_d, isy_d;        // 1 / sx, 1 / sy in float64 (sx, sy the float32 scales)
    double xmax_abs, ymax_abs;  // bounds on |x|, |y| of a cell centre and its float32 terms
    // prep kernel
    int32_t prep_tiles_per_b;   // 64-cell tiles per batch element
    int32_t prep_cblocks;       // 64-channel blocks
    // gather kernel
    int32_t cpw;             // pixels per wavefront group
    int32_t lpc;             // lanes per pixel
    int32_t nvec;            // LW-byte vectors per gradient row
    float rcp_lpc;
    int32_t groups_per_row;  // pixel groups per group of rows
    int32_t row_groups;      // groups of rows per map: H / rows, rounded up
    int64_t groups;          // all pixel groups (B N row_groups groups_per_row)
    int32_t rec_stride;      // records per pixel list
    uint32_t row_bytes;      // C * 4
    uint32_t lds_wave;       // LDS bytes per wavefront
    float z[FLASHBEV_ZMAX];
};

constexpr int kPrepCells = 64;      // cells per prep workgroup
constexpr int kGatherRec = 128;     // records per pixel list (two candidate chunks)
constexpr int kGatherUnroll = 8;    // terms per gather iteration (loads in flight)
constexpr int kHeightBatch = 32;    // heights whose rows one pass packs together
// LDS bytes per wavefront after its pixel lists (see the kernel's layout)
constexpr uint32_t kGatherTail = 4u * kWave * 4u + (5u * 8u + 36u * 2u + kHeightBatch * 5u) * 8u +
                                 4u * kHeightBatch * 4u;

// Prep: Gt rows of 64 consecutive cells for 64 channels, and a share of
// den_z of those cells (the tile's (cell, height) pairs are split over its
// channel blocks).  256 threads; each moves 16 values with its loads all in
// flight.
__global__ void __launch_bounds__(256) sample_vt_bwd_prep(const BwdGatherParams p)
{
    __shared__ float s_mat[FLASHBEV_NMAX * 12];
    __shared__ float s_t[kPrepCells][65];   // transpose tile, odd pitch
    const int tid = threadIdx.x;
    const int per_b = p.prep_tiles_per_b * p.prep_cblocks;
    const int b = blockIdx.x / per_b;
    const int rem = blockIdx.x - b * per_b;
    const int cb = rem / p.prep_tiles_per_b;
    const int q0 = (rem - cb * p.prep_tiles_per_b) * kPrepCells;
    const int c0 = cb * 64;
    const int ncell = (p.XY - q0) < kPrepCells ? (p.XY - q0) : kPrepCells;
    const int nc = (p.C - c0) < 64 ? (p.C - c0) : 64;
    // Gt[b, q, c] = gout[b, c, q]: reads along cells, writes along channels
    const float *gb = p.gout + (size_t)b * p.C * p.XY;
    float *tb = p.gt + (size_t)b * p.XY * p.C;
    {
        const int cl = tid & 63, cc0 = tid >> 6;
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int cc = cc0 + 4 * u;
            v[u] = (cc < nc && cl < ncell) ? gb[(size_t)(c0 + cc) * p.XY + q0 + cl] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) s_t[cl][cc0 + 4 * u] = v[u];
    }
    __syncthreads();
    {
        const int cc = tid & 63, cl0 = tid >> 6;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int cl = cl0 + 4 * u;
            if (cc < nc && cl < ncell) tb[(size_t)(q0 + cl) * p.C + c0 + cc] = s_t[cl][cc];
        }
    }
    const int N = p.N;
    for (int t = tid; t < N * 12; t += 256) {
        const int n = t / 12, r = t - n * 12;
        s_mat[t] = p.l2i[((size_t)b * N + n) * 16 + r];
    }
    __syncthreads();
    // den_z: thread per (cell, height), cameras in a loop, the forward's
    // recipe (a quotient is formed only where the tests before it pass,
    // which leaves every decision as the forward takes it)
    const int items = ncell * p.Z;
    const int share = (items + p.prep_cblocks - 1) / p.prep_cblocks;
    const int t_end = min(items, (cb + 1) * share);
    for (int t = cb * share + tid; t < t_end; t += 256) {
        const int c = t / p.Z, k = t - c * p.Z;
        const int q = q0 + c;
        const int i = q / p.Y, j = q - (q / p.Y) * p.Y;
        const float x = p.x_min + ((float)i + 0.5f) * p.dx;
        const float y = p.y_min + ((float)j + 0.5f) * p.dy;
        const float zv = p.z[k];
        int den = 0;
        for (int n = 0; n < N; ++n) {
            const float *mr = s_mat + n * 12;
            const float up = ((mr[0] * x + mr[1] * y) + mr[2] * zv) + mr[3];
            const float vp = ((mr[4] * x + mr[5] * y) + mr[6] * zv) + mr[7];
            const float d = ((mr[8] * x + mr[9] * y) + mr[10] * zv) + mr[11];
            if (d > p.depth_eps) {
                const float u = up / d;
                if (u >= 0.0f && u < p.img_w) {
                    const float v = vp / d;
                    den += (v >= 0.0f && v < p.img_h) ? 1 : 0;
                }
            }
        }
        p.den[((size_t)b * p.XY + q) * p.Z + k] = (uint8_t)den;
    }
}

// List entry weights: one float per entry for one-row groups, the two rows'
// weights for two-row groups.
template <int ROWS> struct GatherW { using type = float; };
template <> struct GatherW<2> { using type = float2; };
__device__ __forceinline__ float gw_row0(float w) { return w; }
__device__ __forceinline__ float gw_row0(float2 w) { return w.x; }
__device__ __forceinline__ float gw_row1(float) { return 0.0f; }
__device__ __forceinline__ float gw_row1(float2 w) { return w.y; }

// ROWS: feature-map rows per group (two where a group has at most two
// columns: its per-group set-up and regions then serve twice the pixels, and
// one load of a sample's gradient row serves both rows' terms; one where it
// has more, whose lists would carry many single-row terms).
// Wavefronts per SIMD the compiler must leave room for: four (128 VGPRs),
// which the second row's accumulators would otherwise push to three
// (measured: paper_ref 67 -> 64 us, half_batch 160 -> 150 us); the
// compiler's choice where that would spill (two-row groups of 16-byte lanes
// with several vectors per lane).
template <int LW, int VPL, int ROWS>
struct GatherWaves {
    static constexpr int value = (ROWS == 2 && LW == 16 && VPL >= 2) ? 1 : 4;
};

template <int LW, int VPL, int ROWS>
__global__ void __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(GatherWaves<LW, VPL, ROWS>::value, 8)))
sample_vt_bwd_gather(const BwdGatherParams p)
{
    constexpr int EPV = LW / 4;   // float32 gradient elements per vector
    using WT = typename GatherW<ROWS>::type;
    extern __shared__ __align__(16) unsigned char smem[];
    const int lane = threadIdx.x % kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int RS = p.rec_stride;
    const int cpw = p.cpw;
    unsigned char *wbase = smem + (size_t)wave * p.lds_wave;
    // per column list: the weights for the group's rows, and the Gt row
    WT *wl = reinterpret_cast<WT *>(wbase);                                          // [cpw][RS]
    uint32_t *ol = reinterpret_cast<uint32_t *>(wbase + (size_t)cpw * RS * sizeof(WT));  // [cpw][RS]
    // after the lists (16-byte aligned): per candidate row (64) its cell
    // prefix, first cell, height slot and grid row; the height-free plane
    // terms (5 x 8); the pair slopes (36 x 2); per height of a batch its
    // plane offsets (x 5), row prefix, first row, no-region flag and value
    const uint32_t tail = ((uint32_t)cpw * (uint32_t)RS * (uint32_t)(sizeof(WT) + 4) + 15u) & ~15u;
    int *rpre = reinterpret_cast<int *>(wbase + tail);
    int *rjlo = rpre + kWave;
    int *rhs = rjlo + kWave;
    int *rci = rhs + kWave;
    double *ptab = reinterpret_cast<double *>(rci + kWave);
    double *pairt = ptab + 5 * 8;
    double *hg = pairt + 36 * 2;
    int *hpre = reinterpret_cast<int *>(hg + kHeightBatch * 5);
    int *hilo = hpre + kHeightBatch;
    int *hwild = hilo + kHeightBatch;
    float *hz = reinterpret_cast<float *>(hwild + kHeightBatch);

    // pixel group of this wavefront; workgroups go to the 8 XCDs
    // round-robin, and each XCD takes one contiguous band of groups (the
    // cells a band reaches, hence its rows of Gt, stay in one L2)
    const int64_t nwg = gridDim.x;
    const int64_t per = nwg / kXcds;
    int64_t wg = blockIdx.x;
    if (wg < per * kXcds) wg = (wg % kXcds) * per + wg / kXcds;
    const int64_t grp = wg * (blockDim.x / kWave) + wave;
    if (grp >= p.groups) return;   // wavefront-uniform: no barrier follows
    const int gpr = p.groups_per_row;
    const int64_t row = grp / gpr;
    const int px0 = (int)(grp - row * gpr) * cpw;
    const int py = ROWS * (int)(row % p.row_groups);   // the group's rows: py .. py + nrows - 1
    const int nrows = (ROWS == 1) ? 1 : ((p.H - py) < 2 ? (p.H - py) : 2);
    const int64_t bn = row / p.row_groups;
    const int n = (int)(bn % p.N);
    const int b = (int)(bn / p.N);
    const int g = (p.W - px0) < cpw ? (p.W - px0) : cpw;

    // gather role: pixel m_g of the group, vector slot `slot`
    const int L = p.lpc;
    const int m_g = div_small(lane, L, p.rcp_lpc);
    const int slot = lane - m_g * L;
    const bool g_active = m_g < g;
    const int m_lds = m_g < cpw ? m_g : 0;
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(p.gt, (short)0, (int)p.gt_bytes, 0x00020000);

    float acc[VPL][EPV], acc1[VPL][EPV];   // rows py and py + 1
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
        for (int e = 0; e < EPV; ++e) {
            acc[v][e] = 0.0f;
            acc1[v][e] = 0.0f;
        }

    // camera rows (uniform)
    const float *mg = p.l2i + ((size_t)b * p.N + n) * 16;
    float mr[12];
#pragma unroll
    for (int k = 0; k < 12; ++k) mr[k] = mg[k];

    // the group's support in image coordinates: samples whose first tap is
    // in column [px0 - 1, px0 + g - 1] and row [py - 1, py + nrows - 1],
    // inside the image
    const double U0 = fmax(0.0, ((double)px0 - 0.5) * p.isx_d);
    const double U1 = fmin((double)p.img_w, ((double)(px0 + g) + 0.5) * p.isx_d);
    const double V0 = fmax(0.0, ((double)py - 0.5) * p.isy_d);
    const double V1 = fmin((double)p.img_h, ((double)(py + nrows) + 0.5) * p.isy_d);
    const uint32_t cam_gt = (uint32_t)b * (uint32_t)p.XY * p.row_bytes;
    const uint8_t *denb = p.den + (size_t)b * p.XY * p.Z;

    int cnt_lane = 0;   // lane m holds column m's record count
    int maxcnt = 0;

    auto flush = [&]() {
        const int maxpad = (maxcnt + kGatherUnroll - 1) / kGatherUnroll * kGatherUnroll;
        for (int m = 0; m < g; ++m) {
            const int c = __builtin_amdgcn_readlane(cnt_lane, m);
            for (int k = c + lane; k < maxpad; k += kWave) {
                wl[m * RS + k] = WT{};
                ol[m * RS + k] = kNoTap;
            }
        }
        wave_lds_sync();
        if (g_active) {
            const WT *wv = wl + m_lds * RS;
            const uint32_t *ov = ol + m_lds * RS;
            for (int k = 0; k < maxpad; k += kGatherUnroll) {
                uint32_t base[kGatherUnroll];
                WT w[kGatherUnroll];
#pragma unroll
                for (int u = 0; u < kGatherUnroll; ++u) base[u] = ov[k + u];
#pragma unroll
                for (int u = 0; u < kGatherUnroll; ++u) w[u] = wv[k + u];
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int v = 0; v < VPL; ++v) {
                    const int vi = slot + L * v;
                    if (VPL == 1 || vi < p.nvec) {
                        Raw<LW> t[kGatherUnroll];
#pragma unroll
                        for (int u = 0; u < kGatherUnroll; ++u)
                            t[u] = load_vec<LW>(rsrc, base[u] + (uint32_t)vi * LW, 0u);
#pragma unroll
                        for (int u = 0; u < kGatherUnroll; ++u)
#pragma unroll
                            for (int e = 0; e < EPV; ++e) {
                                const float gv = __builtin_bit_cast(float, t[u].w[e]);
                                acc[v][e] = fmaf(gw_row0(w[u]), gv, acc[v][e]);
                                if constexpr (ROWS == 2)
                                    acc1[v][e] = fmaf(gw_row1(w[u]), gv, acc1[v][e]);
                            }
                    }
                }
            }
        }
        wave_lds_sync();
        cnt_lane = 0;
        maxcnt = 0;
    };

    if (U0 < U1 && V0 < V1 && p.X > 0 && p.Y > 0) {
        // slack bounds: magnitudes of the rows' terms over the grid
        const double Mu0 = fabs((double)mr[0]) * p.xmax_abs + fabs((double)mr[1]) * p.ymax_abs +
                           fabs((double)mr[3]);
        const double Mv0 = fabs((double)mr[4]) * p.xmax_abs + fabs((double)mr[5]) * p.ymax_abs +
                           fabs((double)mr[7]);
        const double Md0 = fabs((double)mr[8]) * p.xmax_abs + fabs((double)mr[9]) * p.ymax_abs +
                           fabs((double)mr[11]);
        // slack: 2^-18 of the magnitudes, far above the float32 recipe's
        // rounding of u', v', d, the quotient, the feature coordinate and
        // the cell centre (a few 2^-24 of the same magnitudes)
        const double e = 3.814697265625e-06;   // 2^-18
        const double yc0 = p.y_min_d + 0.5 * p.dy_d;   // centre of column 0
        const double xr0 = p.x_min_d + 0.5 * p.dx_d;   // centre of row 0
        const double Yd = (double)p.Y, Xd = (double)p.X;
        const double xspan = fabs(xr0) + fabs(p.dx_d) * Xd;   // bound on |x| terms of a row
        // Half-plane q (0: depth above depth_eps, 1: u >= U0, 2: u <= U1,
        // 3: v >= V0, 4: v <= V1) on the plane of height z reads
        // pa_q x + pb_q y + pc_q(z) >= 0, and only pc_q depends on z.  On
        // the grid row at x, in column-index form:
        // pa_q x + gam_q(z) + beta_q j >= 0 with beta_q = pb_q dy, so its
        // kind (the sign of beta_q: a lower bound, an upper bound or no
        // column dependence) is the same at every height.  Lane q < 5
        // tabulates the height-free terms of plane q.
        if (lane < 5) {
            const int q = lane;
            const double ad = mr[8], bd = mr[9];
            const double ra = q <= 2 ? (double)mr[0] : (double)mr[4];
            const double rb = q <= 2 ? (double)mr[1] : (double)mr[5];
            const double S = q == 1 ? U0 : (q == 2 ? U1 : (q == 3 ? V0 : V1));
            const double sg = (q == 1 || q == 3) ? 1.0 : -1.0;
            const double pa = q == 0 ? ad : sg * (ra - S * ad);
            const double pb = q == 0 ? bd : sg * (rb - S * bd);
            const double beta = pb * p.dy_d;
            const int kind = beta > 1e-200 ? 1 : (beta < -1e-200 ? -1 : 0);
            const double rho = kind != 0 ? 1.0 / beta : 0.0;
            const double Bs = pa * p.dx_d;
            ptab[q * 8 + 0] = pa;
            ptab[q * 8 + 1] = pb;
            ptab[q * 8 + 2] = rho;
            ptab[q * 8 + 3] = fabs(beta) * Yd;              // slack of a kind-0 plane
            ptab[q * 8 + 4] = (double)kind;
            ptab[q * 8 + 5] = kind != 0 ? -Bs * rho : Bs;   // row slope T1
        }
        wave_lds_sync();
        int kind[5];
#pragma unroll
        for (int q = 0; q < 5; ++q) kind[q] = __builtin_amdgcn_readfirstlane((int)ptab[q * 8 + 4]);
        // pair (p, q) of 6 x 6 (index 5: the clamps Y and -1): the row slope
        // of "upper bound p minus lower bound q" and its reciprocal
        if (lane < 36) {
            const int pp = lane / 6, qq = lane - pp * 6;
            const double be = (pp == 5 ? 0.0 : ptab[pp * 8 + 5]) - (qq == 5 ? 0.0 : ptab[qq * 8 + 5]);
            pairt[lane * 2 + 0] = be;
            pairt[lane * 2 + 1] = be != 0.0 ? 1.0 / be : 0.0;
        }
        wave_lds_sync();
        for (int k0 = 0; k0 < p.Z; k0 += kHeightBatch) {
            const int nb = (p.Z - k0) < kHeightBatch ? (p.Z - k0) : kHeightBatch;
            // lanes over the batch's heights: each height's offsets gam_q
            // and the range of grid rows that can hold a candidate
            float zv = 0.0f;
            for (int h = 0; h < nb; ++h) {
                const float zh = p.z[k0 + h];
                zv = lane == h ? zh : zv;
            }
            int rows = 0;
            if (lane < nb && __builtin_isfinite(zv)) {
                // (a non-finite height makes u', v' and d non-finite or NaN:
                // the forward's mask rejects every sample of it)
                const double zd = (double)zv;
                const double Mu = Mu0 + fabs((double)mr[2] * zd), Mv = Mv0 + fabs((double)mr[6] * zd),
                             Md = Md0 + fabs((double)mr[10] * zd);
                const double cu = (double)mr[2] * zd + (double)mr[3];
                const double cv = (double)mr[6] * zd + (double)mr[7];
                const double cd = (double)mr[10] * zd + (double)mr[11];
                // rows that are non-finite, near float32 overflow or in its
                // subnormal range get no region: every cell is a candidate
                const bool tame = Mu < 1e36 && Mv < 1e36 && Md < 1e36 &&
                                  (Mu == 0.0 || Mu > 1e-30) && (Mv == 0.0 || Mv > 1e-30) &&
                                  (Md == 0.0 || Md > 1e-30);
                const double pc[5] = {cd - (double)p.depth_eps + e * Md,
                                      (cu - U0 * cd) + e * (Mu + U0 * Md),
                                      -(cu - U1 * cd) + e * (Mu + U1 * Md),
                                      (cv - V0 * cd) + e * (Mv + V0 * Md),
                                      -(cv - V1 * cd) + e * (Mv + V1 * Md)};
                // per plane: the column bound -(pa x + gam) rho (kind != 0)
                // or the value pa x + gam + slack (kind 0) on row r is
                // T0 + T1 r; TM bounds the magnitude of its terms
                double T0[5], TM[5];
#pragma unroll
                for (int q = 0; q < 5; ++q) {
                    const double pa = ptab[q * 8 + 0], rho = ptab[q * 8 + 2], sj = ptab[q * 8 + 3];
                    const double gam = pc[q] + ptab[q * 8 + 1] * yc0;
                    hg[lane * 5 + q] = gam;
                    const double A = pa * xr0 + gam;
                    const double Mq = fabs(pa) * xspan + fabs(gam);
                    T0[q] = kind[q] != 0 ? -A * rho : A + sj;
                    TM[q] = kind[q] != 0 ? Mq * fabs(rho) : Mq + sj;
                }
                // "upper bound p >= lower bound q" holds on a half-line of
                // rows, as does a kind-0 plane; each bound is widened by a
                // row, and a slope under 2^-40 of the terms' magnitude
                // bounds nothing unless the pair fails on every row by more
                int rlo = 0, rhi = p.X - 1;
                bool none = false;
                auto bound = [&](double al, double be, double rbe, double mm) {
                    const double tiny = 9.094947017729282e-13 * mm;   // 2^-40
                    if (fabs(be) > tiny) {
                        const double b = fmin(fmax(-al * rbe, -4.0), Xd + 4.0);
                        if (be > 0.0) rlo = max(rlo, (int)floor(b) - 1);
                        else rhi = min(rhi, (int)ceil(b) + 1);
                    } else {
                        none = none || (al + fabs(be) * Xd < -tiny);
                    }
                };
#pragma unroll
                for (int pp = 0; pp < 6; ++pp) {
#pragma unroll
                    for (int qq = 0; qq < 6; ++qq) {
                        const bool up = pp == 5 || kind[pp] < 0;
                        const bool lw = qq == 5 || kind[qq] > 0;
                        if (!up || !lw || (pp == 5 && qq == 5)) continue;   // uniform
                        const double t0p = pp == 5 ? Yd : T0[pp], mp = pp == 5 ? Yd : TM[pp];
                        const double t0q = qq == 5 ? -1.0 : T0[qq], mq = qq == 5 ? 1.0 : TM[qq];
                        const int j = pp * 6 + qq;
                        bound(t0p - t0q, pairt[j * 2], pairt[j * 2 + 1], mp + mq);
                    }
                }
#pragma unroll
                for (int q = 0; q < 5; ++q) {
                    if (kind[q] != 0) continue;   // uniform
                    const double be = ptab[q * 8 + 5];
                    bound(T0[q], be, be != 0.0 ? 1.0 / be : 0.0, TM[q]);
                }
                if (!tame) { rlo = 0; rhi = p.X - 1; none = false; }
                const int ilo = max(0, rlo), ihi = min(p.X - 1, rhi);
                rows = (!none && ilo <= ihi) ? ihi - ilo + 1 : 0;
                hilo[lane] = ilo;
                hwild[lane] = tame ? 0 : 1;
            }
            if (lane < kHeightBatch) hz[lane] = zv;
            int hincl = rows;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const int t = __shfl_up(hincl, d);
                if (lane >= d) hincl += t;
            }
            const int R = __builtin_amdgcn_readlane(hincl, kWave - 1);
            if (lane < kHeightBatch) hpre[lane] = hincl - rows;
            wave_lds_sync();
            for (int s0 = 0; s0 < R; s0 += kWave) {
                // lanes over the batch's candidate rows, heights packed: the
                // run of candidate cells of each
                const int sl = s0 + lane;
                int jlo = 1, jhi = 0, hs = 0, ri = 0;
                if (sl < R) {
                    // its height: the last with row prefix <= sl
#pragma unroll
                    for (int step = kHeightBatch / 2; step >= 1; step >>= 1)
                        if (hpre[hs + step] <= sl) hs += step;
                    ri = hilo[hs] + (sl - hpre[hs]);
                    if (hwild[hs]) {
                        jlo = 0;
                        jhi = p.Y - 1;
                    } else {
                        const double x = p.x_min_d + ((double)ri + 0.5) * p.dx_d;
                        double lo = -1.0, hi = Yd;
                        bool empty = false;
#pragma unroll
                        for (int q = 0; q < 5; ++q) {
                            const double v = ptab[q * 8 + 0] * x + hg[hs * 5 + q];
                            if (kind[q] > 0) lo = fmax(lo, -v * ptab[q * 8 + 2]);
                            else if (kind[q] < 0) hi = fmin(hi, -v * ptab[q * 8 + 2]);
                            else empty = empty || (v + ptab[q * 8 + 3] < 0.0);
                        }
                        lo = fmin(lo, Yd);
                        hi = fmax(hi, -1.0);
                        if (!empty) {
                            jlo = max(0, (int)ceil(lo));
                            jhi = min(p.Y - 1, (int)floor(hi));
                        }
                    }
                }
                const int cn = jhi >= jlo ? jhi - jlo + 1 : 0;
                // inclusive prefix over the lanes
                int incl = cn;
#pragma unroll
                for (int d = 1; d < kWave; d <<= 1) {
                    const int t = __shfl_up(incl, d);
                    if (lane >= d) incl += t;
                }
                const int total = __builtin_amdgcn_readlane(incl, kWave - 1);
                if (total == 0) continue;
                rpre[lane] = incl - cn;
                rjlo[lane] = jlo;
                rhs[lane] = hs;
                rci[lane] = ri;
                wave_lds_sync();
                for (int kb = 0; kb < total; kb += kWave) {
                    // candidate kb + lane: its row is the last with prefix <= it
                    const int kk = kb + lane;
                    int lo = 0;
#pragma unroll
                    for (int step = 32; step >= 1; step >>= 1)
                        if (lo + step < kWave && rpre[lo + step] <= kk) lo += step;
                    const bool c_ok = kk < total;
                    const int ci = rci[lo];
                    const int cj = rjlo[lo] + (kk - rpre[lo]);
                    const int hc = rhs[lo];
                    const int k = k0 + hc;
                    const float zc = hz[hc];
                    const int q = ci * p.Y + cj;
                    // den_z of the point, read ahead of the test that needs it
                    const int den = c_ok ? (int)denb[(size_t)q * p.Z + k] : 0;
                    // exact test: the forward's recipe for camera n
                    bool t0 = false, t1 = false;
                    WT w0{}, w1{};
                    int x0 = 0;
                    uint32_t goff = 0;
                    if (c_ok) {
                        const float x = p.x_min + ((float)ci + 0.5f) * p.dx;
                        const float y = p.y_min + ((float)cj + 0.5f) * p.dy;
                        const float up = ((mr[0] * x + mr[1] * y) + mr[2] * zc) + mr[3];
                        const float vp = ((mr[4] * x + mr[5] * y) + mr[6] * zc) + mr[7];
                        const float d = ((mr[8] * x + mr[9] * y) + mr[10] * zc) + mr[11];
                        const float u = up / d;
                        const float v = vp / d;
                        const bool ok = (d > p.depth_eps) && (u >= 0.0f) && (u < p.img_w) &&
                                        (v >= 0.0f) && (v < p.img_h);
                        if (ok) {
                            const float xf = u * p.sx - 0.5f;
                            const float yf = v * p.sy - 0.5f;
                            const float x0f = floorf(xf), y0f = floorf(yf);
                            const float ax = xf - x0f, ay = yf - y0f;
                            x0 = (int)x0f;
                            const int y0 = (int)y0f;
                            // the sample's rows y0 (weight 1 - ay) and y0 + 1
                            // (weight ay) meet the group's rows py and py + 1
                            const bool yrow = (y0 >= py - 1) && (y0 <= py + nrows - 1);
                            if (yrow) {
                                const float inv = (p.reduce == 0) ? __builtin_amdgcn_rcpf((float)den) : 1.0f;
                                const float wy0 = ((y0 == py) ? 1.0f - ay : ((y0 == py - 1) ? ay : 0.0f)) * inv;
                                // tap column x0 (1 - ax) and x0 + 1 (ax)
                                if constexpr (ROWS == 2) {
                                    const float wy1 = (nrows == 2)
                                        ? ((y0 == py + 1) ? 1.0f - ay : ((y0 == py) ? ay : 0.0f)) * inv
                                        : 0.0f;
                                    w0 = make_float2((1.0f - ax) * wy0, (1.0f - ax) * wy1);
                                    w1 = make_float2(ax * wy0, ax * wy1);
                                } else {
                                    w0 = (1.0f - ax) * wy0;
                                    w1 = ax * wy0;
                                }
                                t0 = x0 >= px0 && x0 < px0 + g;
                                t1 = x0 + 1 >= px0 && x0 + 1 < px0 + g;
                                goff = cam_gt + (uint32_t)q * p.row_bytes;
                            }
                        }
                    }
                    // append the terms to the columns' lists (candidate order)
                    for (int m = 0; m < g; ++m) {
                        const bool mine = (t0 && x0 == px0 + m) || (t1 && x0 + 1 == px0 + m);
                        const uint64_t mask = __ballot(mine);
                        const int base = __builtin_amdgcn_readlane(cnt_lane, m);
                        if (mine) {
                            const int pos = base + __builtin_amdgcn_mbcnt_hi(
                                                       (uint32_t)(mask >> 32),
                                                       __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                            wl[m * RS + pos] = (x0 == px0 + m) ? w0 : w1;
                            ol[m * RS + pos] = goff;
                        }
                        const int c = base + __popcll(mask);
                        cnt_lane = lane == m ? c : cnt_lane;
                        maxcnt = c > maxcnt ? c : maxcnt;
                    }
                    // a list may take up to 64 more terms before the next flush
                    if (maxcnt > RS - 1 - kWave - kGatherUnroll) flush();
                }
                wave_lds_sync();
            }
            wave_lds_sync();   // the height tables are rewritten by the next batch
        }
    }
    if (maxcnt > 0) flush();

    // single write of the group's gradient rows (NHWC, contiguous)
    if (g_active) {
        float *dst = p.gfeat + ((((size_t)b * p.N + n) * p.H + py) * p.W + px0 + m_g) * p.C;
        float *dst1 = dst + (size_t)p.W * p.C;   // row py + 1
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
            const int vi = slot + L * v;
            if (VPL == 1 || vi < p.nvec) {
#pragma unroll
                for (int e = 0; e < EPV; ++e) dst[vi * EPV + e] = acc[v][e];
                if (ROWS == 2 && nrows == 2) {
#pragma unroll
                    for (int e = 0; e < EPV; ++e) dst1[vi * EPV + e] = acc1[v][e];
                }
            }
        }
    }
}

// Zero-fills n floats at dst (any 4-byte alignment): a 16-byte aligned body
// with vector stores plus scalar head and tail.
__global__ void __launch_bounds__(256) zero_fill(float *dst, uint64_t n)
{
    const uintptr_t a = (uintptr_t)dst;
    uint64_t head = ((16u - (a & 15u)) & 15u) / 4u;
    if (head > n) head = n;
    const uint64_t n4 = (n - head) / 4u;
    const uint64_t tail0 = head + n4 * 4u;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    const uint64_t t0 = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    float4 *body = reinterpret_cast<float4 *>(dst + head);
    for (uint64_t i = t0; i < n4; i += stride) body[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (t0 < head) dst[t0] = 0.0f;
    if (t0 < n - tail0) dst[tail0 + t0] = 0.0f;
}

// ---------------------------------------------------------------------------
// host side: validation, geometry, dispatch
// ---------------------------------------------------------------------------
using KernelFn = void (*)(const Params);

template <int DT, int LW, bool CULL>
KernelFn pick_vpl(int vpl)
{
    switch (vpl) {
    case 1: return sample_vt_fwd<DT, LW, 1, CULL>;
    case 2: return sample_vt_fwd<DT, LW, 2, CULL>;
    default: return sample_vt_fwd<DT, LW, 4, CULL>;
    }
}

template <int DT, bool CULL>
KernelFn pick_lw(int lw, int vpl)
{
    switch (lw) {
    case 16: return pick_vpl<DT, 16, CULL>(vpl);
    case 8: return pick_vpl<DT, 8, CULL>(vpl);
    case 4: return pick_vpl<DT, 4, CULL>(vpl);
    default:
        if constexpr (DT == FLASHBEV_F32) return nullptr;
        else return pick_vpl<DT, 2, CULL>(vpl);
    }
}

template <bool CULL>
KernelFn pick_dtype(int dtype, int lw, int vpl)
{
    switch (dtype) {
    case FLASHBEV_F32: return pick_lw<FLASHBEV_F32, CULL>(lw, vpl);
    case FLASHBEV_F16: return pick_lw<FLASHBEV_F16, CULL>(lw, vpl);
    default: return pick_lw<FLASHBEV_BF16, CULL>(lw, vpl);
    }
}

KernelFn pick_kernel(int dtype, int lw, int vpl, bool cull)
{
    return cull ? pick_dtype<true>(dtype, lw, vpl) : pick_dtype<false>(dtype, lw, vpl);
}

struct Plan {
    Params prm;
    int64_t workgroups;
    int threads;
    size_t lds;
    int lw, vpl;
    bool cull_path;     // the culled, packed projection phase
    bool empty;
    bool band_work;     // little enough work for contiguous bands
};

bool finite(float v) { return v == v && v - v == 0.0f; }

bool overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    if (!na || !nb) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
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
    // every size product saturates instead of wrapping (size_prod)
    const uint64_t feat_bytes =
        size_prod({(uint64_t)f->B, (uint64_t)f->N, (uint64_t)f->H, (uint64_t)f->W, row});
    if (feat_bytes > kFeatBytesMax) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t XY = size_prod({(uint64_t)s->X, (uint64_t)s->Y});
    if (XY > 0x7FFFFFFFull) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t out_elems = size_prod({(uint64_t)f->B, (uint64_t)f->C, XY});
    if (out_elems > kSizeCap / 4) return FLASHBEV_ERR_UNSUPPORTED;
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
    // wide rows: give a lane several vectors so that a wavefront covers at
    // least two cells (four from 1 KiB rows on), which shares the set-up
    // pass among more cells (measured on MI355X: C=256 float32 124 -> 81 us,
    // C=512 278 -> 200 us at the paper's reference setting)
    const int min_cpw = row >= 1024 ? 4 : 2;
    while (vpl < 4 && kWave / ((nvec + vpl - 1) / vpl) < min_cpw && nvec >= 2 * vpl) vpl <<= 1;
    const int lpc = (nvec + vpl - 1) / vpl;
    if (lpc > kWave) return FLASHBEV_ERR_UNSUPPORTED;
    int cpw = kWave / lpc;
    if (cpw > kCpwMax) cpw = kCpwMax;
    // Workgroup size (measured on MI355X): with a full group of kCpwMax
    // cells per pass a wavefront has enough work per tile and 4-wavefront
    // workgroups are fastest; with fewer cells per pass (wider rows)
    // 2-wavefront workgroups give twice the tiles and a shorter tail.
    const int waves = cpw >= kCpwMax ? kWavesMax : 2;
    // tile: at least kCellsPerWave cells per wavefront, fewer if the output
    // tile would not fit the LDS budget (very wide rows).  Where a wavefront
    // holds at most two cells or a lane several vectors, one round per tile
    // is faster as long as the grid does not get too many workgroups
    // (measured on MI355X at the paper's reference setting, C=128 float32:
    // 200x200 41.8 -> 35.2 us, 800x800 432 -> 401 us; but 1600x1600
    // 1.44 -> 1.99 ms, where per-workgroup set-up dominates)
    // Projection phase (measured on MI355X, per-cell -> culled: long_range
    // 98.7 -> 72.5 us, z_sweep Z=8 206 -> 176, half_batch 73.3 -> 69.5; but
    // rep 22.2 -> 23.4 and the paper's reference setting 31.3 -> 31.7, whose
    // groups of 2-3 cells already fill one pass per cell): the culled,
    // packed phase for groups of at least 4 cells or cells needing several
    // per-cell passes, where the culling pass (one lane per cell and camera)
    // fits a wavefront.
    const uint64_t zn = size_prod({(uint64_t)zb->Z, (uint64_t)(f->N > 0 ? f->N : 1)});
    const bool cull_path = f->N > 0 && zb->Z > 0 && cpw * f->N <= kWave &&
                           (cpw >= 4 || zn > (uint64_t)kWave);
    // The packed phase also takes one round per tile (half_batch 68.9 ->
    // 67.6 us; rep on the per-cell phase is fastest with two: one 24.9,
    // three 25.0, two 22.1 us).
    int rounds = (kCellsPerWave + cpw - 1) / cpw;
    if ((cpw <= 2 || vpl >= 2 || cull_path) &&
        size_prod({(uint64_t)f->B, XY}) <= (uint64_t)waves * cpw * kOneRoundTilesMax)
        rounds = 1;
    // heights per per-cell pass (at most 64 / N, so zc N <= 64)
    int zc = f->N > 0 ? kWave / f->N : 1;
    if (zc > zb->Z && zb->Z > 0) zc = zb->Z;
    if (zc < 1) zc = 1;
    // a cell's list holds the valid samples of one pass over its heights,
    // padded to whole gather iterations: at most zc N (per-cell passes) or
    // min(64, Z N) (packed passes of at most 64 lanes)
    const int pass_cap = cull_path ? (zn < (uint64_t)kWave ? (int)zn : kWave)
                                   : zc * (f->N > 0 ? f->N : 1);
    const int rec_cap = (pass_cap + kUnroll - 1) / kUnroll * kUnroll;
    const int rs = rec_cap | 1;
    auto pitch = [&](int r) { return (waves * r * cpw) | 1; };
    // after the shared layout: each wavefront's list of visible cameras
    const uint32_t cl_bytes = (uint32_t)waves * kWave * 4u;
    LdsLayout lay = lds_layout(f->N, zb->Z, waves, cpw, f->C, pitch(rounds), rs);
    while (lay.total + cl_bytes > kLdsBudget && rounds > 1) {
        --rounds;
        lay = lds_layout(f->N, zb->Z, waves, cpw, f->C, pitch(rounds), rs);
    }
    const uint32_t lds_cl = lay.total;
    lay.total += cl_bytes;
    if (lay.total > kLdsBudget) return FLASHBEV_ERR_UNSUPPORTED;
    // a wavefront's cells fit its lanes (centre precompute) and a tile fits
    // the workgroup's threads (output store)
    if (rounds * cpw > kWave) return FLASHBEV_ERR_UNSUPPORTED;
    const int tile_cells = waves * rounds * cpw;
    const int otile_ld = pitch(rounds);

    Params &p = pl->prm;
    memset(&p, 0, sizeof(p));
    p.feat = f->data;
    p.l2i = l2i;
    p.out = const_cast<float *>(out);
    p.feat_bytes = (uint32_t)feat_bytes;
    p.B = f->B; p.N = f->N; p.H = f->H; p.W = f->W; p.C = f->C;
    p.X = s->X; p.Y = s->Y; p.Z = zb->Z;
    p.XY = (int32_t)XY;
    p.tile_cells = tile_cells;
    p.rounds = rounds;
    p.tiles_per_b = (int32_t)((XY + tile_cells - 1) / tile_cells);
    p.img_w = (float)f->img_w;
    p.img_h = (float)f->img_h;
    p.sx = (float)f->W / (float)f->img_w;
    p.sy = (float)f->H / (float)f->img_h;
    p.x_min = s->x_min; p.dx = s->dx; p.y_min = s->y_min; p.dy = s->dy;
    p.depth_eps = s->depth_eps;
    p.reduce = s->reduce;
    p.bands = 0;       // forward_order, at launch
    p.tail_prio = 0;
    pl->band_work = size_prod({(uint64_t)f->B, XY, (uint64_t)zb->Z, row}) <= kBandsWorkMax;
    p.row_bytes = (uint32_t)row;
    p.step_x = f->W >= 2 ? (uint32_t)row : 0u;
    p.step_y = f->H >= 2 ? (uint32_t)(row * f->W) : 0u;
    p.nvec = nvec;
    p.lpc = lpc;
    p.cpw = cpw;
    p.rcp_n = 1.0f / (float)(f->N > 0 ? f->N : 1);
    p.rcp_lpc = 1.0f / (float)lpc;
    p.zc = zc;
    p.otile_ld = otile_ld;
    p.rec_stride = rs;
    p.cull = cull_path ? 1 : 0;
    if (zb->Z > 0) {
        float lo = zb->z[0], hi = zb->z[0];
        for (int k = 1; k < zb->Z; ++k) {
            lo = zb->z[k] < lo ? zb->z[k] : lo;
            hi = zb->z[k] > hi ? zb->z[k] : hi;
        }
        p.zlo = lo;
        p.zhi = hi;
        p.zabs = fabsf(lo) > fabsf(hi) ? fabsf(lo) : fabsf(hi);
        // a non-finite height: no culling (the test's margins assume finite ends)
        if (!finite(lo) || !finite(hi)) p.cull = 0;
    }
    p.rcp_y = 1.0 / (double)(s->Y > 0 ? s->Y : 1);
    p.rcp_tiles = 1.0 / (double)(p.tiles_per_b > 0 ? p.tiles_per_b : 1);
    p.store_rows = waves * kWave / tile_cells;
    p.rcp_tile = 1.0f / (float)tile_cells;
    // one camera's map and one map row in bytes (below 2 GiB: the whole
    // tensor is)
    p.cam_bytes = (uint32_t)size_prod({(uint64_t)f->H, (uint64_t)f->W, row});
    p.wrow_bytes = (uint32_t)size_prod({(uint64_t)f->W, row});
    p.small24 = ((uint64_t)f->H < (1u << 24) && (uint64_t)p.wrow_bytes < (1u << 24) &&
                 (uint64_t)f->W < (1u << 24)) ? 1 : 0;
    p.lds_z = lay.z;
    p.lds_w = lay.w;
    p.lds_off = lay.off;
    p.lds_otile = lay.otile;
    p.lds_cl = lds_cl;
    for (int k = 0; k < zb->Z; ++k) p.z[k] = zb->z[k];

    pl->workgroups = empty ? 0 : (int64_t)f->B * p.tiles_per_b;
    if (pl->workgroups > 0x7FFFFFFFll) return FLASHBEV_ERR_UNSUPPORTED;
    pl->threads = waves * kWave;
    pl->lds = lay.total;
    pl->lw = lw;
    pl->vpl = vpl;
    pl->cull_path = cull_path;
    pl->empty = empty;
    return FLASHBEV_OK;
}

// Backward launch plan.  The feature dims come in a flashbev_features whose
// data pointer is not used; the gradient is float32 whatever the feature
// dtype.
struct BwdPlan {
    BwdParams prm;
    int64_t workgroups;   // scatter workgroups (0: nothing to scatter)
    int threads;
    size_t lds;
    int kpl;
    bool tiled;
    bool wide;              // tiled with more than 128 channels
    uint64_t gfeat_elems;
};

using BwdKernelFn = void (*)(const BwdParams);

template <bool TILED>
BwdKernelFn pick_bwd_kpl(int kpl)
{
    switch (kpl) {
    case 4: return sample_vt_bwd<4, TILED, false>;
    case 8: return sample_vt_bwd<8, TILED, false>;
    case 16: return sample_vt_bwd<16, TILED, false>;
    default: return sample_vt_bwd<32, TILED, false>;
    }
}

// tiled mode with rows wider than 128 channels (KPL 4 or 8 there)
BwdKernelFn pick_bwd_wide(int kpl)
{
    return kpl <= 4 ? sample_vt_bwd<4, true, true> : sample_vt_bwd<8, true, true>;
}

BwdKernelFn pick_bwd(int kpl, bool tiled, bool wide)
{
    if (wide) return pick_bwd_wide(kpl);
    return tiled ? pick_bwd_kpl<true>(kpl) : pick_bwd_kpl<false>(kpl);
}

// All argument checks; `need_data` requires the device pointers.
int make_bwd_plan(const flashbev_features *f, const float *l2i, const flashbev_bev_grid_spec *s,
                  const flashbev_z_bins *zb, const float *gout, const float *gfeat, bool need_data,
                  BwdPlan *pl)
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
    if ((uint64_t)f->C * es > FLASHBEV_ROW_BYTES_MAX) return FLASHBEV_ERR_UNSUPPORTED;
    // every size product saturates instead of wrapping (size_prod)
    const uint64_t gelems = size_prod(
        {(uint64_t)f->B, (uint64_t)f->N, (uint64_t)f->H, (uint64_t)f->W, (uint64_t)f->C});
    if (gelems > 0x7FFFFFFFull) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t XY = size_prod({(uint64_t)s->X, (uint64_t)s->Y});
    if (XY > 0x7FFFFFFFull) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t out_elems = size_prod({(uint64_t)f->B, (uint64_t)f->C, XY});
    if (out_elems > kSizeCap / 4) return FLASHBEV_ERR_UNSUPPORTED;
    if (zb->Z > 0 && !zb->z) return FLASHBEV_ERR_NULLPTR;
    if (need_data && gelems > 0) {
        if (!gfeat) return FLASHBEV_ERR_NULLPTR;
        if ((uintptr_t)gfeat % 4) return FLASHBEV_ERR_ALIGN;
    }
    const bool scatter = gelems > 0 && out_elems > 0 && zb->Z > 0;
    if (need_data && scatter) {
        if (!gout || !l2i) return FLASHBEV_ERR_NULLPTR;
        if (((uintptr_t)gout % 4) || ((uintptr_t)l2i % 4)) return FLASHBEV_ERR_ALIGN;
        const size_t gb = gelems * 4;
        if (overlaps(gfeat, gb, gout, out_elems * 4) ||
            overlaps(gfeat, gb, l2i, (size_t)f->B * f->N * 64))
            return FLASHBEV_ERR_ALIAS;
    }

    // lanes per cell: one channel per lane and up to four lanes' worth of
    // channels per lane for narrow rows, at most one wavefront per cell
    int lpc = (f->C + 3) / 4;
    if (lpc > kWave) lpc = kWave;
    const int k_need = (f->C + lpc - 1) / lpc;
    int kpl = 4;
    while (kpl < k_need) kpl <<= 1;
    if (kpl > 32) return FLASHBEV_ERR_UNSUPPORTED;
    int cpw = kWave / lpc;
    if (cpw > kCpwMax) cpw = kCpwMax;
    const int waves = cpw >= kCpwMax ? kWavesMax : 2;
    int rounds = (kCellsPerWave + cpw - 1) / cpw;
    auto pitch = [&](int r) { return (waves * r * cpw) | 1; };
    // same LDS layout as the forward; the output tile holds the gradient
    LdsLayout lay = lds_layout(f->N, zb->Z, waves, cpw, f->C, pitch(rounds));
    while (lay.total > kLdsBudget && rounds > 1) {
        --rounds;
        lay = lds_layout(f->N, zb->Z, waves, cpw, f->C, pitch(rounds));
    }
    if (lay.total > kLdsBudget) return FLASHBEV_ERR_UNSUPPORTED;
    if (rounds * cpw > kWave) return FLASHBEV_ERR_UNSUPPORTED;
    int tile_cells = waves * rounds * cpw;

    // tiled mode: kBwdTileWaves wavefronts of one group each on a 2-D tile
    // with four cells per tile row; LDS holds the per-wave records, the row
    // table, the pass's sorted term list (sized for the pass's largest
    // possible number of terms) and as many per-pixel rows as the budget
    // leaves
    const uint64_t npix = size_prod({(uint64_t)f->N, (uint64_t)f->H, (uint64_t)f->W});
    bool tiled = false;
    int t_waves = 0, t_tx = 0, t_ty = 0, t_cap = 0, t_zc = 0;
    uint32_t t_mask = 0, l_slot = 0, l_tbl = 0, l_spix = 0, l_acc = 0, l_cnt = 0, l_total = 0;
    uint32_t l_rcnt = 0, l_rbase = 0, l_rfill = 0, l_list = 0;
    int t_pitch = 0;
    int t_rs = kRecStride;
    // rows up to kBwdTiledCMax channels (wider ones leave too few LDS rows);
    // grid sides that leave a tile's cell coordinates (side + tile side)
    // within int32
    if (npix < (1u << kKeyBits) - 1u && f->C <= kBwdTiledCMax && f->N > 0 &&
        (uint64_t)s->X + 2u * kWave < 0x7FFFFFFFull && (uint64_t)s->Y + 2u * kWave < 0x7FFFFFFFull) {
        t_waves = kBwdTileWaves;
        const int T = t_waves * cpw;
        t_ty = (T % 4 == 0) ? 4 : T;
        t_tx = T / t_ty;
        t_pitch = T | 1;
        int zc_max = kWave / f->N;
        if (zc_max > zb->Z && zb->Z > 0) zc_max = zb->Z;
        if (zc_max < 1) zc_max = 1;
        // passes of half the heights a wavefront can project at once, fewer
        // where the LDS needs it; records sized to one pass
        for (int zc_try = zc_max > 1 ? zc_max / 2 : 1; zc_try >= 1 && !tiled;
             zc_try = zc_try > 1 ? zc_try / 2 : 0) {
            const int rs_try = ((zc_try * f->N + 1) / 2 * 2) | 1;
            const LdsLayout base = lds_layout(f->N, zb->Z, t_waves, cpw, f->C, t_pitch, rs_try);
            uint32_t o = base.total;
            const uint32_t lslot = o; o = align16(o + (uint32_t)t_waves * cpw * rs_try * 8u);
            const uint32_t lcnt = o; o = align16(o + 16u);
            const uint32_t entries_max = 4u * (uint32_t)t_waves * cpw * (uint32_t)(zc_try * f->N);
            const uint32_t llist = o; o = align16(o + entries_max * 4u);
            // per row: C floats, a pixel id, two table entries and the
            // count, base and fill words
            const uint32_t per_row = (uint32_t)f->C * 4u + 4u + 8u + 12u;
            int cap = o < kLdsBudgetBwd ? (int)((kLdsBudgetBwd - o) / per_row) : 0;
            if (cap > kSlotMax - 1) cap = kSlotMax - 1;
            auto total_for = [&](int c, uint32_t ent) {
                uint32_t t = o;
                t = align16(t + ent * 4u);
                t = align16(t + (uint32_t)c * 4u);          // spix
                t = align16(t + (uint32_t)c * 4u);          // rcnt
                t = align16(t + ((uint32_t)c + 1u) * 4u);   // rbase
                t = align16(t + (uint32_t)c * 4u);          // rfill
                t = align16(t + (uint32_t)c * f->C * 4u);   // rows
                return t;
            };
            uint32_t entries = 1;
            while (entries < 2u * (uint32_t)cap) entries <<= 1;
            while (cap >= 16 && total_for(cap, entries) > kLdsBudgetBwd) {
                --cap;
                entries = 1;
                while (entries < 2u * (uint32_t)cap) entries <<= 1;
            }
            if (cap >= 16) {
                l_slot = lslot;
                l_cnt = lcnt;
                l_list = llist;
                l_tbl = o; o = align16(o + entries * 4u);
                l_spix = o; o = align16(o + (uint32_t)cap * 4u);
                l_rcnt = o; o = align16(o + (uint32_t)cap * 4u);
                l_rbase = o; o = align16(o + ((uint32_t)cap + 1u) * 4u);
                l_rfill = o; o = align16(o + (uint32_t)cap * 4u);
                l_acc = o; o = align16(o + (uint32_t)cap * f->C * 4u);
                l_total = o;
                t_cap = cap;
                t_mask = entries - 1u;
                t_zc = zc_try;
                t_rs = rs_try;
                tiled = true;
            }
        }
    }
    if (tiled) tile_cells = t_waves * cpw;

    BwdParams &p = pl->prm;
    memset(&p, 0, sizeof(p));
    p.l2i = l2i;
    p.gout = gout;
    p.gfeat = const_cast<float *>(gfeat);
    p.B = f->B; p.N = f->N; p.H = f->H; p.W = f->W; p.C = f->C;
    p.X = s->X; p.Y = s->Y; p.Z = zb->Z;
    p.XY = (int32_t)XY;
    p.tile_cells = tile_cells;
    p.rounds = tiled ? 1 : rounds;
    p.tiles_per_b = (int32_t)((XY + tile_cells - 1) / tile_cells);
    if (tiled) {
        p.tx = t_tx;
        p.ty = t_ty;
        const int64_t tiles_y = ((int64_t)s->Y + t_ty - 1) / t_ty;
        const int64_t tiles = (((int64_t)s->X + t_tx - 1) / t_tx) * tiles_y;
        if (tiles > 0x7FFFFFFFll) return FLASHBEV_ERR_UNSUPPORTED;
        p.tiles_y = (int32_t)tiles_y;
        p.tiles_per_b = (int32_t)tiles;
        p.rcp_ty = 1.0f / (float)t_ty;
        p.rcp_c = 1.0f / (float)f->C;
        p.cap = t_cap;
        p.tbl_mask = t_mask;
        p.lds_slot = l_slot;
        p.lds_tbl = l_tbl;
        p.lds_spix = l_spix;
        p.lds_acc = l_acc;
        p.lds_cnt = l_cnt;
        p.lds_rcnt = l_rcnt;
        p.lds_rbase = l_rbase;
        p.lds_rfill = l_rfill;
        p.lds_list = l_list;
    }
    p.img_w = (float)f->img_w;
    p.img_h = (float)f->img_h;
    p.sx = (float)f->W / (float)f->img_w;
    p.sy = (float)f->H / (float)f->img_h;
    p.x_min = s->x_min; p.dx = s->dx; p.y_min = s->y_min; p.dy = s->dy;
    p.depth_eps = s->depth_eps;
    p.reduce = s->reduce;
    p.step_x = f->W >= 2 ? (uint32_t)f->C : 0u;
    p.step_y = f->H >= 2 ? (uint32_t)f->C * (uint32_t)f->W : 0u;
    p.lpc = lpc;
    p.cpw = cpw;
    p.rcp_n = 1.0f / (float)(f->N > 0 ? f->N : 1);
    p.rcp_lpc = 1.0f / (float)lpc;
    int zc = f->N > 0 ? kWave / f->N : 1;
    if (zc > zb->Z && zb->Z > 0) zc = zb->Z;
    p.zc = tiled ? t_zc : (zc < 1 ? 1 : zc);
    p.gtile_ld = tiled ? t_pitch : pitch(rounds);
    if (tiled) lay = lds_layout(f->N, zb->Z, t_waves, cpw, f->C, t_pitch, t_rs);
    p.rec_stride = tiled ? t_rs : kRecStride;
    p.lds_z = lay.z;
    p.lds_w = lay.w;
    p.lds_off = lay.off;
    p.lds_gtile = lay.otile;
    for (int k = 0; k < zb->Z; ++k) p.z[k] = zb->z[k];

    pl->workgroups = scatter ? (int64_t)f->B * p.tiles_per_b : 0;
    if (pl->workgroups > 0x7FFFFFFFll) return FLASHBEV_ERR_UNSUPPORTED;
    pl->threads = (tiled ? t_waves : waves) * kWave;
    pl->lds = tiled ? l_total : lay.total;
    pl->kpl = kpl;
    pl->tiled = tiled;
    pl->wide = tiled && f->C > 2 * kWave;
    if (pl->wide && kpl > 8) return FLASHBEV_ERR_UNSUPPORTED;
    pl->gfeat_elems = gelems;
    return FLASHBEV_OK;
}

// Plan of the gather-form backward (sample_vt_bwd_prep, sample_vt_bwd_gather).
struct BwdGatherPlan {
    BwdGatherParams prm;
    int64_t prep_wgs;      // prep workgroups (0: no cells)
    int64_t gather_wgs;    // gather workgroups (0: no pixels)
    size_t lds;            // gather dynamic LDS per workgroup
    int lw, vpl;
    int rows;              // feature-map rows per gather group
    uint64_t ws_bytes;     // workspace bytes needed
};

constexpr int kGatherWaves = 1;   // gather: wavefronts per workgroup (one: finest balance)

using BwdGatherFn = void (*)(const BwdGatherParams);

template <int LW, int ROWS>
BwdGatherFn pick_gather_vpl(int vpl)
{
    switch (vpl) {
    case 1: return sample_vt_bwd_gather<LW, 1, ROWS>;
    case 2: return sample_vt_bwd_gather<LW, 2, ROWS>;
    default: return sample_vt_bwd_gather<LW, 4, ROWS>;
    }
}

template <int ROWS>
BwdGatherFn pick_gather_lw(int lw, int vpl)
{
    switch (lw) {
    case 16: return pick_gather_vpl<16, ROWS>(vpl);
    case 8: return pick_gather_vpl<8, ROWS>(vpl);
    default: return pick_gather_vpl<4, ROWS>(vpl);
    }
}

BwdGatherFn pick_gather(int lw, int vpl, int rows)
{
    return rows == 2 ? pick_gather_lw<2>(lw, vpl) : pick_gather_lw<1>(lw, vpl);
}

uint64_t align256(uint64_t v) { return (v + 255u) & ~(uint64_t)255u; }

// All argument checks of the gather-form backward, the workspace's layout
// and size.  `need_data` requires the device pointers (and the workspace).
int make_bwd_gather_plan(const flashbev_features *f, const float *l2i,
                         const flashbev_bev_grid_spec *s, const flashbev_z_bins *zb,
                         const float *gout, const float *gfeat, const void *ws, uint64_t ws_bytes,
                         bool need_data, BwdGatherPlan *pl, bool check_ws = true)
{
    // the shape, value, pointer and alias checks of the scatter-form backward
    BwdPlan bp;
    const int rc = make_bwd_plan(f, l2i, s, zb, gout, gfeat, need_data, &bp);
    if (rc) return rc;
    const uint64_t XY = (uint64_t)s->X * (uint64_t)s->Y;
    const uint64_t row = (uint64_t)f->C * 4u;   // float32 gradient rows
    if (row > FLASHBEV_ROW_BYTES_MAX) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t gt_bytes = size_prod({(uint64_t)f->B, XY, row});
    if (gt_bytes > kFeatBytesMax) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t den_bytes = size_prod({(uint64_t)f->B, XY, (uint64_t)zb->Z});
    if (den_bytes > kFeatBytesMax) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t need = align256(gt_bytes) + align256(den_bytes);
    memset(pl, 0, sizeof(*pl));
    pl->ws_bytes = need;
    const uint64_t gelems = bp.gfeat_elems;
    if (need_data && check_ws && gelems > 0 && need > 0) {
        if (!ws) return FLASHBEV_ERR_NULLPTR;
        if ((uintptr_t)ws % 256u) return FLASHBEV_ERR_ALIGN;
        if (ws_bytes < need) return FLASHBEV_ERR_VALUE;
        // the workspace overlaps none of the call's buffers
        if (overlaps(ws, need, gfeat, gelems * 4) ||
            overlaps(ws, need, gout, size_prod({(uint64_t)f->B, (uint64_t)f->C, XY}) * 4) ||
            overlaps(ws, need, l2i, (size_t)f->B * f->N * 64))
            return FLASHBEV_ERR_ALIAS;
    }
    // lanes over a gradient row: the widest of 16/8/4-byte vectors, one to
    // four per lane so that a wavefront holds at least two pixels (four from
    // 1 KiB rows on), as the forward lays out its feature rows
    int lw = 16;
    while (lw > 4 && (row % lw) != 0) lw >>= 1;
    const int nvec = (int)(row / lw);
    int vpl = 1;
    while (vpl < 4 && (nvec + vpl - 1) / vpl > kWave) vpl <<= 1;
    const int min_cpw = row >= 1024 ? 4 : 2;
    while (vpl < 4 && kWave / ((nvec + vpl - 1) / vpl) < min_cpw && nvec >= 2 * vpl) vpl <<= 1;
    const int lpc = (nvec + vpl - 1) / vpl;
    if (lpc > kWave) return FLASHBEV_ERR_UNSUPPORTED;
    int cpw = kWave / lpc;
    if (cpw > kCpwMax) cpw = kCpwMax;

    BwdGatherParams &p = pl->prm;
    p.l2i = l2i;
    p.gout = gout;
    p.gfeat = const_cast<float *>(gfeat);
    p.gt = reinterpret_cast<float *>(const_cast<void *>(ws));
    p.den = ws ? reinterpret_cast<uint8_t *>(const_cast<void *>(ws)) + align256(gt_bytes) : nullptr;
    p.gt_bytes = (uint32_t)gt_bytes;
    p.B = f->B; p.N = f->N; p.H = f->H; p.W = f->W; p.C = f->C;
    p.X = s->X; p.Y = s->Y; p.Z = zb->Z;
    p.XY = (int32_t)XY;
    p.img_w = (float)f->img_w;
    p.img_h = (float)f->img_h;
    p.sx = (float)f->W / (float)f->img_w;
    p.sy = (float)f->H / (float)f->img_h;
    p.x_min = s->x_min; p.dx = s->dx; p.y_min = s->y_min; p.dy = s->dy;
    p.depth_eps = s->depth_eps;
    p.reduce = s->reduce;
    p.dx_d = s->dx; p.dy_d = s->dy; p.x_min_d = s->x_min; p.y_min_d = s->y_min;
    p.isx_d = 1.0 / (double)p.sx;
    p.isy_d = 1.0 / (double)p.sy;
    // a bound on |x| of every cell centre and on the terms that form it in
    // float32 (x_min and (i + 1/2) dx), so that the rounding of a centre is
    // a few 2^-24 of it
    p.xmax_abs = fabs((double)s->x_min) + ((double)s->X + 1.0) * fabs((double)s->dx);
    p.ymax_abs = fabs((double)s->y_min) + ((double)s->Y + 1.0) * fabs((double)s->dy);
    p.prep_tiles_per_b = (int32_t)((XY + kPrepCells - 1) / kPrepCells);
    p.prep_cblocks = (f->C + 63) / 64;
    p.cpw = cpw;
    p.lpc = lpc;
    p.nvec = nvec;
    p.rcp_lpc = 1.0f / (float)lpc;
    p.groups_per_row = (f->W + cpw - 1) / cpw;
    // two rows per group where a group has at most two columns (measured on
    // MI355X: paper_ref 73 -> 64 us, half_batch 168 -> 150 us; with three or
    // four columns two rows were slower: rep 67 -> 76 us, z_sweep 621 -> 719)
    const int rows = cpw <= 2 ? 2 : 1;
    p.row_groups = (f->H + rows - 1) / rows;
    p.groups = (int64_t)f->B * f->N * p.row_groups * p.groups_per_row;
    p.rec_stride = kGatherRec | 1;
    p.row_bytes = (uint32_t)row;
    p.lds_wave = align16(align16((uint32_t)cpw * (uint32_t)p.rec_stride * (rows == 2 ? 12u : 8u)) +
                         kGatherTail);
    for (int k = 0; k < zb->Z; ++k) p.z[k] = zb->z[k];

    pl->prep_wgs = (gelems > 0) ? (int64_t)f->B * p.prep_tiles_per_b * p.prep_cblocks : 0;
    pl->gather_wgs = (gelems > 0) ? (p.groups + kGatherWaves - 1) / kGatherWaves : 0;
    if (pl->prep_wgs > 0x7FFFFFFFll || pl->gather_wgs > 0x7FFFFFFFll) return FLASHBEV_ERR_UNSUPPORTED;
    pl->lds = (size_t)p.lds_wave * kGatherWaves;
    if (pl->lds > kLdsBudget) return FLASHBEV_ERR_UNSUPPORTED;
    pl->lw = lw;
    pl->vpl = vpl;
    pl->rows = rows;
    return FLASHBEV_OK;
}

int launch_bwd_gather(const BwdGatherPlan &pl, hipStream_t st)
{
    void *args[] = {const_cast<BwdGatherParams *>(&pl.prm)};
    if (pl.prep_wgs > 0 &&
        hipLaunchKernel(reinterpret_cast<const void *>(sample_vt_bwd_prep),
                        dim3((unsigned)pl.prep_wgs), dim3(256), args, 0, st) != hipSuccess)
        return FLASHBEV_ERR_HIP;
    if (pl.gather_wgs > 0 &&
        hipLaunchKernel(reinterpret_cast<const void *>(pick_gather(pl.lw, pl.vpl, pl.rows)),
                        dim3((unsigned)pl.gather_wgs), dim3(kGatherWaves * kWave), args, pl.lds,
                        st) != hipSuccess)
        return FLASHBEV_ERR_HIP;
    return FLASHBEV_OK;
}

}  // namespace

// Workgroups of one forward kernel resident at once on the current device
// (occupancy of its registers and LDS times the compute units), 0 if HIP
// cannot say.  Kept per (kernel, threads, LDS, device).
int64_t resident_workgroups(const void *fn, int threads, size_t lds)
{
    struct Entry {
        const void *fn;
        int threads;
        size_t lds;
        int dev;
        int64_t resident;
    };
    static std::mutex mu;
    static Entry cache[64];
    static int used = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    std::lock_guard<std::mutex> lock(mu);
    for (int i = 0; i < used; ++i)
        if (cache[i].fn == fn && cache[i].threads == threads && cache[i].lds == lds &&
            cache[i].dev == dev)
            return cache[i].resident;
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    const int64_t r = (int64_t)per_cu * cus;
    if (used < 64) cache[used++] = Entry{fn, threads, lds, dev, r};
    return r;
}

// Launch-time choices of a forward call: contiguous bands of tiles per XCD
// for calls up to kBandsWorkMax (else stripes), and whether every workgroup
// is resident from the start, which turns on the waves' tail priorities
// (tail_prio).  Resident workgroups come from HIP's occupancy query for the
// kernel; if HIP cannot say, there are no priorities.
void forward_order(const void *fn, Plan &pl)
{
    const int64_t resident = resident_workgroups(fn, pl.threads, pl.lds);
    pl.prm.tail_prio = (resident > 0 && pl.workgroups <= resident) ? 1 : 0;
    pl.prm.bands = pl.band_work ? 1 : 0;
}

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
    case FLASHBEV_ERR_SCRATCH: return "needs more than the static scratch (FLASHBEV_SCRATCH_BYTES)";
    default: return "unknown status";
    }
}

int flashbev_launch_info(const flashbev_features *features, const flashbev_bev_grid_spec *spec,
                         const flashbev_z_bins *z_bins, int64_t *workgroups,
                         int32_t *threads_per_workgroup, int32_t *lds_bytes,
                         int32_t *cells_per_wave, int32_t *lanes_per_cell)
{
    Plan pl;
    const int rc = make_plan(features, nullptr, spec, z_bins, nullptr, false, &pl);
    if (rc) return rc;
    if (workgroups) *workgroups = pl.workgroups;
    if (threads_per_workgroup) *threads_per_workgroup = pl.threads;
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
    const int rc = make_plan(features, lidar2img, spec, z_bins, out, true, &pl);
    if (rc) return rc;
    if (pl.empty) return FLASHBEV_OK;
    const KernelFn fn = pick_kernel(features->dtype, pl.lw, pl.vpl, pl.cull_path);
    if (!fn) return FLASHBEV_ERR_UNSUPPORTED;
    forward_order(reinterpret_cast<const void *>(fn), pl);
    void *args[] = {&pl.prm};
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(fn),
                                         dim3((unsigned)pl.workgroups), dim3(pl.threads), args,
                                         pl.lds, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? FLASHBEV_OK : FLASHBEV_ERR_HIP;
}

}  // extern "C"

extern "C" int flashbev_backward_launch_info(const flashbev_features *features,
                                            const flashbev_bev_grid_spec *spec,
                                            const flashbev_z_bins *z_bins, int64_t *workgroups,
                                            int32_t *threads_per_workgroup, int32_t *lds_bytes,
                                            int32_t *rows_per_tile, int32_t *lanes_per_cell)
{
    BwdPlan pl;
    const int rc = make_bwd_plan(features, nullptr, spec, z_bins, nullptr, nullptr, false, &pl);
    if (rc) return rc;
    if (workgroups) *workgroups = pl.workgroups;
    if (threads_per_workgroup) *threads_per_workgroup = pl.threads;
    if (lds_bytes) *lds_bytes = (int32_t)pl.lds;
    if (rows_per_tile) *rows_per_tile = pl.tiled ? pl.prm.cap : 0;
    if (lanes_per_cell) *lanes_per_cell = pl.prm.lpc;
    return FLASHBEV_OK;
}

extern "C" int flashbev_sample_vt_backward(const flashbev_features *features,
                                           const float *lidar2img,
                                           const flashbev_bev_grid_spec *spec,
                                           const flashbev_z_bins *z_bins, const float *grad_out,
                                           float *grad_features, void *stream)
{
    BwdPlan pl;
    const int rc = make_bwd_plan(features, lidar2img, spec, z_bins, grad_out, grad_features, true,
                                 &pl);
    if (rc) return rc;
    if (pl.gfeat_elems == 0) return FLASHBEV_OK;
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    uint64_t blocks = (pl.gfeat_elems / 4 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    {
        // the launch's own status (hipGetLastError could report an earlier call's)
        float *dst = grad_features;
        uint64_t n = pl.gfeat_elems;
        void *fargs[] = {&dst, &n};
        if (hipLaunchKernel(reinterpret_cast<const void *>(zero_fill), dim3((unsigned)blocks),
                            dim3(256), fargs, 0, st) != hipSuccess)
            return FLASHBEV_ERR_HIP;
    }
    if (pl.workgroups == 0) return FLASHBEV_OK;
    void *args[] = {&pl.prm};
    const void *fn = reinterpret_cast<const void *>(pick_bwd(pl.kpl, pl.tiled, pl.wide));
    if (pl.lds > 65536 &&
        hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds) != hipSuccess)
        return FLASHBEV_ERR_HIP;
    const hipError_t e = hipLaunchKernel(fn,
                                         dim3((unsigned)pl.workgroups), dim3(pl.threads), args,
                                         pl.lds, st);
    return e == hipSuccess ? FLASHBEV_OK : FLASHBEV_ERR_HIP;
}

extern "C" int flashbev_backward_workspace_size(const flashbev_features *features,
                                                const flashbev_bev_grid_spec *spec,
                                                const flashbev_z_bins *z_bins, uint64_t *bytes)
{
    if (!bytes) return FLASHBEV_ERR_NULLPTR;
    BwdGatherPlan pl;
    const int rc = make_bwd_gather_plan(features, nullptr, spec, z_bins, nullptr, nullptr, nullptr,
                                        0, false, &pl);
    if (rc) return rc;
    *bytes = pl.ws_bytes;
    return FLASHBEV_OK;
}

// The no-allocation variant's workspace: a file-scope device array.  Host
// code never takes the array's name as a device address (in host code it
// names a host-side stand-in); the address on each device comes from
// hipGetSymbolAddress, once per device, and is kept.
static __device__ __align__(256) unsigned char scratch[FLASHBEV_SCRATCH_BYTES];

namespace {

constexpr int kScratchDevices = 256;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kScratchDevices];

// The scratch array's address on the current device.
int scratch_on_current_device(void **out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices)
        return FLASHBEV_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return FLASHBEV_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return FLASHBEV_OK;
}

}  // namespace

extern "C" int flashbev_sample_vt_backward_noalloc(const flashbev_features *features,
                                                   const float *lidar2img,
                                                   const flashbev_bev_grid_spec *spec,
                                                   const flashbev_z_bins *z_bins,
                                                   const float *grad_out, float *grad_features,
                                                   void *stream)
{
    // every argument check first (no HIP call), then the size limit
    BwdGatherPlan pl;
    int rc = make_bwd_gather_plan(features, lidar2img, spec, z_bins, grad_out, grad_features,
                                  nullptr, 0, true, &pl, false);
    if (rc) return rc;
    if (pl.ws_bytes > (uint64_t)FLASHBEV_SCRATCH_BYTES) return FLASHBEV_ERR_SCRATCH;
    if (pl.prep_wgs == 0 && pl.gather_wgs == 0) return FLASHBEV_OK;
    void *ws = nullptr;
    rc = scratch_on_current_device(&ws);
    if (rc) return rc;
    rc = make_bwd_gather_plan(features, lidar2img, spec, z_bins, grad_out, grad_features, ws,
                              (uint64_t)FLASHBEV_SCRATCH_BYTES, true, &pl);
    if (rc) return rc;
    return launch_bwd_gather(pl, reinterpret_cast<hipStream_t>(stream));
}

extern "C" int flashbev_sample_vt_backward_ws(const flashbev_features *features,
                                              const float *lidar2img,
                                              const flashbev_bev_grid_spec *spec,
                                              const flashbev_z_bins *z_bins,
                                              const float *grad_out, float *grad_features,
                                              void *workspace, uint64_t workspace_bytes,
                                              void *stream)
{
    BwdGatherPlan pl;
    const int rc = make_bwd_gather_plan(features, lidar2img, spec, z_bins, grad_out, grad_features,
                                        workspace, workspace_bytes, true, &pl);
    if (rc) return rc;
    return launch_bwd_gather(pl, reinterpret_cast<hipStream_t>(stream));
}

#ifdef FLASHBEV_PHASE_CLOCK
// Instrumented builds only: where the forward's wavefronts write their phase
// clocks (NULL: nowhere).  Returns 0, or -1 if the copy to the device
// variable fails.
extern "C" int flashbev_phase_log(void *log)
{
    return hipMemcpyToSymbol(HIP_SYMBOL(phase_log), &log, sizeof(log)) == hipSuccess ? 0 : -1;
}
#endif
