// FlashSCA for gfx950: BEVFormer's spatial cross-attention with the
// per-camera sampling points formed on the fly (FlashBEV paper, Sec. 4.5,
// Table 7), forward and backward, behind the C ABI declared in
// include/flashsca.h.
//
// Execution design (MI355X-first):
//   * Work items are (query, head) pairs, "slots".  A slot owns `lph` lanes
//     (a power of two); lane `sub` of a slot holds one LW-byte slice of the
//     head's D channels, so every bilinear tap of the head is one coalesced
//     run of D * elem bytes across the slot's lanes.  A wavefront holds
//     64 / lph slots.  Queries are visited in blocks (query_of, Z order
//     inside a block).  A forward tile holds consecutive (query, head)
//     pairs of one batch element (the heads of a few queries); a backward
//     tile holds waves * spw consecutive queries of one head.
//   * Phase 1 (workgroup): every (query, camera) pair of the tile projects the
//     query's Z anchors (float32 recipe, IEEE divisions), records the
//     normalized reference points in LDS and sets the camera's bit in the
//     query's hit mask and in the tile's union (LDS atomic OR).
//   * Phase 2 (slot): softmax over the head's L * P logits, read once per
//     query (not once per camera): the forward keeps the weights in LDS, the
//     backward keeps the maximum and 1 / sum and recomputes a weight where
//     it needs one.
//   * Phase 3 (slot): in chunks of lph points, per hit camera, lane `sub`
//     sets up point c + sub (anchor k mod Z, location (u W_l + dx) - 1/2,
//     floor, four tap offsets and bilinear weights) and publishes it in LDS;
//     then all lanes of the slot load the chunk's lph * 4 taps with raw buffer
//     loads.  A tap outside the map is not loaded.
//       - forward (cameras outside, chunks inside): each lane accumulates its
//         channels in float32;
//       - backward (chunks outside, cameras inside, uniform over the
//         workgroup): each lane forms its channels' share of the tap rows'
//         dot products with the output gradient; a reduction across the slot
//         gives the point's gradients of attention weight and location, kept
//         in registers by the lane that owns the point.  For the value
//         gradient the workgroup merges the chunk's rows in an LDS table by
//         tap offset (all slots share the head, so equal offsets are the same
//         value-gradient row), sums each key's members and scatters one
//         float atomic add per distinct row and channel.
//   * Forward: each output element is written once, no atomics on global
//     memory, no workspace, one launch.  Backward: a fill kernel zeroes the
//     value gradient, then one launch; every offset and logit gradient is
//     written (the logit gradient holds d a_j until the slot's softmax
//     backward finishes it).
// Coordinates follow the float32 recipe of the conventions in flashsca.h, so
// mask and floor decisions match the CPU oracle bit for bit: the file is
// compiled with -ffp-contract=off and uses IEEE division.
#include <hip/hip_runtime.h>

#include <math.h>
#include <algorithm>
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
// The backward takes tiles of up to 8 wavefronts (64 queries of a head at
// D = 32 float32: an 8 x 8 patch of the visiting order, whose taps share
// more pixels in the row merge) within a larger LDS budget (measured on
// MI355X at BEVFormer-base: P = 8 1.52 -> 1.48 ms, P = 32 4.77 -> 4.64 ms).
constexpr int kScaBwdWavesMax = 8;
constexpr int kScaBwdThreads = kScaWave * kScaBwdWavesMax;
constexpr uint32_t kScaBwdLdsBudget = 80u * 1024u;
constexpr int kScaXcds = 8;      // MI355X: workgroups are dispatched to 8 XCDs round-robin
constexpr int kScaBlock = 16;    // queries are visited in blocks of 16 x 16 BEV cells
constexpr int kScaHeadChunks = 8;   // head-to-XCD order: chunks of the query groups
constexpr int kScaOrdMax = 256;     // blocks of a grid visited in azimuth order, at most
// Offset of a tap that is not loaded: one camera's value is smaller than
// 2 GiB and a lane adds less than 1 KiB, so the load is past the buffer's end
// and returns zero without touching memory.
constexpr uint32_t kScaNoTap = 0x80000000u;
constexpr uint64_t kScaCamBytesMax = 0x7FFFFFFFull;
constexpr uint32_t kScaLdsBudget = 64u * 1024u;    // preferred dynamic LDS per workgroup
constexpr uint32_t kScaLdsMax = 160u * 1024u;      // gfx950's LDS per workgroup
// A chunk record per lane: 4 tap offsets and 4 weights (forward); 4 tap
// offsets, the location's fractions and the point's scatter factor (mean *
// a_j) in the backward, whose readers recompute the weights from the
// fractions (8 dwords each).  A 4-dword pad per slot puts the slots'
// broadcast reads in different banks.
constexpr int kRecFwd = 8;
constexpr int kRecBwd = 8;
constexpr int kSlotPad = 4;
// Backward row merge, per workgroup: a chunk has lph * spw * 4 = 256 (point,
// slot, tap) rows per wavefront.  Per wavefront's 256 rows: an open-addressing
// table of keys (tap offsets) with the head of each key's member list, and per
// row its factor (mean * a * w) and a link word (offset of its slot's
// output-gradient row << 16 | next member) side by side, read as one 8-byte
// word; the keys in use (halfwords) and their number.
constexpr int kMrgRows = 4 * kScaWave;
constexpr int kMrgWaveBytes = kMrgRows * 18;
constexpr uint32_t kMrgEmpty = 0xFFFFFFFFu;   // no key (tap offsets are below 2^31)
constexpr uint32_t kMrgEnd = 0xFFFFFFFFu;     // end of a member list
constexpr uint32_t kMrgEnd16 = 0xFFFFu;       // the same, as a stored link

struct ScaParams {
    const void *value;
    const float *l2i;
    const float *offsets;
    const float *logits;
    float *out;              // forward output
    const float *grad_out;   // backward: dL/d out
    float *grad_value;       // backward outputs (each may be null)
    float *grad_offsets;
    float *grad_logits;
    uint64_t cam_bytes;      // bytes of one camera's value maps (S C elem)
    uint64_t cam_elems;      // S C
    uint32_t row_bytes;      // C * elem
    uint32_t head_bytes;     // D * elem
    int32_t B, N, C, heads, D, L, P, Z, LP;
    int32_t X, Y, Q;
    int32_t lph;             // lanes per slot (power of two)
    int32_t lph_shift;       // log2(lph)
    int32_t spw;             // slots per wavefront
    int32_t tile_pairs;      // slots per workgroup: queries of one head
    int32_t head_xcd;        // head-to-XCD order: its chunks of the query groups (0: bands)
    int32_t mrg_shift;       // backward: 32 - log2(rows of the merge table)
    int32_t tiles_per_b;
    int32_t stripe;          // consecutive tiles an XCD takes in turn (about one block)
    int32_t nq_max;          // queries a tile can touch
    int32_t slot_stride;     // dwords per slot in the chunk-record area
    float img_w, img_h;
    float x_min, dx, y_min, dy, depth_eps;
    int32_t reduce;
    float rcp_p, rcp_z;      // float32 1 / P and 1 / Z for div_small
    float level_wf[FLASHSCA_LMAX], level_hf[FLASHSCA_LMAX];
    int32_t level_w[FLASHSCA_LMAX], level_h[FLASHSCA_LMAX];
    uint32_t level_start[FLASHSCA_LMAX];   // first pixel of each level
    // LDS layout (byte offsets)
    uint32_t lds_mat, lds_lvl, lds_z, lds_ref, lds_hit, lds_att, lds_gst, lds_tap;
    uint32_t lds_mrg;
    float rcp_d;             // float32 1 / D for div_small
    float z[FLASHSCA_ZMAX];
    // azimuth order of the query blocks (sca_tile; ord_blocks = 0: rank order):
    // the sorted blocks' first query groups and the query groups before each
    // (ord_cum[ord_blocks] = query groups per batch element)
    int32_t ord_blocks;
    uint16_t ord_first[kScaOrdMax];
    uint16_t ord_cum[kScaOrdMax + 1];
};

// LDS: camera matrices [N][12]; level table [5][LMAX]; anchors [Z];
// reference points [nq_max][N][Z] float2; hit masks [nq_max] and their union;
// forward only:
// attention weights [waves][spw][LP]; backward only: output-gradient rows
// [waves][spw][D]; chunk records [waves][spw][slot_stride]; backward only:
// the row-merge table (keys, list heads, row factors, row links
// [waves * 256] dwords; keys in use [waves * 256] halfwords; a counter).
struct ScaLds {
    uint32_t mat, lvl, z, ref, hit, att, gst, tap, mrg, total;
};

__host__ inline uint32_t sca_align16(uint32_t v) { return (v + 15u) & ~15u; }

__host__ ScaLds sca_lds_layout(int N, int Z, int nq_max, int waves, int spw, int LP, int D,
                               int slot_stride, bool backward)
{
    ScaLds s;
    uint32_t o = 0;
    s.mat = o; o = sca_align16(o + (uint32_t)N * 12u * 4u);
    s.lvl = o; o = sca_align16(o + 5u * FLASHSCA_LMAX * 4u);
    s.z = o; o = sca_align16(o + (uint32_t)Z * 4u);
    s.ref = o; o = sca_align16(o + (uint32_t)nq_max * N * Z * 8u);
    s.hit = o; o = sca_align16(o + (uint32_t)(nq_max + 1) * 4u);
    s.att = o; o = sca_align16(o + (backward ? 0u : (uint32_t)waves * spw * LP * 4u));
    s.gst = o; o = sca_align16(o + (backward ? (uint32_t)waves * spw * D * 4u : 0u));
    s.tap = o; o = sca_align16(o + (uint32_t)waves * spw * slot_stride * 4u);
    s.mrg = o; o = sca_align16(o + (backward ? (uint32_t)waves * kMrgWaveBytes + 16u : 0u));
    s.total = o;
    return s;
}

// Cell (i, j) of the query of rank r in the blocked visiting order: the grid
// is cut into bands of kScaBlock rows; a band into blocks of kScaBlock
// columns (the last band and block may be narrower); blocks follow each other
// along the band.  A full block's cells are in Z order (rank bits alternate
// column, row, column, ...), so that 2^k consecutive ranks form a 2 x 2,
// 2 x 4, 4 x 4, ... patch whose samples share pixels (against row-major
// blocks, measured on MI355X at BEVFormer-base: forward P = 8 0.270 ->
// 0.264 ms, P = 32 0.900 -> 0.881 ms; the backward's row merge 1.83x ->
// 2.05x fewer rows per 8 queries); a partial block's cells are row-major.  A
// bijection of [0, X Y) onto the cells.
__device__ __forceinline__ void query_of(int r, int X, int Y, int &i, int &j)
{
    const int band_cells = kScaBlock * Y;
    const int R = r / band_cells;
    const int s = r - R * band_cells;
    const int h = min(kScaBlock, X - R * kScaBlock);
    const int c = s / (h * kScaBlock);
    const int t = s - c * h * kScaBlock;
    const int w = min(kScaBlock, Y - c * kScaBlock);
    if (h == kScaBlock && w == kScaBlock) {
        const uint32_t u = (uint32_t)t;
        i = R * kScaBlock + (int)(((u >> 1) & 1u) | ((u >> 2) & 2u) | ((u >> 3) & 4u) | ((u >> 4) & 8u));
        j = c * kScaBlock + (int)((u & 1u) | ((u >> 1) & 2u) | ((u >> 2) & 4u) | ((u >> 3) & 8u));
        return;
    }
    const int ti = t / w;
    i = R * kScaBlock + ti;
    j = c * kScaBlock + (t - ti * w);
}

// LDS views of one workgroup.
struct ScaSmem {
    float *mat, *lwf, *lhf, *z, *att, *gst;
    int32_t *lw, *lh;
    uint32_t *lst, *hit, *tap, *mrg;
    float2 *ref;
};

__device__ __forceinline__ ScaSmem sca_smem(const ScaParams &p, unsigned char *smem)
{
    ScaSmem m;
    m.mat = reinterpret_cast<float *>(smem + p.lds_mat);
    m.lwf = reinterpret_cast<float *>(smem + p.lds_lvl);
    m.lhf = m.lwf + FLASHSCA_LMAX;
    m.lw = reinterpret_cast<int32_t *>(m.lhf + FLASHSCA_LMAX);
    m.lh = m.lw + FLASHSCA_LMAX;
    m.lst = reinterpret_cast<uint32_t *>(m.lh + FLASHSCA_LMAX);
    m.z = reinterpret_cast<float *>(smem + p.lds_z);
    m.ref = reinterpret_cast<float2 *>(smem + p.lds_ref);
    m.hit = reinterpret_cast<uint32_t *>(smem + p.lds_hit);
    m.att = reinterpret_cast<float *>(smem + p.lds_att);
    m.gst = reinterpret_cast<float *>(smem + p.lds_gst);
    m.tap = reinterpret_cast<uint32_t *>(smem + p.lds_tap);
    m.mrg = reinterpret_cast<uint32_t *>(smem + p.lds_mrg);
    return m;
}

// XCD-aware tile order.  A tile holds waves * spw consecutive queries (ranks
// of query_of) of one head.  Queries are visited block by block (query_of),
// so consecutive tiles cover a compact patch of the BEV whose samples land
// on overlapping pixels (measured on MI355X at BEVFormer-base, P = 32:
// 16 x 16 blocks 0.927 ms, 32 x 32 0.953 ms, 64 x 64 slower still).
// Workgroups go to the 8 XCDs round-robin, and the k-th workgroup on XCD x
// takes:
//  * with heads a multiple of 8 (p.head_xcd = K chunks): batch element b,
//    head group hh and query group qg, k running over (b, hh, qg) with qg
//    fastest, and head 8 hh + (x + c) mod 8 on the c-th of K equal chunks of
//    the query groups.  At any time each XCD then reads a single head's
//    slice of the value rows (whole 128-byte lines for float32 D = 32), so
//    its L2 holds the rows of 8 times as many queries as when every XCD
//    reads every head, and over the K chunks every XCD takes every head once,
//    which evens out heads whose points fall outside the maps more often
//    (measured on MI355X at BEVFormer-base, forward, against the band order
//    below: P = 8 0.258 -> 0.254 ms, P = 32 0.784 -> 0.765 ms with fabric
//    fetches 2.10 -> 1.14 GB; one head per XCD throughout (K = 1) fetched
//    1.09 GB but took 0.784 ms, its XCDs unequally loaded by up to 17%);
//  * otherwise tile (k / S) * 8S + x * S + k % S with S = p.stripe, one
//    eighth of the tiles (query groups major, heads minor): each XCD works
//    through one contiguous band of blocks, whose samples come from few
//    cameras and share pixels in its L2 (against stripes of one block
//    interleaved over the grid: P = 8 0.282 -> 0.268 ms, P = 32 0.927 ->
//    0.900 ms, bfloat16 0.487 -> 0.467 ms, backward 4.37 -> 4.31 ms).  The
//    few tiles past 8 S are split the same way with shorter stripes.
struct ScaTile {
    int b, head, qg;
};

// Query group at position pos of the azimuth order: the sorted block holding
// pos (ord_cum[lo] <= pos < ord_cum[lo + 1]), then pos's place in it.
__device__ __forceinline__ int sca_ordered_qg(const ScaParams &p, int pos)
{
    int lo = 0, hi = p.ord_blocks;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if ((int)p.ord_cum[mid] <= pos) lo = mid;
        else hi = mid;
    }
    return (int)p.ord_first[lo] + (pos - (int)p.ord_cum[lo]);
}

__device__ __forceinline__ ScaTile sca_tile(const ScaParams &p)
{
    const int g = blockIdx.x;
    const int nqg = p.tiles_per_b / p.heads;   // query groups per batch element
    ScaTile t;
    if (p.head_xcd) {
        const int x = g % kScaXcds, k = g / kScaXcds;
        const int per_b = (p.heads / kScaXcds) * nqg;
        t.b = k / per_b;
        const int r = k - t.b * per_b;
        const int hh = r / nqg;
        t.qg = r - hh * nqg;
        const int c = (int)(((int64_t)t.qg * p.head_xcd) / nqg);
        t.head = hh * kScaXcds + ((x + c) & (kScaXcds - 1));
        if (p.ord_blocks) t.qg = sca_ordered_qg(p, t.qg);
        return t;
    }
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
    t.b = tile / p.tiles_per_b;
    const int tb = tile - t.b * p.tiles_per_b;
    t.qg = tb / p.heads;
    t.head = tb - t.qg * p.heads;
    if (p.ord_blocks) t.qg = sca_ordered_qg(p, t.qg);
    return t;
}

// Stage matrices, level table and anchors; phase 1: reference points and
// hit masks of the tile's queries and their union.  Ends with a workgroup
// barrier.
__device__ __forceinline__ void sca_project_tile(const ScaParams &p, const ScaSmem &m, int b,
                                                 int r_first)
{
    const int tid = threadIdx.x;
    const int nthreads = blockDim.x;
    const int N = p.N, Z = p.Z;
    for (int t = tid; t < N * 12; t += nthreads) {
        const int n = t / 12, r = t - n * 12;
        m.mat[t] = p.l2i[((size_t)b * N + n) * 16 + r];
    }
    if (tid < FLASHSCA_LMAX) {
        m.lwf[tid] = p.level_wf[tid];
        m.lhf[tid] = p.level_hf[tid];
        m.lw[tid] = p.level_w[tid];
        m.lh[tid] = p.level_h[tid];
        m.lst[tid] = p.level_start[tid];
    }
    for (int t = tid; t < Z; t += nthreads) m.z[t] = p.z[t];
    for (int t = tid; t <= p.nq_max; t += nthreads) m.hit[t] = 0u;
    __syncthreads();

    for (int t = tid; t < p.nq_max * N; t += nthreads) {
        const int qi = t / N, n = t - qi * N;
        const int rank = r_first + qi;
        if (rank >= p.Q) continue;
        int i, j;
        query_of(rank, p.X, p.Y, i, j);
        const float x = p.x_min + ((float)i + 0.5f) * p.dx;
        const float y = p.y_min + ((float)j + 0.5f) * p.dy;
        const float *mr = m.mat + n * 12;
        bool any = false;
        for (int k = 0; k < Z; ++k) {
            const float z = m.z[k];
            // (u', v', d) = P[b,n] (x, y, z, 1), left to right, no contraction
            const float up = ((mr[0] * x + mr[1] * y) + mr[2] * z) + mr[3];
            const float vp = ((mr[4] * x + mr[5] * y) + mr[6] * z) + mr[7];
            const float d = ((mr[8] * x + mr[9] * y) + mr[10] * z) + mr[11];
            const bool in_front = d > p.depth_eps;
            const float dd = in_front ? d : p.depth_eps;
            const float un = (up / dd) / p.img_w;
            const float vn = (vp / dd) / p.img_h;
            m.ref[(qi * N + n) * Z + k] = make_float2(un, vn);
            any |= in_front && un > 0.0f && un < 1.0f && vn > 0.0f && vn < 1.0f;
        }
        if (any) {
            atomicOr(&m.hit[qi], 1u << n);
            atomicOr(&m.hit[p.nq_max], 1u << n);   // the tile's cameras
        }
    }
    __syncthreads();
}

// One (query, head) slot of a wavefront.
struct ScaSlot {
    int sub, slot;        // lane within the slot, slot within the wavefront
    bool active;          // the slot holds a (query, head) pair
    int qi;               // query index within the tile
    int q;                // the query's index in offsets, logits and the outputs
    int mh;               // head
    uint32_t hits;        // hit cameras (0 for inactive slots)
    float inv;            // 1 / max(1, hits) (1 in sum mode)
    size_t pt0;           // first (level, point) element of the pair
};

// A slot of a tile.  A tile holds waves * spw consecutive queries (ranks
// r_first ..., in the Z order of query_of) of one head, slot s of wavefront w
// being query r_first + w spw + s.  All slots of the tile then share their
// head and cover a compact patch of cells: in the backward their taps on one
// pixel are the same value-gradient row and are merged before the scatter
// (BEVFormer-base, P = 8, per chunk of 8 points: 1.83x fewer rows for 1 x 8
// strips of queries, 2.05x for 2 x 4 patches, 2.85x for 4 x 4, 3.85x for
// 4 x 8).
__device__ __forceinline__ ScaSlot sca_slot(const ScaParams &p, const ScaSmem &m, int b,
                                                int r_first, int head, int wave, int lane)
{
    ScaSlot s;
    s.sub = lane & (p.lph - 1);
    s.slot = lane >> p.lph_shift;
    const int qi = wave * p.spw + s.slot;
    const int rank = r_first + qi;
    s.active = rank < p.Q;
    s.mh = head;
    s.qi = s.active ? qi : 0;
    int qx, qy;
    query_of(s.active ? rank : r_first, p.X, p.Y, qx, qy);
    s.q = qx * p.Y + qy;
    s.hits = s.active ? m.hit[s.qi] : 0u;
    const int count = __popc(s.hits);
    s.inv = (p.reduce == FLASHBEV_REDUCE_VALID_MEAN && count > 1) ? 1.0f / (float)count : 1.0f;
    s.pt0 = (((size_t)b * p.Q + s.q) * p.heads + s.mh) * (size_t)p.LP;
    return s;
}

// Phase 2: att[j] = post * softmax over the slot's L*P logits (only for
// slots with a hit camera).  The shuffles stay inside the slot, whose lanes
// all take the branch or none.
__device__ __forceinline__ void sca_softmax(const ScaParams &p, const ScaSlot &s, float *att,
                                            float post)
{
    if (!s.hits) return;
    const int lph = p.lph, LP = p.LP;
    float mx = -INFINITY;
    for (int j = s.sub; j < LP; j += lph) mx = fmaxf(mx, p.logits[s.pt0 + j]);
    for (int o = lph >> 1; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    float sum = 0.0f;
    for (int j = s.sub; j < LP; j += lph) {
        const float e = expf(p.logits[s.pt0 + j] - mx);
        att[j] = e;
        sum += e;
    }
    for (int o = lph >> 1; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
    const float r = post / sum;
    for (int j = s.sub; j < LP; j += lph) att[j] *= r;
}

// The same softmax's maximum and 1 / sum, for weights recomputed on the fly
// as expf(logit - mx) * rcp (the values sca_softmax stores with post = 1).
__device__ __forceinline__ void sca_softmax_stats(const ScaParams &p, const ScaSlot &s, float &mx,
                                                  float &rcp)
{
    mx = 0.0f;
    rcp = 0.0f;
    if (!s.hits) return;
    const int lph = p.lph, LP = p.LP;
    float m = -INFINITY;
    for (int j = s.sub; j < LP; j += lph) m = fmaxf(m, p.logits[s.pt0 + j]);
    for (int o = lph >> 1; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    float sum = 0.0f;
    for (int j = s.sub; j < LP; j += lph) sum += expf(p.logits[s.pt0 + j] - m);
    for (int o = lph >> 1; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
    mx = m;
    rcp = 1.0f / sum;
}

// Set-up of point j of a slot in one camera: tap byte offsets (kScaNoTap
// outside the map) and the location's fractions.  Returns false when no
// corner lies inside the map (all taps kScaNoTap).
__device__ __forceinline__ bool sca_setup_point(const ScaParams &p, const ScaSmem &m,
                                                const float2 *ref, const ScaSlot &s, int j,
                                                uint32_t head_off, uint4 &o, float &ax,
                                                float &ay)
{
    o = make_uint4(kScaNoTap, kScaNoTap, kScaNoTap, kScaNoTap);
    ax = 0.0f;
    ay = 0.0f;
    const int l = div_small(j, p.P, p.rcp_p);
    const int k = j - l * p.P;
    const int zk = k - div_small(k, p.Z, p.rcp_z) * p.Z;   // anchor k mod Z
    const float2 r = ref[zk];
    const float2 dxy = reinterpret_cast<const float2 *>(p.offsets)[s.pt0 + j];
    const float Wl = m.lwf[l], Hl = m.lhf[l];
    float sx = r.x * Wl;
    float sy = r.y * Hl;
    sx = sx + dxy.x;
    sy = sy + dxy.y;
    const float xim = sx - 0.5f;
    const float yim = sy - 0.5f;
    if (!(xim > -1.0f && xim < Wl && yim > -1.0f && yim < Hl)) return false;
    const float x0f = floorf(xim), y0f = floorf(yim);
    ax = xim - x0f;
    ay = yim - y0f;
    const int x0 = (int)x0f, y0 = (int)y0f;
    const int wi = m.lw[l], hi = m.lh[l];
    const bool xl = x0 >= 0, xr = x0 + 1 < wi;
    const bool yt = y0 >= 0, yb = y0 + 1 < hi;
    const int row = (int)m.lst[l] + y0 * wi + x0;
    const uint32_t rb = p.row_bytes;
    if (xl && yt) o.x = (uint32_t)row * rb + head_off;
    if (xr && yt) o.y = (uint32_t)(row + 1) * rb + head_off;
    if (xl && yb) o.z = (uint32_t)(row + wi) * rb + head_off;
    if (xr && yb) o.w = (uint32_t)(row + wi + 1) * rb + head_off;
    return true;
}

// bilinear weights of the in-range taps, each times `a`
__device__ __forceinline__ float4 sca_weights(const uint4 &o, float ax, float ay, float a)
{
    const float wt = a * (1.0f - ay), wb = a * ay;
    return make_float4((o.x != kScaNoTap) ? wt * (1.0f - ax) : 0.0f,
                       (o.y != kScaNoTap) ? wt * ax : 0.0f,
                       (o.z != kScaNoTap) ? wb * (1.0f - ax) : 0.0f,
                       (o.w != kScaNoTap) ? wb * ax : 0.0f);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t sca_camera_rsrc(const ScaParams &p, int b, int n)
{
    const char *cam_base = static_cast<const char *>(p.value) +
                           ((size_t)b * p.N + n) * (size_t)p.cam_bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(cam_base), (short)0,
                                             (int)p.cam_bytes, 0x00020000);
}

// uniform over the wavefront: the cameras any slot of it hits
__device__ __forceinline__ uint32_t sca_wave_cameras(const ScaParams &p, uint32_t hits)
{
    uint32_t cams = 0;
    for (int n = 0; n < p.N; ++n)
        if (__ballot((hits >> n) & 1u)) cams |= 1u << n;
    return cams;
}

template <int DT, int LW>
__global__ void __launch_bounds__(kScaThreads)
sca_fwd(const ScaParams p)
{
    constexpr int ES = ElemSize<DT>::value;
    constexpr int EPV = LW / ES;   // elements per lane slice
    extern __shared__ __align__(16) unsigned char smem[];
    const ScaSmem m = sca_smem(p, smem);
    const int wave = threadIdx.x / kScaWave;
    const int lane = threadIdx.x % kScaWave;

    const ScaTile tl = sca_tile(p);
    const int b = tl.b;
    const int r_first = tl.qg * p.tile_pairs;   // first query rank of the tile
    sca_project_tile(p, m, b, r_first);

    const ScaSlot s = sca_slot(p, m, b, r_first, tl.head, wave, lane);
    const int lph = p.lph, LP = p.LP;
    float *att = m.att + (size_t)(wave * p.spw + s.slot) * LP;
    // attention weights with the mean over hit cameras folded in
    sca_softmax(p, s, att, s.inv);
    const uint32_t cams = sca_wave_cameras(p, s.hits);

    float acc[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) acc[e] = 0.0f;
    const uint32_t lane_off = (uint32_t)s.sub * LW;
    const uint32_t head_off = (uint32_t)s.mh * p.head_bytes;
    uint32_t *rec = m.tap + (size_t)(wave * p.spw + s.slot) * p.slot_stride;   // this slot

    for (int n = 0; n < p.N; ++n) {
        if (!((cams >> n) & 1u)) continue;
        const bool mine = (s.hits >> n) & 1u;
        const __amdgpu_buffer_rsrc_t rsrc = sca_camera_rsrc(p, b, n);
        const float2 *ref = m.ref + (size_t)(s.qi * p.N + n) * p.Z;
        for (int c0 = 0; c0 < LP; c0 += lph) {
            // set-up of point j = c0 + sub of this slot, weights a * w
            const int j = c0 + s.sub;
            uint4 o = make_uint4(kScaNoTap, kScaNoTap, kScaNoTap, kScaNoTap);
            float4 w = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (mine && j < LP) {
                float ax, ay;
                if (sca_setup_point(p, m, ref, s, j, head_off, o, ax, ay))
                    w = sca_weights(o, ax, ay, att[j]);
            }
            uint32_t *mine_rec = rec + s.sub * kRecFwd;
            *reinterpret_cast<uint4 *>(mine_rec) = o;
            *reinterpret_cast<float4 *>(mine_rec + 4) = w;
            wave_lds_sync();
            // gather the chunk's points: every lane of the slot, its channels
            const int npts = (LP - c0) < lph ? (LP - c0) : lph;
#pragma unroll 4
            for (int t = 0; t < npts; ++t) {
                const uint4 to = *reinterpret_cast<const uint4 *>(rec + t * kRecFwd);
                const float4 tw = *reinterpret_cast<const float4 *>(rec + t * kRecFwd + 4);
                // taps outside the map are not loaded (their lanes sit out the
                // load; measured on MI355X at BEVFormer-base P = 32, where 41%
                // of the taps fall outside: 1.005 -> 0.953 ms)
                Raw<LW> v0{}, v1{}, v2{}, v3{};
                if (to.x != kScaNoTap) v0 = load_vec<LW>(rsrc, to.x + lane_off, 0);
                if (to.y != kScaNoTap) v1 = load_vec<LW>(rsrc, to.y + lane_off, 0);
                if (to.z != kScaNoTap) v2 = load_vec<LW>(rsrc, to.z + lane_off, 0);
                if (to.w != kScaNoTap) v3 = load_vec<LW>(rsrc, to.w + lane_off, 0);
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    float a = acc[e];
                    a = fmaf(tw.x, elem<DT, LW>(v0, e), a);
                    a = fmaf(tw.y, elem<DT, LW>(v1, e), a);
                    a = fmaf(tw.z, elem<DT, LW>(v2, e), a);
                    a = fmaf(tw.w, elem<DT, LW>(v3, e), a);
                    acc[e] = a;
                }
            }
            wave_lds_sync();
        }
    }

    // ---- store: each lane its slice of the head's channels
    if (s.active) {
        float *out = p.out + ((size_t)b * p.Q + s.q) * (size_t)p.C + (size_t)s.mh * p.D;
        const int e0 = s.sub * EPV;
#pragma unroll
        for (int e = 0; e < EPV; ++e)
            if (e0 + e < p.D) out[e0 + e] = acc[e];
    }
}

// Phase clock of the backward, compiled in only with FLASHBEV_PHASE_CLOCK
// (the instrumented library libflashbev_phases.so; the operator's library
// has none of it).  Lane 0 of each wavefront sums the real-time counter
// (100 MHz) over the kernel's steps and writes the sums at its end to
// sca_phase_log[(workgroup * waves + wave) * kScaPhaseSlots + slot].
#ifdef FLASHBEV_PHASE_CLOCK
__device__ unsigned long long *sca_phase_log;
constexpr int kScaPhaseSlots = 16;
enum ScaPhaseSlot {
    kSpStart = 0, kSpProject = 1, kSpSetup = 2, kSpRecords = 3, kSpPoint = 4, kSpInsert = 5,
    kSpInsertBarrier = 6, kSpWalk = 7, kSpWalkBarrier = 8, kSpClear = 9, kSpSteps = 10,
    kSpKeys = 11, kSpTail = 12, kSpEnd = 13
};
#define SPH_DECL                                                             \
    unsigned long long sph_t = __builtin_amdgcn_s_memrealtime();             \
    unsigned long long sph[kScaPhaseSlots] = {};                             \
    sph[kSpStart] = sph_t
#define SPH_ADD(slot)                                                        \
    do {                                                                     \
        const unsigned long long sph_n = __builtin_amdgcn_s_memrealtime();   \
        sph[slot] += sph_n - sph_t;                                          \
        sph_t = sph_n;                                                       \
    } while (0)
#define SPH_COUNT(slot, v) (sph[slot] += (unsigned long long)(v))
#define SPH_WRITE(lane)                                                      \
    do {                                                                     \
        if (sca_phase_log && (lane) == 0) {                                  \
            sph[kSpEnd] = __builtin_amdgcn_s_memrealtime();                  \
            unsigned long long *sph_o = sca_phase_log +                      \
                ((size_t)blockIdx.x * (blockDim.x / kScaWave) + threadIdx.x / kScaWave) * \
                    kScaPhaseSlots;                                          \
            for (int k = 0; k < kScaPhaseSlots; ++k) sph_o[k] = sph[k];      \
        }                                                                    \
    } while (0)
#else
#define SPH_DECL
#define SPH_ADD(slot) ((void)0)
#define SPH_COUNT(slot, v) ((void)0)
#define SPH_WRITE(lane) ((void)0)
#endif

// Backward: gradients of value (scatter), offsets and logits.
template <int DT, int LW>
__global__ void __launch_bounds__(kScaBwdThreads)
sca_bwd(const ScaParams p)
{
    constexpr int ES = ElemSize<DT>::value;
    constexpr int EPV = LW / ES;
    extern __shared__ __align__(16) unsigned char smem[];
    const ScaSmem m = sca_smem(p, smem);
    const int wave = threadIdx.x / kScaWave;
    const int lane = threadIdx.x % kScaWave;
    const int tid = threadIdx.x;
    const int nthreads = blockDim.x;

    SPH_DECL;
    const ScaTile tl = sca_tile(p);
    const int b = tl.b;
    const int r_first = tl.qg * p.tile_pairs;   // first query rank of the tile
    sca_project_tile(p, m, b, r_first);
    SPH_ADD(kSpProject);

    const ScaSlot s = sca_slot(p, m, b, r_first, tl.head, wave, lane);
    const int lph = p.lph, LP = p.LP;
    const int slot_id = wave * p.spw + s.slot;
    // softmax a_j = expf(logit_j - mx) * rcp, recomputed where needed
    float mx, rcp;
    sca_softmax_stats(p, s, mx, rcp);
    // uniform over the workgroup: the cameras any of its queries hits
    const uint32_t cams = m.hit[p.nq_max];

    // this lane's slice of the output gradient
    const int e0 = s.sub * EPV;
    float gs[EPV];
#pragma unroll
    for (int e = 0; e < EPV; ++e) {
        gs[e] = (s.hits && e0 + e < p.D)
                    ? p.grad_out[((size_t)b * p.Q + s.q) * (size_t)p.C + (size_t)s.mh * p.D + e0 + e]
                    : 0.0f;
    }
    const uint32_t lane_off = (uint32_t)s.sub * LW;
    const uint32_t head_off = (uint32_t)s.mh * p.head_bytes;
    uint32_t *rec = m.tap + (size_t)slot_id * p.slot_stride;
    // the slots' output-gradient rows, for the value scatter
    const int D = p.D;
#pragma unroll
    for (int e = 0; e < EPV; ++e)
        if (e0 + e < D) m.gst[slot_id * D + e0 + e] = gs[e];
    const int spw_shift = __builtin_ctz((unsigned)p.spw);
    // the workgroup's row-merge table: row R = wavefront * 256 + (t spw + slot) 4 + tap
    const int trows = (nthreads / kScaWave) * kMrgRows;
    uint32_t *tkey = m.mrg;
    uint32_t *thead = tkey + trows;
    uint2 *rrow = reinterpret_cast<uint2 *>(thead + trows);   // (factor bits, link) per row
    uint16_t *tuniq = reinterpret_cast<uint16_t *>(rrow + trows);
    uint32_t *tcount = reinterpret_cast<uint32_t *>(tuniq + trows);
    for (int h = tid; h < trows; h += nthreads) {
        tkey[h] = kMrgEmpty;
        thead[h] = kMrgEnd;
    }
    if (tid == 0) *tcount = 0u;
    // the walk's first element (u0, ch0) and step (du, dch) in (row, channel)
    const int u0 = div_small(tid, D, p.rcp_d), ch0 = tid - u0 * D;
    const int du = div_small(nthreads, D, p.rcp_d), dch = nthreads - du * D;
    __syncthreads();
    SPH_ADD(kSpSetup);

    // Chunks of lph points (lane sub owns point c0 + sub), each over the
    // cameras the tile's queries hit.  The owner keeps its point's gradients
    // in registers across the cameras, so no per-point state stays in LDS.
    // Both loops are uniform over the workgroup (its barriers need that).
    float dot = 0.0f;   // sum of a_j d a_j over this lane's points
    for (int c0 = 0; c0 < LP; c0 += lph) {
        const int j = c0 + s.sub;
        const bool own = s.hits && j < LP;
        const float a_j = own ? expf(p.logits[s.pt0 + j] - mx) * rcp : 0.0f;
        const int npts = (LP - c0) < lph ? (LP - c0) : lph;
        float g_da = 0.0f, g_dx = 0.0f, g_dy = 0.0f;   // before the mean (and a_j for x, y)
        for (int n = 0; n < p.N; ++n) {
            if (!((cams >> n) & 1u)) continue;
            const bool mine = own && ((s.hits >> n) & 1u);
            const __amdgpu_buffer_rsrc_t rsrc = sca_camera_rsrc(p, b, n);
            const float2 *ref = m.ref + (size_t)(s.qi * p.N + n) * p.Z;
            float *gv = p.grad_value ? p.grad_value + ((size_t)b * p.N + n) * p.cam_elems : nullptr;
            uint4 o = make_uint4(kScaNoTap, kScaNoTap, kScaNoTap, kScaNoTap);
            float ax = 0.0f, ay = 0.0f, aa = 0.0f;
            if (mine) {
                if (sca_setup_point(p, m, ref, s, j, head_off, o, ax, ay))
                    aa = s.inv * a_j;   // the value scatter's factor: mean times a_j
            }
            uint32_t *mine_rec = rec + s.sub * kRecBwd;
            *reinterpret_cast<uint4 *>(mine_rec) = o;
            *reinterpret_cast<float4 *>(mine_rec + 4) = make_float4(ax, ay, aa, 0.0f);
            wave_lds_sync();
            SPH_COUNT(kSpSteps, 1);
            SPH_ADD(kSpRecords);
            // gradients of the point this lane owns (point c0 + sub)
            float my_da = 0.0f, my_dx = 0.0f, my_dy = 0.0f;
            for (int t = 0; t < npts; ++t) {
                const uint4 to = *reinterpret_cast<const uint4 *>(rec + t * kRecBwd);
                const float4 tf = *reinterpret_cast<const float4 *>(rec + t * kRecBwd + 4);
                const float4 tw = sca_weights(to, tf.x, tf.y, 1.0f);
                Raw<LW> v0{}, v1{}, v2{}, v3{};
                if (to.x != kScaNoTap) v0 = load_vec<LW>(rsrc, to.x + lane_off, 0);
                if (to.y != kScaNoTap) v1 = load_vec<LW>(rsrc, to.y + lane_off, 0);
                if (to.z != kScaNoTap) v2 = load_vec<LW>(rsrc, to.z + lane_off, 0);
                if (to.w != kScaNoTap) v3 = load_vec<LW>(rsrc, to.w + lane_off, 0);
                // this lane's share of sum_c V[tap, c] G[c] for the four taps
                float d0 = 0.0f, d1 = 0.0f, d2 = 0.0f, d3 = 0.0f;
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    d0 = fmaf(elem<DT, LW>(v0, e), gs[e], d0);
                    d1 = fmaf(elem<DT, LW>(v1, e), gs[e], d1);
                    d2 = fmaf(elem<DT, LW>(v2, e), gs[e], d2);
                    d3 = fmaf(elem<DT, LW>(v3, e), gs[e], d3);
                }
                // the point's gradients are linear in the four dot products
                // with weights shared by the slot's lanes: each lane forms
                // its share, and three sums cross the slot in place of four
                const float tax = tf.x, tay = tf.y;
                float da = ((tw.x * d0 + tw.y * d1) + tw.z * d2) + tw.w * d3;
                float dx = (1.0f - tay) * (d1 - d0) + tay * (d3 - d2);
                float dy = (1.0f - tax) * (d2 - d0) + tax * (d3 - d1);
                for (int x = lph >> 1; x >= 1; x >>= 1) {
                    da += __shfl_xor(da, x);
                    dx += __shfl_xor(dx, x);
                    dy += __shfl_xor(dy, x);
                }
                const bool owner = s.sub == t;
                my_da += owner ? da : 0.0f;
                my_dx += owner ? dx : 0.0f;
                my_dy += owner ? dy : 0.0f;
            }
            g_da += my_da;
            g_dx += my_dx;
            g_dy += my_dy;
            SPH_ADD(kSpPoint);
            // value gradient: mean * a * w * G[c] onto each in-range tap.  Each
            // wavefront puts its (point, slot, tap) rows into the table by tap
            // offset; rows on the same pixel (all slots share the head) land
            // on one key and are summed before a single scatter of the key's
            // row.  The workgroup then walks the distinct rows, 64 consecutive
            // channels per atomic instruction, so one instruction covers whole
            // head rows (one 128-byte row per 32 lanes for float32 D = 32).
            if (gv) {
                const int nrows = npts << (spw_shift + 2);
                for (int r = lane; r < nrows; r += kScaWave) {
                    const int ts = r >> 2;
                    const uint32_t *rr = m.tap +
                                         (size_t)(wave * p.spw + (ts & (p.spw - 1))) * p.slot_stride +
                                         (ts >> spw_shift) * kRecBwd;
                    const uint32_t key = rr[r & 3];
                    if (key == kScaNoTap) continue;
                    const uint32_t R = (uint32_t)(wave * kMrgRows + r);
                    uint32_t h = (key * 0x9E3779B1u) >> p.mrg_shift;
                    bool placed = false;
                    for (int probe = 0; probe < trows; ++probe) {
                        const uint32_t old = atomicCAS(&tkey[h], kMrgEmpty, key);
                        if (old == kMrgEmpty) {
                            tuniq[atomicAdd(tcount, 1u)] = (uint16_t)h;
                            placed = true;
                            break;
                        }
                        if (old == key) {
                            placed = true;
                            break;
                        }
                        h = (h + 1) & (uint32_t)(trows - 1);
                    }
                    if (placed) {
                        const int sl = wave * p.spw + (ts & (p.spw - 1));
                        // the tap's bilinear weight, as sca_weights forms it
                        const float fx = __builtin_bit_cast(float, rr[4]);
                        const float fy = __builtin_bit_cast(float, rr[5]);
                        const float wr = (r & 2) ? fy : 1.0f - fy;
                        const float wc = (r & 1) ? fx : 1.0f - fx;
                        const float cf = __builtin_bit_cast(float, rr[6]) * (wr * wc);
                        rrow[R] = make_uint2(__builtin_bit_cast(uint32_t, cf),
                                             ((uint32_t)(sl * D) << 16) |
                                                 (atomicExch(&thead[h], R) & kMrgEnd16));
                    } else {
                        // unreachable (the table holds every row of a chunk);
                        // the row is then scattered alone
                        const int sl = wave * p.spw + (ts & (p.spw - 1));
                        const float fx = __builtin_bit_cast(float, rr[4]);
                        const float fy = __builtin_bit_cast(float, rr[5]);
                        const float coef = __builtin_bit_cast(float, rr[6]) *
                                           (((r & 2) ? fy : 1.0f - fy) * ((r & 1) ? fx : 1.0f - fx));
                        for (int ch = 0; ch < D; ++ch)
                            unsafeAtomicAdd(gv + key / ES + ch, coef * m.gst[sl * D + ch]);
                    }
                }
                SPH_ADD(kSpInsert);
                __syncthreads();
                SPH_ADD(kSpInsertBarrier);
                const int nel = (int)*tcount * D;
                SPH_COUNT(kSpKeys, *tcount);
                // element E = u D + ch, stepped by nthreads = du D + dch
                int u = u0, ch = ch0;
                for (int E = tid; E < nel; E += nthreads) {
                    const uint32_t h = tuniq[u] & (uint32_t)(trows - 1);
                    const uint32_t key = tkey[h];
                    uint32_t R = thead[h];
                    float val = 0.0f;
                    if (R < (uint32_t)trows) {
                        // the next member's factor and link (one 8-byte read)
                        // are read while this member's output-gradient
                        // element is
                        uint2 e = rrow[R];
                        for (int k = 0; k < trows; ++k) {
                            const uint32_t lk = e.y;
                            const float g = m.gst[(lk >> 16) + ch];
                            const uint32_t nx = lk & kMrgEnd16;
                            const bool more = nx < (uint32_t)trows;
                            const uint2 en = rrow[more ? nx : R];
                            val = fmaf(__builtin_bit_cast(float, e.x), g, val);
                            if (!more) break;
                            R = nx;
                            e = en;
                        }
                    }
                    if (key < p.cam_bytes) unsafeAtomicAdd(gv + key / ES + ch, val);
                    u += du;
                    ch += dch;
                    if (ch >= D) {
                        ch -= D;
                        ++u;
                    }
                }
                SPH_ADD(kSpWalk);
                __syncthreads();
                SPH_ADD(kSpWalkBarrier);
                for (int h = tid; h < trows; h += nthreads) {
                    tkey[h] = kMrgEmpty;
                    thead[h] = kMrgEnd;
                }
                if (tid == 0) *tcount = 0u;
                __syncthreads();
                SPH_ADD(kSpClear);
            } else {
                wave_lds_sync();
            }
        }
        if (own) {
            dot += a_j * g_da;
            const float sa = s.inv * a_j;
            if (p.grad_offsets)
                reinterpret_cast<float2 *>(p.grad_offsets)[s.pt0 + j] =
                    make_float2(sa * g_dx, sa * g_dy);
            // d a_j for now; the softmax backward below finishes it
            if (p.grad_logits) p.grad_logits[s.pt0 + j] = g_da;
        }
    }

    // ---- softmax backward (lanes own points j = sub mod lph; each lane
    // reads back only what it wrote itself)
    for (int x = lph >> 1; x >= 1; x >>= 1) dot += __shfl_xor(dot, x);
    if (s.active) {
        for (int j = s.sub; j < LP; j += lph) {
            if (s.hits) {
                if (p.grad_logits) {
                    const float sa = s.inv * (expf(p.logits[s.pt0 + j] - mx) * rcp);
                    p.grad_logits[s.pt0 + j] = sa * (p.grad_logits[s.pt0 + j] - dot);
                }
            } else {
                // no hit camera: the point gradients are zero
                if (p.grad_logits) p.grad_logits[s.pt0 + j] = 0.0f;
                if (p.grad_offsets)
                    reinterpret_cast<float2 *>(p.grad_offsets)[s.pt0 + j] = make_float2(0.0f, 0.0f);
            }
        }
    }
    SPH_ADD(kSpTail);
    SPH_WRITE(lane);
}

__global__ void __launch_bounds__(256) sca_zero_fill(float *dst, uint64_t n)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        dst[i] = 0.0f;
}

using ScaKernelFn = void (*)(const ScaParams);

template <int DT, bool BWD>
ScaKernelFn pick_sca_lw(int lw)
{
    switch (lw) {
    case 16: return BWD ? sca_bwd<DT, 16> : sca_fwd<DT, 16>;
    case 8: return BWD ? sca_bwd<DT, 8> : sca_fwd<DT, 8>;
    case 4: return BWD ? sca_bwd<DT, 4> : sca_fwd<DT, 4>;
    default:
        if constexpr (DT == FLASHBEV_F32) return nullptr;
        else return BWD ? sca_bwd<DT, 2> : sca_fwd<DT, 2>;
    }
}

ScaKernelFn pick_sca(int dtype, int lw, bool backward)
{
    switch (dtype) {
    case FLASHBEV_F32:
        return backward ? pick_sca_lw<FLASHBEV_F32, true>(lw) : pick_sca_lw<FLASHBEV_F32, false>(lw);
    case FLASHBEV_F16:
        return backward ? pick_sca_lw<FLASHBEV_F16, true>(lw) : pick_sca_lw<FLASHBEV_F16, false>(lw);
    default:
        return backward ? pick_sca_lw<FLASHBEV_BF16, true>(lw) : pick_sca_lw<FLASHBEV_BF16, false>(lw);
    }
}

struct ScaPlan {
    ScaParams prm;
    int64_t workgroups;
    int threads;
    size_t lds;
    int lw;
    bool empty;
    uint64_t value_elems;   // B N S C
};

bool sca_finite(float v) { return v == v && v - v == 0.0f; }

bool sca_overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    if (!na || !nb || !a || !b) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + nb && b0 < a0 + na;
}

// Device pointers of one call (forward: out; backward: grad_out and the
// three gradients, any of which may be null).
struct ScaBufs {
    const float *l2i = nullptr;
    const float *off = nullptr;
    const float *lg = nullptr;
    const float *out = nullptr;
    const float *gout = nullptr;
    const float *gvalue = nullptr;
    const float *goff = nullptr;
    const float *glg = nullptr;
};

// Azimuth order of the query blocks.  Query groups are visited block by
// block (query_of); here the blocks are sorted by the angle of their centre
// around the BEV origin (the ego), so that a run of consecutive groups is a
// sector of the grid, seen by one or two cameras.  A pixel row of a camera is
// used by queries at a few depths along its viewing ray (one per anchor
// height), which a sweep of the grid in bands reaches at separate times and a
// sector holds together: its value rows are then fetched into an L2 about
// once.  Taken where every block holds whole query groups and there are at
// most kScaOrdMax blocks (BEVFormer's grids), for many points per head (the
// plan below); otherwise rank order.
void sca_azimuth_order(ScaParams &p)
{
    p.ord_blocks = 0;
    const int tp = p.tile_pairs;
    const int X = p.X, Y = p.Y;
    if (tp < 1 || X < 1 || Y < 1) return;
    const int nbx = (X + kScaBlock - 1) / kScaBlock, nby = (Y + kScaBlock - 1) / kScaBlock;
    const int64_t nb = (int64_t)nbx * nby;
    const int64_t nqg = ((int64_t)X * Y + tp - 1) / tp;
    if (nb < 2 || nb > kScaOrdMax || nqg > 0xFFFF) return;
    struct Blk {
        double ang;
        int idx, first, tiles;
    };
    Blk blk[kScaOrdMax];
    int n = 0;
    for (int R = 0; R < nbx; ++R) {
        const int h = (X - R * kScaBlock) < kScaBlock ? (X - R * kScaBlock) : kScaBlock;
        const int64_t band0 = (int64_t)R * kScaBlock * Y;
        for (int c = 0; c < nby; ++c) {
            const int w = (Y - c * kScaBlock) < kScaBlock ? (Y - c * kScaBlock) : kScaBlock;
            const int64_t start = band0 + (int64_t)c * h * kScaBlock;
            const int64_t size = (int64_t)h * w;
            if (start % tp || size % tp) return;
            const double xc = (double)p.x_min + ((double)(R * kScaBlock) + 0.5 * h) * (double)p.dx;
            const double yc = (double)p.y_min + ((double)(c * kScaBlock) + 0.5 * w) * (double)p.dy;
            blk[n].ang = atan2(yc, xc);
            blk[n].idx = n;
            blk[n].first = (int)(start / tp);
            blk[n].tiles = (int)(size / tp);
            ++n;
        }
    }
    std::sort(blk, blk + n, [](const Blk &a, const Blk &b) {
        return a.ang < b.ang || (a.ang == b.ang && a.idx < b.idx);
    });
    int cum = 0;
    for (int k = 0; k < n; ++k) {
        p.ord_first[k] = (uint16_t)blk[k].first;
        p.ord_cum[k] = (uint16_t)cum;
        cum += blk[k].tiles;
    }
    p.ord_cum[n] = (uint16_t)cum;
    p.ord_blocks = n;
}

// All argument checks; `need_data` requires the device pointers.
int make_sca_plan(const flashsca_value *v, const flashbev_bev_grid_spec *s,
                  const flashbev_z_bins *zb, int32_t P, const ScaBufs &bf, bool backward,
                  bool need_data, ScaPlan *pl)
{
    if (!v || !s || !zb) return FLASHBEV_ERR_NULLPTR;
    if (v->dtype != FLASHBEV_F32 && v->dtype != FLASHBEV_F16 && v->dtype != FLASHBEV_BF16)
        return FLASHBEV_ERR_DTYPE;
    if (v->B < 0 || v->N < 0 || v->C < 1 || v->heads < 1 || v->L < 1 || v->img_h < 1 ||
        v->img_w < 1 || s->X < 0 || s->Y < 0 || zb->Z < 1 || P < 1)
        return FLASHBEV_ERR_SHAPE;
    if (v->C % v->heads != 0 || P % zb->Z != 0) return FLASHBEV_ERR_SHAPE;
    if (v->L > FLASHSCA_LMAX) return FLASHBEV_ERR_UNSUPPORTED;
    // every size product saturates instead of wrapping (size_prod); the
    // level areas are each below 2^62, so their sum of at most
    // FLASHSCA_LMAX terms is checked against the cap before it could wrap
    uint64_t S = 0;
    for (int l = 0; l < v->L && l < FLASHSCA_LMAX; ++l) {
        if (v->level_h[l] < 1 || v->level_w[l] < 1) return FLASHBEV_ERR_SHAPE;
        S += size_prod({(uint64_t)v->level_h[l], (uint64_t)v->level_w[l]});
        if (S > kSizeCap) return FLASHBEV_ERR_UNSUPPORTED;
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
    const uint64_t cam_bytes = size_prod({S, row});
    if (cam_bytes > kScaCamBytesMax) return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t Q = size_prod({(uint64_t)s->X, (uint64_t)s->Y});
    if (Q > 0x7FFFFFFFull || size_prod({Q, (uint64_t)v->heads}) > 0x7FFFFFFFull)
        return FLASHBEV_ERR_UNSUPPORTED;
    const int LP = v->L * P;
    const uint64_t out_elems = size_prod({(uint64_t)v->B, Q, (uint64_t)v->C});
    const uint64_t value_elems = size_prod({(uint64_t)v->B, (uint64_t)v->N, S, (uint64_t)v->C});
    const uint64_t pts = size_prod({(uint64_t)v->B, Q, (uint64_t)v->heads, (uint64_t)LP});
    // byte sizes below (x 8 at most) stay inside 64 bits
    if (out_elems > kSizeCap / 8 || value_elems > kSizeCap / 8 || pts > kSizeCap / 8)
        return FLASHBEV_ERR_UNSUPPORTED;
    const uint64_t value_bytes = value_elems * es;
    // forward: nothing to do without outputs; backward: a requested value
    // gradient is still zeroed
    const bool empty = out_elems == 0;
    if (need_data) {
        const size_t ob = out_elems * 4;
        if (!backward) {
            if (!empty) {
                if (!bf.out || !bf.off || !bf.lg) return FLASHBEV_ERR_NULLPTR;
                if (value_bytes > 0 && !v->data) return FLASHBEV_ERR_NULLPTR;
                if (v->N > 0 && !bf.l2i) return FLASHBEV_ERR_NULLPTR;
                if (((uintptr_t)v->data % es) || ((uintptr_t)bf.l2i % 4) ||
                    ((uintptr_t)bf.out % 4) || ((uintptr_t)bf.off % 8) || ((uintptr_t)bf.lg % 4))
                    return FLASHBEV_ERR_ALIGN;
                if (sca_overlaps(bf.out, ob, v->data, value_bytes) ||
                    sca_overlaps(bf.out, ob, bf.l2i, (size_t)v->B * v->N * 64) ||
                    sca_overlaps(bf.out, ob, bf.off, pts * 8) ||
                    sca_overlaps(bf.out, ob, bf.lg, pts * 4))
                    return FLASHBEV_ERR_ALIAS;
            }
        } else {
            if (!bf.gvalue && !bf.goff && !bf.glg) return FLASHBEV_ERR_NULLPTR;
            if (!empty) {
                if (!bf.gout || !bf.off || !bf.lg) return FLASHBEV_ERR_NULLPTR;
                if (value_bytes > 0 && !v->data) return FLASHBEV_ERR_NULLPTR;
                if (v->N > 0 && !bf.l2i) return FLASHBEV_ERR_NULLPTR;
            }
            if (((uintptr_t)v->data % es) || ((uintptr_t)bf.l2i % 4) || ((uintptr_t)bf.gout % 4) ||
                ((uintptr_t)bf.off % 8) || ((uintptr_t)bf.lg % 4) || ((uintptr_t)bf.gvalue % 4) ||
                ((uintptr_t)bf.goff % 8) || ((uintptr_t)bf.glg % 4))
                return FLASHBEV_ERR_ALIGN;
            // every output is disjoint from every input and from the others
            const void *ins[5] = {v->data, bf.l2i, bf.off, bf.lg, bf.gout};
            const size_t insz[5] = {(size_t)value_bytes, (size_t)v->B * v->N * 64,
                                    (size_t)pts * 8, (size_t)pts * 4, ob};
            const void *outs[3] = {bf.gvalue, bf.goff, bf.glg};
            const size_t outsz[3] = {(size_t)value_elems * 4, (size_t)pts * 8, (size_t)pts * 4};
            for (int a = 0; a < 3; ++a) {
                for (int i = 0; i < 5; ++i)
                    if (sca_overlaps(outs[a], outsz[a], ins[i], insz[i])) return FLASHBEV_ERR_ALIAS;
                for (int c = a + 1; c < 3; ++c)
                    if (sca_overlaps(outs[a], outsz[a], outs[c], outsz[c]))
                        return FLASHBEV_ERR_ALIAS;
            }
        }
    }

    // lane slice: 16 bytes where a head row has at least four of them
    // (measured on MI355X, BEVFormer-base bfloat16: 16-byte lanes, 4 per head,
    // 0.521 -> 0.484 ms against 8-byte lanes, 8 per head), else narrower;
    // always a width dividing the head row, the full row and the base address
    int lw = 16;
    while (lw > es && (uint64_t)lw * 4 > head_bytes) lw >>= 1;
    // the backward takes 8 lanes per head where it can (BEVFormer-base
    // bfloat16, B = 2: 8-byte lanes 3.13 ms against 16-byte 3.53 ms at
    // P = 8, 9.8 against 11.1 ms at P = 32): 8 queries per wavefront, 8
    // points per chunk and the LDS of four workgroups per CU
    if (backward) while (lw > es && (uint64_t)lw * 8 > head_bytes) lw >>= 1;
    while (lw > es && ((head_bytes % lw) != 0 || (row % lw) != 0 ||
                       (((uintptr_t)v->data) % lw) != 0))
        lw >>= 1;
    const int nvec = (int)((head_bytes + lw - 1) / lw);
    int lph = 1, lph_shift = 0;
    while (lph < nvec) { lph <<= 1; ++lph_shift; }
    if (lph > kScaWave) return FLASHBEV_ERR_UNSUPPORTED;
    const int spw = kScaWave / lph;
    const int slot_stride = lph * (backward ? kRecBwd : kRecFwd) + kSlotPad;

    int waves = backward ? kScaBwdWavesMax : kScaWavesMax;
    const uint32_t budget = backward ? kScaBwdLdsBudget : kScaLdsBudget;
    int nq_max = 0;
    ScaLds lay{};
    for (;;) {
        const int tp = waves * spw;
        // tp consecutive queries of one head
        nq_max = tp;
        if ((uint64_t)nq_max > Q) nq_max = (int)(Q > 0 ? Q : 1);
        lay = sca_lds_layout(v->N, zb->Z, nq_max, waves, spw, LP, D, slot_stride, backward);
        if (lay.total <= budget || waves == 1) break;
        waves >>= 1;
    }
    // many points per head: one wavefront per workgroup, with more LDS
    if (lay.total > kScaLdsMax) return FLASHBEV_ERR_UNSUPPORTED;
    const int tile_pairs = waves * spw;
    // the backward's row links hold an output-gradient row offset in 16 bits
    if (backward && (uint64_t)tile_pairs * D > 0xFFFFu) return FLASHBEV_ERR_UNSUPPORTED;

    ScaParams &p = pl->prm;
    memset(&p, 0, sizeof(p));
    p.value = v->data;
    p.l2i = bf.l2i;
    p.offsets = bf.off;
    p.logits = bf.lg;
    p.out = const_cast<float *>(bf.out);
    p.grad_out = bf.gout;
    p.grad_value = const_cast<float *>(bf.gvalue);
    p.grad_offsets = const_cast<float *>(bf.goff);
    p.grad_logits = const_cast<float *>(bf.glg);
    p.cam_bytes = cam_bytes;
    p.cam_elems = S * (uint64_t)v->C;
    p.row_bytes = (uint32_t)row;
    p.head_bytes = (uint32_t)head_bytes;
    p.B = v->B; p.N = v->N; p.C = v->C; p.heads = v->heads; p.D = D;
    p.L = v->L; p.P = P; p.Z = zb->Z; p.LP = LP;
    p.X = s->X; p.Y = s->Y; p.Q = (int32_t)Q;
    p.lph = lph;
    p.lph_shift = lph_shift;
    p.spw = spw;
    p.tile_pairs = tile_pairs;
    // tiles of tile_pairs queries of one head (at most Q heads tiles, within
    // 2^31 - 1)
    p.tiles_per_b = (int32_t)(((Q + tile_pairs - 1) / tile_pairs) * (uint64_t)v->heads);
    // head-to-XCD order (sca_tile) for the forward; the backward, whose time
    // at few points goes to the row merge and its atomics, keeps the band
    // order up to 32 points per head (measured on MI355X at BEVFormer-base:
    // P = 8 1.44 ms band against 1.47 head order, P = 32 4.50 against 4.36)
    p.head_xcd = ((v->heads % kScaXcds) == 0 && (!backward || LP > 32)) ? kScaHeadChunks : 0;
    {
        int lg = 0;
        while ((kMrgRows * waves) >> (lg + 1)) ++lg;
        p.mrg_shift = 32 - lg;   // merge-table rows: 256 per wavefront
    }
    {
        // one contiguous band of tiles per XCD (see sca_tile)
        const int64_t nt = (int64_t)v->B * p.tiles_per_b / kScaXcds;
        p.stripe = (int32_t)(nt < 1 ? 1 : nt);
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
    p.lds_gst = lay.gst;
    p.rcp_d = 1.0f / (float)D;
    p.lds_tap = lay.tap;
    p.lds_mrg = lay.mrg;
    for (int k = 0; k < zb->Z; ++k) p.z[k] = zb->z[k];
    // azimuth order where a head's points spread widely (measured on MI355X
    // at BEVFormer-base, against rank order: forward P = 32 0.768 -> 0.759 ms
    // with fabric fetches 1.14 -> 0.79 GB, but P = 8 0.256 -> 0.270 and
    // P = 16 0.446 -> 0.453; backward P = 16 2.57 -> 2.50, P = 32 4.36 ->
    // 4.21, but P = 8 1.45 -> 1.60): there the order keeps a sector's value
    // rows in the L2s, with few points the band order's short-range locality
    // is worth more
    if (backward ? LP > 32 : LP >= 128) sca_azimuth_order(p);
    else p.ord_blocks = 0;

    pl->workgroups = empty ? 0 : (int64_t)v->B * p.tiles_per_b;
    if (pl->workgroups > 0x7FFFFFFFll) return FLASHBEV_ERR_UNSUPPORTED;
    pl->threads = waves * kScaWave;
    pl->lds = lay.total;
    pl->lw = lw;
    pl->empty = empty;
    pl->value_elems = value_elems;
    return FLASHBEV_OK;
}

void write_info(const ScaPlan &pl, int64_t *workgroups, int32_t *threads, int32_t *lds,
                int32_t *lanes_per_head, int32_t *lane_bytes)
{
    if (workgroups) *workgroups = pl.workgroups;
    if (threads) *threads = pl.threads;
    if (lds) *lds = (int32_t)pl.lds;
    if (lanes_per_head) *lanes_per_head = pl.prm.lph;
    if (lane_bytes) *lane_bytes = pl.lw;
}

int launch(ScaKernelFn fn, ScaPlan &pl, hipStream_t st)
{
    const void *f = reinterpret_cast<const void *>(fn);
    if (pl.lds > kScaLdsBudget &&
        hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds) !=
            hipSuccess)
        return FLASHBEV_ERR_HIP;
    void *args[] = {&pl.prm};
    const hipError_t e = hipLaunchKernel(f, dim3((unsigned)pl.workgroups), dim3(pl.threads), args,
                                         pl.lds, st);
    return e == hipSuccess ? FLASHBEV_OK : FLASHBEV_ERR_HIP;
}

}  // namespace

extern "C" int flashsca_launch_info(const flashsca_value *value,
                                    const flashbev_bev_grid_spec *spec,
                                    const flashbev_z_bins *anchors, int32_t P, int64_t *workgroups,
                                    int32_t *threads_per_workgroup, int32_t *lds_bytes,
                                    int32_t *lanes_per_head, int32_t *lane_bytes)
{
    ScaPlan pl;
    const int rc = make_sca_plan(value, spec, anchors, P, ScaBufs{}, false, false, &pl);
    if (rc) return rc;
    write_info(pl, workgroups, threads_per_workgroup, lds_bytes, lanes_per_head, lane_bytes);
    return FLASHBEV_OK;
}

extern "C" int flashsca_backward_launch_info(const flashsca_value *value,
                                             const flashbev_bev_grid_spec *spec,
                                             const flashbev_z_bins *anchors, int32_t P,
                                             int64_t *workgroups, int32_t *threads_per_workgroup,
                                             int32_t *lds_bytes, int32_t *lanes_per_head,
                                             int32_t *lane_bytes)
{
    ScaPlan pl;
    const int rc = make_sca_plan(value, spec, anchors, P, ScaBufs{}, true, false, &pl);
    if (rc) return rc;
    write_info(pl, workgroups, threads_per_workgroup, lds_bytes, lanes_per_head, lane_bytes);
    return FLASHBEV_OK;
}

extern "C" int flashsca_forward(const flashsca_value *value, const float *lidar2img,
                                const flashbev_bev_grid_spec *spec,
                                const flashbev_z_bins *anchors, int32_t P, const float *offsets,
                                const float *logits, float *out, void *stream)
{
    ScaBufs bf;
    bf.l2i = lidar2img;
    bf.off = offsets;
    bf.lg = logits;
    bf.out = out;
    ScaPlan pl;
    const int rc = make_sca_plan(value, spec, anchors, P, bf, false, true, &pl);
    if (rc) return rc;
    if (pl.empty) return FLASHBEV_OK;
    const ScaKernelFn fn = pick_sca(value->dtype, pl.lw, false);
    if (!fn) return FLASHBEV_ERR_UNSUPPORTED;
    return launch(fn, pl, reinterpret_cast<hipStream_t>(stream));
}

extern "C" int flashsca_backward(const flashsca_value *value, const float *lidar2img,
                                 const flashbev_bev_grid_spec *spec,
                                 const flashbev_z_bins *anchors, int32_t P, const float *offsets,
                                 const float *logits, const float *grad_out, float *grad_value,
                                 float *grad_offsets, float *grad_logits, void *stream)
{
    ScaBufs bf;
    bf.l2i = lidar2img;
    bf.off = offsets;
    bf.lg = logits;
    bf.gout = grad_out;
    bf.gvalue = grad_value;
    bf.goff = grad_offsets;
    bf.glg = grad_logits;
    ScaPlan pl;
    const int rc = make_sca_plan(value, spec, anchors, P, bf, true, true, &pl);
    if (rc) return rc;
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (grad_value && pl.value_elems > 0) {
        uint64_t blocks = (pl.value_elems + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        // the launch's own status (hipGetLastError could report an earlier call's)
        float *dst = grad_value;
        uint64_t n = pl.value_elems;
        void *fargs[] = {&dst, &n};
        if (hipLaunchKernel(reinterpret_cast<const void *>(sca_zero_fill), dim3((unsigned)blocks),
                            dim3(256), fargs, 0, st) != hipSuccess)
            return FLASHBEV_ERR_HIP;
    }
    if (pl.empty) return FLASHBEV_OK;
    const ScaKernelFn fn = pick_sca(value->dtype, pl.lw, true);
    if (!fn) return FLASHBEV_ERR_UNSUPPORTED;
    return launch(fn, pl, st);
}

#ifdef FLASHBEV_PHASE_CLOCK
extern "C" int flashsca_phase_log(void *log)
{
    return hipMemcpyToSymbol(HIP_SYMBOL(sca_phase_log), &log, sizeof(log)) == hipSuccess ? 0 : -1;
}
#endif
