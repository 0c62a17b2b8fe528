// Helpers shared by the library's kernels (flashbev.hip, flashsca.hip):
// 16/8/4/2-byte buffer loads, exact conversion of stored elements to
// float32, wavefront-local LDS ordering, a small exact integer division, and
// on the host a size product that cannot wrap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <initializer_list>

#include "flashbev.h"

namespace {

// ---------------------------------------------------------------------------
// feature vector loads and conversion to float32
// ---------------------------------------------------------------------------
template <int DT>
struct ElemSize { static constexpr int value = (DT == FLASHBEV_F32) ? 4 : 2; };

template <int LW>
struct Raw { uint32_t w[LW >= 4 ? LW / 4 : 1]; };

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
        const uint32_t w = r.w[e >> 1];
        const uint32_t bits = (e & 1) ? (w & 0xffff0000u) : (w << 16);
        return __builtin_bit_cast(float, bits);
    } else {
        const uint32_t w = r.w[e >> 1];
        const uint16_t h = (e & 1) ? (uint16_t)(w >> 16) : (uint16_t)(w & 0xffffu);
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

// a / d for 0 <= a < 2^22 and 1 <= d < 2^22, with rcp = float32(1 / d): the
// float estimate is within one of the quotient and one correction step
// each way makes it exact
__device__ __forceinline__ int div_small(int a, int d, float rcp)
{
    int q = (int)((float)a * rcp);
    const int r = a - q * d;
    q += (r >= d) ? 1 : 0;
    q -= (r < 0) ? 1 : 0;
    return q;
}

// ---------------------------------------------------------------------------
// host: sizes
// ---------------------------------------------------------------------------
// Product of non-negative sizes that cannot wrap: the exact product while
// every partial product stays at most kSizeCap (2^62), else kSizeOver, which
// every size limit of the library rejects.  A zero factor gives zero.
constexpr uint64_t kSizeCap = 1ull << 62;
constexpr uint64_t kSizeOver = ~0ull;

inline uint64_t size_prod(std::initializer_list<uint64_t> factors)
{
    for (const uint64_t v : factors)
        if (v == 0) return 0;
    uint64_t p = 1;
    for (const uint64_t v : factors) {
        if (p > kSizeCap / v) return kSizeOver;
        p *= v;
    }
    return p;
}

}  // namespace
