// Memory-ceiling micro-benchmarks behind include/flashbev_membench.h.
//
// gather: the access shape of the fused Sampling-VT gather (16-byte lane
// slices of pixel rows, several cells per wavefront, four taps per sample)
// at pseudo-random rows of a small buffer.  stream: coalesced 16-byte reads
// of a large buffer.  Both run on the caller's stream and allocate nothing.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "flashbev_membench.h"

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t mix(uint32_t x)
{
    // integer hash (xorshift-multiply rounds) for pseudo-random rows
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// One sample = four 16-byte loads per lane (two rows, two columns of a
// pixel's bilinear support).  SPI samples are issued before any is summed,
// so a lane keeps 4 SPI loads in flight.  Rows come from a per-cell linear
// congruential sequence masked to a power-of-two span (one multiply-add, a
// shift and an AND per sample), so address arithmetic stays far below the
// loads' issue cost.  The launch's dynamic LDS (never accessed) limits the
// workgroups resident per CU, which sets the occupancy.
// The waves-per-SIMD hint lets the compiler keep all 4 SPI loads of a step
// in registers (it would otherwise shorten the window to fit 8 waves).
template <int SPI>
__global__ void __launch_bounds__(kThreads)
__attribute__((amdgpu_waves_per_eu(1, SPI == 8 ? 2 : (SPI == 4 ? 4 : 8))))
gather_kernel(const void *buf, uint32_t nrows, uint32_t span_mask, uint32_t row_bytes,
              uint32_t row_pitch, int32_t iters, int32_t lpc, int32_t cpw, float *sink)
{
    const int lane = threadIdx.x % 64;
    const int wave = (blockIdx.x * kThreads + threadIdx.x) / 64;
    const int m = lane / lpc;
    const int slot = lane - m * lpc;
    const bool active = m < cpw;
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void *>(buf), (short)0, (int)(nrows * row_bytes), 0x00020000);
    // first-tap rows r <= span_mask satisfy r + row_pitch + 1 < nrows
    const uint32_t sx = row_bytes, sy = row_bytes * row_pitch;
    uint32_t state = mix((uint32_t)wave * 0x9e3779b9u + (uint32_t)m * 0x85ebca6bu);
    const uint32_t lane_off = slot * 16u;
    float acc0 = 0.0f, acc1 = 0.0f, acc2 = 0.0f, acc3 = 0.0f;
    for (int it = 0; it < iters; it += SPI) {
        uint32_t t[4 * SPI][4];
#pragma unroll
        for (int u = 0; u < SPI; ++u) {
            state = state * 1664525u + 1013904223u;
            const uint32_t vo = active ? ((state >> 8) & span_mask) * row_bytes + lane_off
                                       : 0x80000000u;
            auto a = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo, 0u, 0);
            auto b = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo, sx, 0);
            auto c = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo, sy, 0);
            auto d = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo, sx + sy, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                t[4 * u + 0][e] = a[e];
                t[4 * u + 1][e] = b[e];
                t[4 * u + 2][e] = c[e];
                t[4 * u + 3][e] = d[e];
            }
        }
#pragma unroll
        for (int k = 0; k < 4 * SPI; ++k) {
            acc0 = fmaf(0.25f, __builtin_bit_cast(float, t[k][0]), acc0);
            acc1 = fmaf(0.25f, __builtin_bit_cast(float, t[k][1]), acc1);
            acc2 = fmaf(0.25f, __builtin_bit_cast(float, t[k][2]), acc2);
            acc3 = fmaf(0.25f, __builtin_bit_cast(float, t[k][3]), acc3);
        }
    }
    sink[blockIdx.x * kThreads + threadIdx.x] = (acc0 + acc1) + (acc2 + acc3);
}

__global__ void __launch_bounds__(kThreads)
stream_kernel(const uint4 *buf, uint64_t n16, float *sink)
{
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    uint32_t a = 0, b = 0, c = 0, d = 0;
    for (uint64_t i = (uint64_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += stride) {
        const uint4 v = buf[i];
        a ^= v.x; b ^= v.y; c ^= v.z; d ^= v.w;
    }
    sink[blockIdx.x * kThreads + threadIdx.x] = __builtin_bit_cast(float, (a ^ b ^ c ^ d) & 0x007fffffu);
}

__global__ void __launch_bounds__(kThreads)
atomic_kernel(float *buf, uint32_t nrows, int32_t iters)
{
    const int lane = threadIdx.x % 64;
    const uint32_t wave = (blockIdx.x * kThreads + threadIdx.x) / 64;
    for (int it = 0; it < iters; ++it) {
        const uint32_t row = mix(wave * 0x9e3779b9u + (uint32_t)it * 0x85ebca6bu) % nrows;
        unsafeAtomicAdd(buf + (size_t)row * 64u + lane, 1.0f);
    }
}

}  // namespace

// Launch status of this launch alone (hipGetLastError could report an
// earlier call's error).
static int launch_status(const void *fn, int32_t workgroups, void **args, void *stream)
{
    return hipLaunchKernel(fn, dim3((unsigned)workgroups), dim3(kThreads), args, 0,
                           (hipStream_t)stream) == hipSuccess ? 0 : -4;
}

extern "C" {

int flashbev_membench_gather(const void *buf, uint64_t buf_bytes, int32_t row_bytes,
                             int32_t row_pitch, int32_t iters, int32_t loads_in_flight,
                             int32_t lds_bytes, int32_t workgroups, float *sink, void *stream)
{
    if (!buf || !sink) return -1;
    const int spi = loads_in_flight / 4;
    if (row_bytes < 16 || row_bytes > 1024 || row_bytes % 16 || row_pitch < 1 ||
        (spi != 2 && spi != 4 && spi != 8) || iters < spi || iters % spi || workgroups < 1 ||
        lds_bytes < 0 || lds_bytes > 65536 || ((uintptr_t)buf % 16))
        return -2;
    if (buf_bytes > 0x7FFFFFFFull) return -3;
    const uint64_t nrows = buf_bytes / (uint64_t)row_bytes;
    if (nrows < (uint64_t)row_pitch + 3) return -2;
    // the largest power-of-two span of first-tap rows that keeps every tap
    // inside the buffer
    uint32_t span = 1;
    while ((uint64_t)span * 2 + row_pitch + 1 < nrows) span *= 2;
    const int lpc = row_bytes / 16;
    int cpw = 64 / lpc;
    if (cpw > 8) cpw = 8;
    const void *a0 = buf;
    uint32_t a1 = (uint32_t)nrows, a2 = span - 1u, a3 = (uint32_t)row_bytes, a4 = (uint32_t)row_pitch;
    int32_t a5 = iters, a6 = lpc, a7 = cpw;
    float *a8 = sink;
    void *args[] = {&a0, &a1, &a2, &a3, &a4, &a5, &a6, &a7, &a8};
    const void *fn = spi == 2 ? reinterpret_cast<const void *>(gather_kernel<2>)
                   : spi == 4 ? reinterpret_cast<const void *>(gather_kernel<4>)
                              : reinterpret_cast<const void *>(gather_kernel<8>);
    return hipLaunchKernel(fn, dim3((unsigned)workgroups), dim3(kThreads), args, (size_t)lds_bytes,
                           (hipStream_t)stream) == hipSuccess ? 0 : -4;
}

int flashbev_membench_stream(const void *buf, uint64_t bytes, int32_t workgroups, float *sink,
                             void *stream)
{
    if (!buf || !sink) return -1;
    if (bytes == 0 || bytes % (16u * kThreads) || workgroups < 1 || ((uintptr_t)buf % 16)) return -2;
    const uint4 *a0 = (const uint4 *)buf;
    uint64_t a1 = bytes / 16;
    float *a2 = sink;
    void *args[] = {&a0, &a1, &a2};
    return launch_status(reinterpret_cast<const void *>(stream_kernel), workgroups, args, stream);
}

}  // extern "C"

extern "C" int flashbev_membench_atomic(float *buf, uint64_t buf_floats, int32_t iters,
                                        int32_t workgroups, void *stream)
{
    if (!buf) return -1;
    if (buf_floats < 64 || iters < 1 || workgroups < 1 || ((uintptr_t)buf % 4)) return -2;
    if (buf_floats / 64 > 0xFFFFFFFFull) return -3;
    float *a0 = buf;
    uint32_t a1 = (uint32_t)(buf_floats / 64);
    int32_t a2 = iters;
    void *args[] = {&a0, &a1, &a2};
    return launch_status(reinterpret_cast<const void *>(atomic_kernel), workgroups, args, stream);
}
