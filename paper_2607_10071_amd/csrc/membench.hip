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

__global__ void __launch_bounds__(kThreads)
gather_kernel(const void *buf, uint32_t nrows, uint32_t row_bytes, uint32_t row_pitch,
              int32_t iters, int32_t lpc, int32_t cpw, float *sink)
{
    const int lane = threadIdx.x % 64;
    const int wave = (blockIdx.x * kThreads + threadIdx.x) / 64;
    const int m = lane / lpc;
    const int slot = lane - m * lpc;
    const bool active = m < cpw;
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void *>(buf), (short)0, (int)(nrows * row_bytes), 0x00020000);
    // first-tap rows r satisfy r + row_pitch + 1 < nrows
    const uint32_t span = nrows - row_pitch - 1;
    const uint32_t sx = row_bytes, sy = row_bytes * row_pitch;
    float acc0 = 0.0f, acc1 = 0.0f, acc2 = 0.0f, acc3 = 0.0f;
    for (int it = 0; it < iters; it += 2) {
        const uint32_t h0 = mix((uint32_t)wave * 0x9e3779b9u + (uint32_t)it * 0x85ebca6bu + m);
        const uint32_t h1 = mix(h0 + 0x27d4eb2fu);
        const uint32_t v0 = active ? (h0 % span) * row_bytes + slot * 16u : 0x80000000u;
        const uint32_t v1 = active ? (h1 % span) * row_bytes + slot * 16u : 0x80000000u;
        uint32_t t[8][4];
        const uint32_t vo[2] = {v0, v1};
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            auto a = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo[u], 0u, 0);
            auto b = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo[u], sx, 0);
            auto c = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo[u], sy, 0);
            auto d = __builtin_amdgcn_raw_buffer_load_b128(rsrc, vo[u], sx + sy, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                t[4 * u + 0][e] = a[e];
                t[4 * u + 1][e] = b[e];
                t[4 * u + 2][e] = c[e];
                t[4 * u + 3][e] = d[e];
            }
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
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
                             int32_t row_pitch, int32_t iters, int32_t workgroups, float *sink,
                             void *stream)
{
    if (!buf || !sink) return -1;
    if (row_bytes < 16 || row_bytes > 1024 || row_bytes % 16 || row_pitch < 1 || iters < 2 ||
        iters % 2 ||
        workgroups < 1 || ((uintptr_t)buf % 16))
        return -2;
    if (buf_bytes > 0x7FFFFFFFull) return -3;
    const uint64_t nrows = buf_bytes / (uint64_t)row_bytes;
    if (nrows < (uint64_t)row_pitch + 3) return -2;
    const int lpc = row_bytes / 16;
    int cpw = 64 / lpc;
    if (cpw > 8) cpw = 8;
    const void *a0 = buf;
    uint32_t a1 = (uint32_t)nrows, a2 = (uint32_t)row_bytes, a3 = (uint32_t)row_pitch;
    int32_t a4 = iters, a5 = lpc, a6 = cpw;
    float *a7 = sink;
    void *args[] = {&a0, &a1, &a2, &a3, &a4, &a5, &a6, &a7};
    return launch_status(reinterpret_cast<const void *>(gather_kernel), workgroups, args, stream);
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
