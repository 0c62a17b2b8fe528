// The fused Sampling-VT forward driven through the C ABI alone: plain HIP
// memory and a HIP stream, no Python and no torch.  Test infrastructure: the
// GPU test writes the inputs, runs this program and checks its output
// against the oracle.
//
//   c_abi_forward <inputs> <output>
//
// Input file (little-endian): int32 B, N, H, W, C, img_h, img_w, X, Y, Z,
// reduce; float32 x_min, dx, y_min, dy, depth_eps; float32 features
// [B, N, H, W, C]; float32 lidar2img [B, N, 4, 4]; float32 heights [Z].
// Output file: float32 out [B, C, X, Y].
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

#include "flashbev.h"

namespace {

bool read_all(std::FILE *f, void *dst, size_t bytes)
{
    return bytes == 0 || std::fread(dst, 1, bytes, f) == bytes;
}

int fail(const char *what, int code)
{
    std::fprintf(stderr, "c_abi_forward: %s (%d)\n", what, code);
    return 1;
}

}  // namespace

int main(int argc, char **argv)
{
    if (argc != 3) return fail("usage: c_abi_forward <inputs> <output>", 2);
    std::FILE *in = std::fopen(argv[1], "rb");
    if (!in) return fail("cannot open inputs", 0);
    int32_t d[11];
    float g[5];
    if (!read_all(in, d, sizeof d) || !read_all(in, g, sizeof g)) return fail("short header", 0);
    const int32_t B = d[0], N = d[1], H = d[2], W = d[3], C = d[4], X = d[7], Y = d[8], Z = d[9];
    if (B < 0 || N < 0 || H < 1 || W < 1 || C < 1 || X < 0 || Y < 0 || Z < 0 || Z > FLASHBEV_ZMAX)
        return fail("bad dimensions", 0);
    const size_t nfeat = (size_t)B * N * H * W * C, nmat = (size_t)B * N * 16;
    const size_t nout = (size_t)B * C * X * Y;
    std::vector<float> feat(nfeat), mat(nmat), z(Z > 0 ? Z : 1), out(nout);
    if (!read_all(in, feat.data(), nfeat * 4) || !read_all(in, mat.data(), nmat * 4) ||
        !read_all(in, z.data(), (size_t)Z * 4))
        return fail("short data", 0);
    std::fclose(in);

    void *dfeat = nullptr, *dmat = nullptr, *dout = nullptr;
    hipError_t e = hipMalloc(&dfeat, nfeat * 4 + 16);
    if (e == hipSuccess) e = hipMalloc(&dmat, nmat * 4 + 16);
    if (e == hipSuccess) e = hipMalloc(&dout, nout * 4 + 16);
    if (e == hipSuccess) e = hipMemcpy(dfeat, feat.data(), nfeat * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(dmat, mat.data(), nmat * 4, hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(hipGetErrorString(e), (int)e);
    hipStream_t st = nullptr;
    if ((e = hipStreamCreate(&st)) != hipSuccess) return fail(hipGetErrorString(e), (int)e);

    flashbev_features f;
    f.data = dfeat;
    f.dtype = FLASHBEV_F32;
    f.B = B; f.N = N; f.H = H; f.W = W; f.C = C;
    f.img_h = d[5]; f.img_w = d[6];
    flashbev_bev_grid_spec spec;
    spec.x_min = g[0]; spec.dx = g[1]; spec.X = X;
    spec.y_min = g[2]; spec.dy = g[3]; spec.Y = Y;
    spec.depth_eps = g[4];
    spec.reduce = d[10];
    flashbev_z_bins zb;
    zb.z = z.data();
    zb.Z = Z;

    const int rc = flashbev_sample_vt(&f, static_cast<const float *>(dmat), &spec, &zb,
                                      static_cast<float *>(dout), st);
    if (rc != FLASHBEV_OK) return fail(flashbev_status_string(rc), rc);
    if ((e = hipStreamSynchronize(st)) != hipSuccess) return fail(hipGetErrorString(e), (int)e);
    if ((e = hipMemcpy(out.data(), dout, nout * 4, hipMemcpyDeviceToHost)) != hipSuccess)
        return fail(hipGetErrorString(e), (int)e);
    (void)hipStreamDestroy(st);
    (void)hipFree(dfeat);
    (void)hipFree(dmat);
    (void)hipFree(dout);

    std::FILE *o = std::fopen(argv[2], "wb");
    if (!o || std::fwrite(out.data(), 4, nout, o) != nout) return fail("cannot write output", 0);
    std::fclose(o);
    std::printf("c_abi_forward: %zu outputs written\n", nout);
    return 0;
}
