"""The C headers as plain C (CPU only).

A C99 program that includes every header under include/ is compiled with
gcc -std=c99 -Wall -Wextra -Werror -pedantic, linked against the built
libraries and run.  It calls the entry points that need no GPU: the ABI
version, the status strings, and the launch-geometry and argument-checking
paths of both operators, which return before any HIP call.
"""
import os
import shutil
import subprocess

import pytest

import paper_2607_10071_amd as fb
from paper_2607_10071_amd import membench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "flashbev.h"
#include "flashsca.h"
#include "flashbev_membench.h"

static int fail(const char *what) { fprintf(stderr, "FAIL %s\n", what); return 1; }

int main(void)
{
    float z[8];
    int k;
    flashbev_features f;
    flashbev_bev_grid_spec g;
    flashbev_z_bins zb;
    flashsca_value v;
    int64_t wg = 0;
    int32_t thr = 0, lds = 0, a = 0, b = 0;

    for (k = 0; k < 8; ++k) z[k] = -4.5f + (float)k;
    if (flashbev_abi_version() != FLASHBEV_ABI_VERSION) return fail("abi version");
    if (strcmp(flashbev_status_string(FLASHBEV_OK), "ok") != 0) return fail("status string");

    memset(&f, 0, sizeof f);
    f.dtype = FLASHBEV_F32; f.B = 1; f.N = 6; f.H = 32; f.W = 88; f.C = 80;
    f.img_h = 256; f.img_w = 704;
    g.x_min = -50.0f; g.dx = 0.5f; g.X = 200; g.y_min = -50.0f; g.dy = 0.5f; g.Y = 200;
    g.depth_eps = 1e-5f; g.reduce = FLASHBEV_REDUCE_VALID_MEAN;
    zb.z = z; zb.Z = 8;
    if (flashbev_launch_info(&f, &g, &zb, &wg, &thr, &lds, &a, &b) != FLASHBEV_OK || wg <= 0)
        return fail("launch info");
    if (flashbev_backward_launch_info(&f, &g, &zb, &wg, &thr, &lds, &a, &b) != FLASHBEV_OK)
        return fail("backward launch info");
    /* argument errors come back before any HIP call */
    if (flashbev_sample_vt(NULL, NULL, &g, &zb, NULL, NULL) != FLASHBEV_ERR_NULLPTR)
        return fail("null features");
    f.dtype = 7;
    if (flashbev_sample_vt(&f, NULL, &g, &zb, NULL, NULL) != FLASHBEV_ERR_DTYPE)
        return fail("dtype");

    memset(&v, 0, sizeof v);
    v.dtype = FLASHBEV_F32; v.B = 1; v.N = 6; v.C = 256; v.heads = 8; v.L = 1;
    v.level_h[0] = 116; v.level_w[0] = 200; v.img_h = 900; v.img_w = 1600;
    zb.Z = 4;
    if (flashsca_launch_info(&v, &g, &zb, 8, &wg, &thr, &lds, &a, &b) != FLASHBEV_OK || wg <= 0)
        return fail("sca launch info");
    if (flashsca_backward_launch_info(&v, &g, &zb, 8, &wg, &thr, &lds, &a, &b) != FLASHBEV_OK)
        return fail("sca backward launch info");
    if (flashsca_forward(&v, NULL, &g, &zb, 6, NULL, NULL, NULL, NULL) != FLASHBEV_ERR_SHAPE)
        return fail("sca P not a multiple of Z");
    if (flashbev_membench_stream(NULL, 0, 1, NULL, NULL) >= 0) return fail("membench null");
    printf("headers ok\n");
    return 0;
}
"""


def test_headers_compile_as_c99_and_link(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not found")
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM)
    exe = str(tmp_path / "abi")
    libdir = os.path.dirname(fb.library_path())
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I" + os.path.join(ROOT, "include"), str(src), "-o", exe,
                    fb.library_path(), membench._LIB_PATH, "-Wl,-rpath," + libdir],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr + r.stdout
    assert "headers ok" in r.stdout
