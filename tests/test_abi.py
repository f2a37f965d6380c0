"""The C-ABI boundary without a GPU: the library loads, exports exactly the
entry points include/solfp4.h declares, and rejects bad arguments on the host
before any HIP call."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

import paper_2604_06916_amd as sol

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "solfp4.h")

OK, EINVAL, ESHAPE, EALIGN, EWORKSPACE, EHIP = 0, -1, -2, -3, -4, -5

# fake device addresses: never dereferenced, because every call below fails
# validation on the host first
P = ctypes.c_void_p(0x7F0000000000)
P2 = ctypes.c_void_p(0x7F0000100000)
P3 = ctypes.c_void_p(0x7F0000200000)
MIS = ctypes.c_void_p(0x7F0000000008)   # 8-byte aligned only
NULL = None
S = None                                  # null stream


def declared_functions():
    text = open(HEADER).read()
    return re.findall(r"SOLFP4_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)


def test_header_declares_the_entry_points():
    names = declared_functions()
    assert sorted(names) == sorted(sol.EXPORTED)
    assert {"nvfp4_quantize", "nvfp4_gemm", "nvfp4_linear"} <= set(names)


def test_library_exports_every_declared_symbol():
    for name in declared_functions():
        assert getattr(sol.lib, name) is not None


@pytest.mark.skipif(shutil.which("nm") is None, reason="nm not available")
def test_library_exports_nothing_else():
    out = subprocess.run(["nm", "-D", "--defined-only", sol.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    funcs = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert funcs == set(declared_functions())


def test_strerror_and_version():
    texts = {c: sol.lib.solfp4_strerror(c) for c in (OK, EINVAL, ESHAPE, EALIGN, EWORKSPACE, EHIP, 7)}
    assert all(texts.values())
    assert len(set(texts.values())) == len(texts)
    assert sol.lib.solfp4_version() >= 100


def test_workspace_queries():
    q = sol.nvfp4_quantize_workspace_bytes
    assert q(0, 0) >= 4 and q(128, 1152) >= 4 and q(10 ** 6, 4096) <= 4096 * 4
    assert q(-1, 16) == 0 and q(4, 24) == 0
    L = sol.nvfp4_linear_workspace_bytes
    G = sol.nvfp4_gemm_workspace_bytes
    for M, N, K in [(1, 1, 16), (128, 1152, 1152), (18432, 3072, 3072), (26574, 2432, 9728),
                    (18432, 3072, 12288)]:
        assert L(M, N, K) >= M * K // 2 + M * K // 16 + 4 + q(M, K) + G(M, N, K)
    assert L(-1, 16, 16) == 0 and L(3, 8, 40) == 0 and L(3, -8, 16) == 0
    assert G(-1, 16, 16) == 0 and G(3, 8, 40) == 0 and G(3, 8, 1 << 24) == 0


def test_gemm_workspace_plan():
    """Which shapes split their last round's tiles (or those tiles'
    128 x 128 quadrants) into two K halves, and the workspace that takes (an
    8-byte slot per split tile or quadrant, 256-byte aligned, then two FP32
    partial tiles per tile: 256 KB each for 256 x 256 tiles, 64 KB for
    128 x 128 ones and for quadrants).  Without a GPU the CU count is
    MI355X's 256."""
    G = sol.nvfp4_gemm_workspace_bytes

    def bytes_for(rem, part=256 * 256 * 4):
        return (rem * 8 + 255) // 256 * 256 + rem * 2 * part

    def small_bytes_for(rem):
        return bytes_for(rem, 128 * 128 * 4)

    def quad_bytes_for(rem):
        return small_bytes_for(4 * rem)
    # FLUX.1 layers, 18432 tokens: 2592, 864, 3456 and 864 tiles of 256 x 256;
    # a last round of 32 tiles runs as 128 quadrants, each in two K halves
    assert G(18432, 9216, 3072) == quad_bytes_for(2592 % 256)
    assert G(18432, 3072, 3072) == bytes_for(864 % 256)
    assert G(18432, 12288, 3072) == bytes_for(3456 % 256)
    assert G(18432, 3072, 12288) == bytes_for(864 % 256)
    # whole rounds, remainders too large to split in two within one round,
    # too little K to gain, and shapes on other kernels or tile sizes
    assert G(4096, 4096, 4096) == 0            # 256 tiles
    assert G(26574, 7296, 2432) == 0           # 3016 tiles: 200 left over
    assert G(18432, 3072, 512) == 0            # 4 K stages
    assert G(8192, 5600, 2240) == 0            # 704 tiles: 192 left over
    assert G(8192, 36, 48) == 0                # K % 32 == 16: shared-conversion kernel
    # a last round of at most 64 tiles runs as whole quadrants, without a
    # workspace, when it has more than 32 tiles or fewer than 16 K stages;
    # 8 to 32 tiles of at least 16 stages split their quadrants
    assert G(4352, 4200, 1440) == 0            # 289 tiles: 33 left over
    assert G(4352, 4096, 1536) == 0            # 272 tiles: 12 K stages
    assert G(8192, 2240, 2240) == quad_bytes_for(32)    # 288 tiles, 18 K stages
    assert G(26574, 2432, 9728) == quad_bytes_for(16)   # 1040 tiles
    # K % 128 == 64 (a half last stage) splits too: the split (or the
    # quadrants) is what makes the lane kernel worth taking over the shared
    # one there
    assert G(8192, 6720, 2240) == bytes_for(864 % 256)
    # 128 x 128 tiles split as well, given enough K stages: 72 tiles of 24
    # and of 36 stages, and 72 of 18 (a half last stage) do
    assert G(384, 3072, 3072) == small_bytes_for(72)
    assert G(256, 4608, 4608) == small_bytes_for(72)
    assert G(512, 2240, 2240) == small_bytes_for(72)
    # fewer tokens with K % 128 == 0 run on 64 x 64 tiles, which never split
    assert G(128, 1152, 1152) == 0 and G(128, 3072, 3072) == 0 and G(128, 1152, 4608) == 0
    assert G(0, 3072, 3072) == 0 and G(18432, 0, 3072) == 0


def quant(x=P, rows=4, K=32, codes=P2, scales=P3, gs=P, ws=P, wsb=4096):
    return sol.lib.nvfp4_quantize(x, rows, K, codes, scales, gs, ws, wsb, S)


def test_quantize_rejects_bad_arguments():
    assert quant(rows=-1) == EINVAL
    assert quant(K=-16) == EINVAL
    assert quant(K=24) == ESHAPE
    assert quant(K=1 << 31) == ESHAPE
    assert quant(x=NULL) == EINVAL
    assert quant(codes=NULL) == EINVAL
    assert quant(scales=NULL) == EINVAL
    assert quant(gs=NULL) == EINVAL
    assert quant(ws=NULL) == EINVAL
    assert quant(x=MIS) == EALIGN
    assert quant(codes=MIS) == EALIGN
    assert quant(gs=MIS) == EALIGN
    assert quant(wsb=0) == EWORKSPACE


def test_two_pass_quantize_rejects_bad_arguments():
    amax = lambda x=P, rows=4, K=32, ws=P, wsb=4096: sol.lib.nvfp4_quantize_amax(x, rows, K, ws, wsb, S)
    enc = lambda x=P, rows=4, K=32, codes=P2, scales=P3, gs=P, ws=P, wsb=4096: \
        sol.lib.nvfp4_quantize_encode(x, rows, K, codes, scales, gs, ws, wsb, S)
    assert amax(rows=-1) == EINVAL and amax(K=24) == ESHAPE and amax(x=NULL) == EINVAL
    assert amax(ws=NULL) == EINVAL and amax(x=MIS) == EALIGN and amax(ws=MIS) == EALIGN
    assert amax(wsb=0) == EWORKSPACE
    assert enc(rows=-1) == EINVAL and enc(K=24) == ESHAPE and enc(codes=NULL) == EINVAL
    assert enc(gs=NULL) == EINVAL and enc(scales=MIS) == EALIGN and enc(wsb=0) == EWORKSPACE


def gemm(ac=P, as_=P2, ag=P3, bc=P, bs=P2, bg=P3, bias=NULL, out=P, ws=NULL, wsb=0, M=8, N=8,
         K=32):
    return sol.lib.nvfp4_gemm(ac, as_, ag, bc, bs, bg, bias, out, ws, wsb, M, N, K, S)


def test_gemm_rejects_bad_arguments():
    assert gemm(M=-1) == EINVAL
    assert gemm(N=-1) == EINVAL
    assert gemm(K=-16) == EINVAL
    assert gemm(K=40) == ESHAPE
    assert gemm(M=1 << 31) == ESHAPE
    assert gemm(out=NULL) == EINVAL
    assert gemm(ag=NULL) == EINVAL
    assert gemm(bc=NULL) == EINVAL
    assert gemm(as_=MIS) == EALIGN
    assert gemm(bias=MIS) == EALIGN
    assert gemm(out=MIS) == EALIGN
    # a workspace is optional, but one that is passed must be aligned and
    # large enough for the shape's split
    big = dict(M=18432, N=3072, K=12288)
    need = sol.nvfp4_gemm_workspace_bytes(**big)
    assert need > 0
    assert gemm(ws=MIS, wsb=need, **big) == EALIGN
    assert gemm(ws=P, wsb=need - 1, **big) == EWORKSPACE
    assert gemm(ws=P, wsb=need - 1, out=NULL, **big) == EINVAL
    # nothing to compute: valid, and no HIP call is made
    assert gemm(M=0, out=NULL) == OK
    assert gemm(N=0, out=NULL) == OK


def linear(x=P, wc=P2, ws_=P3, wg=P, bias=NULL, out=P2, ws=P3, wsb=1 << 20, M=8, N=8, K=32):
    return sol.lib.nvfp4_linear(x, wc, ws_, wg, bias, out, ws, wsb, M, N, K, S)


def test_linear_rejects_bad_arguments():
    big = dict(M=18432, N=3072, K=12288)
    need = sol.nvfp4_linear_workspace_bytes(**big)
    assert need > sol.nvfp4_linear_workspace_bytes(18432, 3072, 512)
    assert linear(wsb=need - 1, **big) == EWORKSPACE
    assert linear(M=-1) == EINVAL
    assert linear(K=20) == ESHAPE
    assert linear(ws=NULL) == EINVAL
    assert linear(ws=MIS) == EALIGN
    assert linear(wsb=16) == EWORKSPACE
    assert linear(x=NULL) == EINVAL
    assert linear(wc=NULL) == EINVAL
    assert linear(wg=NULL) == EINVAL
    assert linear(bias=MIS) == EALIGN
    assert linear(out=MIS) == EALIGN


def test_gemm_rejects_sizes_beyond_tile_addressing():
    assert gemm(K=1 << 24) == ESHAPE
    assert linear(K=1 << 24) == ESHAPE
    assert gemm(N=1 << 22) == ESHAPE
    assert linear(N=1 << 22) == ESHAPE


def test_mx_workspace_query():
    L = sol.mxfp4_linear_workspace_bytes
    for M, K in [(1, 32), (128, 1152), (18432, 3072), (26574, 9728)]:
        assert L(M, K) >= M * K // 2 + M * K // 32
    assert L(0, 0) > 0
    assert L(-1, 32) == 0 and L(3, 48) == 0


def mxq(x=P, rows=4, K=64, codes=P2, scales=P3):
    return sol.lib.mxfp4_quantize(x, rows, K, codes, scales, S)


def test_mx_quantize_rejects_bad_arguments():
    assert mxq(rows=-1) == EINVAL
    assert mxq(K=-32) == EINVAL
    assert mxq(K=48) == ESHAPE          # a multiple of 16 but not of 32
    assert mxq(K=1 << 31) == ESHAPE
    assert mxq(x=NULL) == EINVAL
    assert mxq(codes=NULL) == EINVAL
    assert mxq(scales=NULL) == EINVAL
    assert mxq(x=MIS) == EALIGN
    assert mxq(scales=MIS) == EALIGN
    # nothing to encode: valid, and no HIP call is made
    assert mxq(rows=0, x=NULL, codes=NULL, scales=NULL) == OK


def mxgemm(ac=P, as_=P2, bc=P, bs=P2, bias=NULL, out=P3, M=8, N=8, K=64):
    return sol.lib.mxfp4_gemm(ac, as_, bc, bs, bias, out, M, N, K, S)


def test_mx_gemm_rejects_bad_arguments():
    assert mxgemm(M=-1) == EINVAL
    assert mxgemm(K=-32) == EINVAL
    assert mxgemm(K=16) == ESHAPE
    assert mxgemm(K=1 << 24) == ESHAPE
    assert mxgemm(M=1 << 31) == ESHAPE
    assert mxgemm(N=1 << 22) == ESHAPE
    assert mxlinear(N=1 << 22) == ESHAPE
    assert mxgemm(out=NULL) == EINVAL
    assert mxgemm(bs=NULL) == EINVAL
    assert mxgemm(ac=MIS) == EALIGN
    assert mxgemm(bias=MIS) == EALIGN
    assert mxgemm(M=0, out=NULL) == OK


def mxlinear(x=P, wc=P2, ws_=P3, bias=NULL, out=P2, ws=P3, wsb=1 << 20, M=8, N=8, K=64):
    return sol.lib.mxfp4_linear(x, wc, ws_, bias, out, ws, wsb, M, N, K, S)


def test_mx_linear_rejects_bad_arguments():
    assert mxlinear(M=-1) == EINVAL
    assert mxlinear(K=80) == ESHAPE
    assert mxlinear(ws=NULL) == EINVAL
    assert mxlinear(ws=MIS) == EALIGN
    assert mxlinear(wsb=16) == EWORKSPACE
    assert mxlinear(x=NULL) == EINVAL
    assert mxlinear(wc=NULL) == EINVAL
    assert mxlinear(out=MIS) == EALIGN
