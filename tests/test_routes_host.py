"""The seeded route shapes (tests/route_shapes.py) meet every GEMM kernel,
tile size and the split last round, as the library plans them without a
GPU (256 compute units, as on MI355X)."""
import paper_2604_06916_amd as sol
from route_shapes import SHAPES


def test_route_shapes_meet_every_kernel():
    nv = {(p["kernel"], p["tile"]) for p in (sol.gemm_plan(*s) for s in SHAPES)}
    assert {("nvfp4_gemm_wavek_kernel", 32), ("nvfp4_gemm_small_kernel", 64),
            ("nvfp4_gemm_lane_kernel", 128), ("nvfp4_gemm_lane_kernel", 256),
            ("nvfp4_gemm_kernel", 256)} <= nv
    assert any(sol.gemm_plan(*s)["splits"] == 2 for s in SHAPES)
    mx = {(p["kernel"], p["tile"]) for p in (sol.gemm_plan(M, N, K - K % 32, sol.FORMAT_MXFP4)
                                              for M, N, K in SHAPES if K >= 32)}
    assert mx == {("mxfp4_gemm_wavek_kernel", 32), ("mxfp4_gemm_kernel", 64),
                  ("mxfp4_gemm_kernel", 128), ("mxfp4_gemm_kernel", 256)}


def test_last_round_plan_boundaries():
    """Where the last round of 256 x 256 tiles runs as 128 x 128 quadrants
    (at most 64 tiles, a quarter of MI355X's 256 CUs), where those quadrants
    split in K halves (at most 32 tiles and at least 16 K stages of 128),
    and where whole tiles split instead (65 to 128 tiles).  The plan counts
    the workgroups of both launches; MXFP4 never splits K."""
    def plan(M, N, K, fmt=sol.FORMAT_NVFP4, ws=True):
        p = sol.gemm_plan(M, N, K, fmt, with_workspace=ws)
        assert p["tile"] == 256
        return p["workgroups"], p["splits"]
    # 288 tiles, 32 over: quadrants in K halves from 16 stages, whole below
    assert plan(4096, 4608, 2048) == (256 + 8 * 32, 2)
    assert plan(4096, 4608, 2048, ws=False) == (256 + 4 * 32, 1)
    assert plan(4096, 4608, 1920) == (256 + 4 * 32, 1)
    # 289 and 320 tiles: 33 and 64 over, whole quadrants
    assert plan(4352, 4352, 3072) == (256 + 4 * 33, 1)
    assert plan(4096, 5120, 3072) == (256 + 4 * 64, 1)
    # 321 tiles: 65 over, each of them in two K halves
    assert plan(768, 27392, 3072) == (256 + 2 * 65, 2)
    # whole rounds, and fewer tiles than CUs: one launch of whole tiles
    assert plan(4096, 4096, 3072) == (256, 1)
    assert plan(4096, 3840, 3072) == (240, 1)
    mx = sol.FORMAT_MXFP4
    assert plan(4096, 4608, 2048, mx) == (256 + 4 * 32, 1)
    assert plan(4096, 5120, 3072, mx) == (256 + 4 * 64, 1)
    assert plan(768, 27392, 3072, mx) == (321, 1)
