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
