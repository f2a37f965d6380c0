"""The benchmark's host-side contract, without a GPU: more than one GPU is
refused with a message, and the CPU-oracle baseline leg reports the fields
the JSON line carries."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_cpu_baseline_leg_on_a_tiny_sample():
    pytest.importorskip("threadpoolctl")
    sys.path.insert(0, ROOT)
    import bench
    from workloads import WORKLOADS
    cb = bench.cpu_baseline(WORKLOADS["single-1152"], rows=8, wrows=16)
    assert cb["kind"] == "oracle" and cb["unit"] == "TFLOP/s"
    assert cb["value"] > 0 and cb["cores"] >= 1
    assert "min(8, M) activation rows x min(16, N) weight rows" in cb["sample"]
    assert cb["cpu"] and cb["blas"]


def test_cpu_baseline_clips_the_sample_to_the_layer():
    # a weight sample larger than a layer's N (the default sample against the
    # 3072-row FLUX out-projection) is clipped, not drawn past the tensor
    pytest.importorskip("threadpoolctl")
    sys.path.insert(0, ROOT)
    import bench
    from workloads import WORKLOADS
    cb = bench.cpu_baseline(WORKLOADS["single-1152"], rows=4, wrows=1300)
    assert cb["value"] > 0


def test_row_range_outside_the_tensor_is_rejected():
    sys.path.insert(0, ROOT)
    from workloads import draw_activations, draw_weights
    with pytest.raises(ValueError):
        draw_weights(300, 32, 0.02, seed=1, row_range=(0, 400))
    with pytest.raises(ValueError):
        draw_activations("normal", 300, 32, seed=1, row_range=(10, 5))


def test_paper_context_is_marked_not_comparable():
    sys.path.insert(0, ROOT)
    import bench
    ctx = bench.PAPER_CONTEXT
    assert ctx["comparable"] is False and "B200" in ctx["hardware"]
    for model, (naive, ours) in ctx["rollout_s"].items():
        assert abs(naive / ours - ctx["rollout_speedup"][model]) < 0.01
    for model, (naive, ours) in ctx["end_to_end_s"].items():
        assert abs(naive / ours - ctx["end_to_end_speedup"][model]) < 0.01


def test_roofline_kernel_name_follows_the_dispatch():
    """The name bench.py reports for the NVFP4 GEMM roofline follows the
    library's kernel choice (the CU count is MI355X's 256 without a GPU)."""
    import bench
    lane, shared = "nvfp4_gemm_lane_kernel", "nvfp4_gemm_kernel"
    for M, N, K in [(18432, 9216, 3072), (18432, 3072, 12288), (8192, 2240, 5600)]:
        assert bench.nvfp4_gemm_kernel_name(M, N, K) == lane
    assert bench.nvfp4_gemm_kernel_name(8192, 5600, 2240) == shared   # whole rounds, no split
    assert bench.nvfp4_gemm_kernel_name(8192, 2240, 2240) == lane     # split last round
    assert bench.nvfp4_gemm_kernel_name(300, 260, 2240) == lane       # 128 x 128 tiles
    assert bench.nvfp4_gemm_kernel_name(300, 260, 48) == shared       # K % 32 == 16
    assert bench.nvfp4_gemm_kernel_name(128, 1152, 1152) == "nvfp4_gemm_wavek_kernel"
    assert bench.nvfp4_gemm_kernel_name(256, 3072, 1152) == "nvfp4_gemm_small_kernel"


def test_kernel_source_hashes_cover_every_include():
    """A committed profile goes stale when its kernel's source or any
    header it includes changes: the hashed file list names every local
    include of each source."""
    import re
    import bench
    for src, files in bench.KERNEL_SOURCES.items():
        text = open(os.path.join(bench.CSRC, src)).read()
        includes = set(re.findall(r'#include "([^"]+)"', text))
        for h in includes - {"kernels.h", "solfp4.h"}:
            assert h in files, (src, h)
            sub = set(re.findall(r'#include "([^"]+)"', open(os.path.join(bench.CSRC, h)).read()))
            assert sub <= set(files) | {"kernels.h", "solfp4.h"}, (h, sub)


def test_every_profile_names_the_sources_it_was_taken_on(tmp_path, monkeypatch):
    """Every committed profile summary carries a `kernel_sources` line that
    bench.py checks against the current sources, so a stale profile shows
    up as stale in the bench line rather than as current."""
    import bench
    status = bench.profile_status()
    names = [n for n in os.listdir(bench.PROFILES) if n.endswith(".txt")]
    assert names and set(status) == set(names)
    assert "unhashed" not in status.values(), status
    # the check itself: a changed source turns a profile stale
    good = " ".join(f"{s}={bench.kernel_source_hash(s)}" for s in ("gemm.hip", "quantize.hip"))
    (tmp_path / "a.txt").write_text(f"# x\nkernel_sources {good}\n")
    (tmp_path / "b.txt").write_text("# x\nkernel_sources gemm.hip=0000000000000000\n")
    (tmp_path / "c.txt").write_text("# no tag\n")
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.profile_status() == {"a.txt": "current", "b.txt": "stale", "c.txt": "unhashed"}


def test_gpu_state_reads_power_and_clocks(monkeypatch):
    # an amd-smi reply of the shape `amd-smi metric -p -c --json` prints
    # (values made up), and replies it cannot use
    sys.path.insert(0, ROOT)
    import json
    import types

    import bench
    reply = {"gpu_data": [{"gpu": 0,
                           "power": {"socket_power": {"value": 700, "unit": "W"}, "gfx_voltage": "N/A"},
                           "clock": {"gfx_0": {"clk": {"value": 2100, "unit": "MHz"}},
                                     "gfx_1": {"clk": {"value": 2300, "unit": "MHz"}},
                                     "gfx_2": {"clk": "N/A"},
                                     "mem_0": {"clk": {"value": 2000, "unit": "MHz"}}}}]}
    monkeypatch.setattr(subprocess, "run",
                        lambda *a, **k: types.SimpleNamespace(stdout=json.dumps(reply), returncode=0))
    assert bench.gpu_state() == {"socket_power_w": 700, "gfx_clk_mhz": [2100, 2200, 2300],
                                 "mem_clk_mhz": 2000}
    monkeypatch.setattr(subprocess, "run",
                        lambda *a, **k: types.SimpleNamespace(stdout="not json", returncode=1))
    assert bench.gpu_state() is None

    def missing(*a, **k):
        raise FileNotFoundError("amd-smi")
    monkeypatch.setattr(subprocess, "run", missing)
    assert bench.gpu_state() is None
