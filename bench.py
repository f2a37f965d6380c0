#!/usr/bin/env python3
"""Benchmark of the NVFP4 linear-layer hot path on one MI355X.

One step = every linear of one DiT block of the chosen workload (default: the
FLUX.1-12B-like layers, M = 4 x (4096 + 512) = 18432 tokens; QKV 3072->9216,
out 3072->3072, MLP 3072->12288->3072), each as
    nvfp4_quantize(W)            weight re-quantization (once per update)
    nvfp4_quantize(X)            activation amax + encode passes
    nvfp4_gemm(Xq, Wq, bias)     block-scaled FP4 GEMM, BF16 out
which is exactly the launch sequence of nvfp4_quantize(W) + nvfp4_linear for
these sizes; the two passes of the activation quantize are also timed one at
a time (nvfp4_quantize_amax, nvfp4_quantize_encode).  Inputs are synthetic (seeded, from
workloads/) and resident in HBM before the timed region.  "workloads"
repeats the step for the other configurations (the SANA-1.6B-like and
SD3.5-Large-like layers, each with its own GEMM roofline) and holds the
launch-bound 128-token layer; "mxfp4" runs the same FLUX layers through the
MXFP4 variant; "graphs" times weight re-quantization and the per-step
linears as replayed HIP graphs; "stage1" runs the synthetic Stage-1 rollout
loop (paper_2604_06916_amd/stage1.py) with BF16, NVFP4 and MXFP4 linears.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X published dense peaks
PEAK_HBM_GBS = 8000.0
PEAK_FP16_MFMA_TFLOPS = 2500.0
PEAK_FP4_MFMA_TFLOPS = 10100.0
METRIC = "NVFP4 GEMM TFLOPS & % of FP4 MFMA peak; quantize GB/s & % HBM peak"
# MXFP4 quantize: 2 B read, 0.5 B codes + 1/32 B scales written per element
MX_QUANT_BYTES = 2.53125


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="flux-12b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-mxfp4", action="store_true", help="skip the MXFP4 variant")
    ap.add_argument("--no-graphs", action="store_true",
                    help="skip the graph-replay and small-layer measurements")
    ap.add_argument("--no-stage1", action="store_true", help="skip the synthetic Stage-1 rollouts")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other configurations (SANA-like, SD3.5-like, 128-token layer)")
    ap.add_argument("--no-vendor", action="store_true",
                    help="skip the vendor MXFP4 GEMM reference (it launches mxfp4_gemm once more per layer)")
    ap.add_argument("--cpu-rows", type=int, default=5120, help="oracle sample: activation rows")
    ap.add_argument("--cpu-wrows", type=int, default=5120, help="oracle sample: weight rows")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="after the benchmark, run a plain device-to-device copy of BYTES "
                         "three times (reference for HBM traffic counters)")
    return ap.parse_args()


CSRC = os.path.join(ROOT, "paper_2604_06916_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
PROFILED_WORKLOAD = "flux-12b"


def source_hash(*paths):
    import hashlib
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


# the files each kernel is built from (its source and the device headers it
# includes); a committed profile records their hash and goes stale with them
KERNEL_SOURCES = {
    "gemm.hip": ("gemm.hip", "device_common.h", "nvfp4_gemm_common.h"),
    "gemm_small.hip": ("gemm_small.hip", "device_common.h", "nvfp4_gemm_common.h"),
    "mx_gemm.hip": ("mx_gemm.hip", "device_common.h"),
    "quantize.hip": ("quantize.hip", "device_common.h"),
    "mx_quantize.hip": ("mx_quantize.hip", "device_common.h"),
}


def kernel_source_hash(source):
    return source_hash(*(os.path.join(CSRC, f) for f in KERNEL_SOURCES[source]))


def measured_traffic(summary, source):
    """HBM bytes per GEMM launch (FETCH_SIZE + WRITE_SIZE, scaled by a plain
    copy's reading of the same counters) from a committed counter summary of
    the FLUX layers, or None when the kernel source (or the device header it
    includes) changed since the counters were taken."""
    try:
        lines = open(os.path.join(PROFILES, summary)).read().splitlines()
    except OSError:
        return None
    kv = dict(l.split("=", 1) for l in lines if "=" in l and not l.startswith("#"))
    if kv.get("source_sha256_16") != kernel_source_hash(source):
        return None
    return float(kv["hbm_bytes_per_launch_avg"])


def profile_status():
    """Each committed profile summary under profiles/ with the kernel sources
    it was taken on (its `kernel_sources name=sha ...` line): "current" when
    every one of them still hashes the same, "stale" when any changed,
    "unhashed" when the file names none."""
    out = {}
    try:
        names = sorted(n for n in os.listdir(PROFILES) if n.endswith(".txt"))
    except OSError:
        return out
    for name in names:
        with open(os.path.join(PROFILES, name)) as f:
            tags = [l.split()[1:] for l in f if l.startswith("kernel_sources ")]
        if not tags:
            out[name] = "unhashed"
            continue
        pairs = [t.split("=", 1) for t in tags[0]]
        ok = all(src in KERNEL_SOURCES and kernel_source_hash(src) == sha for src, sha in pairs)
        out[name] = "current" if ok else "stale"
    return out


def nvfp4_gemm_kernel_name(M, N, K):
    """The kernel nvfp4_gemm launches for this shape, as the library reports
    it (solfp4_gemm_plan; a workspace is passed, as in the step)."""
    import paper_2604_06916_amd as sol
    return sol.gemm_plan(M, N, K)["kernel"]


def vendor_mxfp4(layers, bufs, steps):
    """The vendor library's MXFP4 GEMM (torch._scaled_mm on the ROCm stack)
    on the same quantized operands, for reference: its time per layer and
    the relative Frobenius difference of its output from mxfp4_gemm's.
    None when this torch build has no MXFP4 scaled matmul."""
    import torch

    import paper_2604_06916_amd as sol
    if not (hasattr(torch, "float4_e2m1fn_x2") and hasattr(torch, "float8_e8m0fnu")):
        return None
    res = []
    try:
        for L, B in zip(layers, bufs):
            a = B["xc"].view(torch.float4_e2m1fn_x2)
            b = B["wc"].view(torch.float4_e2m1fn_x2)
            sa = B["xs"].view(torch.float8_e8m0fnu)
            sb = B["ws"].view(torch.float8_e8m0fnu)
            ref = torch._scaled_mm(a, b.t(), scale_a=sa, scale_b=sb, out_dtype=torch.bfloat16)
            ours = sol.mxfp4_gemm(B["xc"], B["xs"], B["wc"], B["ws"])
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(steps):
                torch._scaled_mm(a, b.t(), scale_a=sa, scale_b=sb, out_dtype=torch.bfloat16)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            diff = ((ref.float() - ours.float()).norm() / ours.float().norm()).item()
            res.append({"vendor_gemm_us": round(ms * 1e3, 2),
                        "vendor_gemm_tflops": round(2.0 * L["M"] * L["N"] * L["K"] / (ms * 1e-3) / 1e12, 1),
                        "vendor_rel_diff": float(f"{diff:.3e}")})
            del ref, ours
    except (RuntimeError, TypeError) as e:      # no MXFP4 path in this build
        return [{"vendor_error": str(e)[:120]}]
    return res


def run_mxfp4(layers, steps, warmup, profiled, vendor=True):
    """Time the MXFP4 variant of the step on the same resident inputs: per
    layer mxfp4_quantize(W), mxfp4_quantize(X), mxfp4_gemm(+bias), each
    bracketed by HIP events on the stream the kernels are launched on."""
    import numpy as np
    import torch

    import paper_2604_06916_amd as sol
    dev = layers[0]["x"].device
    bufs = []
    for L in layers:
        M, N, K = L["M"], L["N"], L["K"]
        bufs.append(dict(
            wc=torch.empty((N, K // 2), dtype=torch.uint8, device=dev),
            ws=torch.empty((N, K // 32), dtype=torch.uint8, device=dev),
            xc=torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
            xs=torch.empty((M, K // 32), dtype=torch.uint8, device=dev)))

    def step(events=None):
        for i, (L, B) in enumerate(zip(layers, bufs)):
            e = events[i] if events is not None else None
            if e:
                e[0].record()
            sol.mxfp4_quantize(L["w"], B["wc"], B["ws"])
            if e:
                e[1].record()
            sol.mxfp4_quantize(L["x"], B["xc"], B["xs"])
            if e:
                e[2].record()
            sol.mxfp4_gemm(B["xc"], B["xs"], B["wc"], B["ws"], L["b"], L["out"])
            if e:
                e[3].record()

    for _ in range(warmup):
        step()
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in layers]
          for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        step(ev[s])
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) / steps * 1e3
    gemm_ms = xq_ms = 0.0
    per_layer = []
    for i, L in enumerate(layers):
        xqs = np.array([ev[s][i][1].elapsed_time(ev[s][i][2]) for s in range(steps)])
        gms = np.array([ev[s][i][2].elapsed_time(ev[s][i][3]) for s in range(steps)])
        xq, gm = float(np.mean(xqs)), float(np.mean(gms))
        gemm_ms += gm
        xq_ms += xq
        fl = 2.0 * L["M"] * L["N"] * L["K"]
        per_layer.append({"layer": L["name"], "gemm_us": round(gm * 1e3, 2),
                          "gemm_tflops": round(fl / (gm * 1e-3) / 1e12, 1),
                          "gemm_us_p10_p50_p90": [round(float(np.percentile(gms, q)) * 1e3, 2)
                                                  for q in (10, 50, 90)],
                          "quantize_x_us": round(xq * 1e3, 2),
                          "quantize_x_us_p10_p50_p90": [round(float(np.percentile(xqs, q)) * 1e3, 2)
                                                        for q in (10, 50, 90)]})
    flops = sum(2.0 * L["M"] * L["N"] * L["K"] for L in layers)
    gemm_tflops = flops / (gemm_ms * 1e-3) / 1e12
    vendor = vendor_mxfp4(layers, bufs, steps) if vendor else None
    for row, v in zip(per_layer, vendor or []):
        row.update(v)
    xq_bytes = sum(MX_QUANT_BYTES * L["M"] * L["K"] for L in layers)
    quant_gbs = xq_bytes / (xq_ms * 1e-3) / 1e9
    return {
        "operands": "MXFP4 (E2M1 + E8M0/32), v_mfma_scale_f32_32x32x64_f8f6f4, FP32 accumulate",
        "step_tflops": round(flops / (ms_per_step * 1e-3) / 1e12, 1),
        "ms_per_step": round(ms_per_step, 4),
        "gemm": {"kernel": "mxfp4_gemm_kernel", "achieved": round(gemm_tflops, 1),
                 "peak": PEAK_FP4_MFMA_TFLOPS, "unit": "TFLOP/s",
                 "frac": round(gemm_tflops / PEAK_FP4_MFMA_TFLOPS, 4),
                 "traffic": (measured_traffic("mxfp4_gemm_flux-12b_traffic.txt", "mx_gemm.hip")
                             if profiled else None),
                 "traffic_unit": "HBM bytes per launch (mean over the step's GEMMs)"},
        "quantize": {"kernel": "mxfp4_quantize_kernel (activations)",
                     "achieved_gbs": round(quant_gbs, 1), "bytes_per_element": MX_QUANT_BYTES,
                     "peak_gbs": PEAK_HBM_GBS, "frac_hbm": round(quant_gbs / PEAK_HBM_GBS, 4)},
        "time_split_ms": {"gemm": round(gemm_ms, 4), "quantize_x": round(xq_ms, 4)},
        "layers": per_layer,
    }


def run_graphs(layers, reps):
    """In-place weight re-quantization with graph replay on the bench layers:
    one graph re-quantizes every weight into its existing buffers (what runs
    after a policy update), one replays the per-step linears (activation
    quantize + GEMM); both captured once.  Returns replay and eager times."""
    import torch

    import paper_2604_06916_amd as sol

    def update():
        for L in layers:
            sol.nvfp4_quantize(L["w"], L["wc"], L["ws"], L["wa"], L["qws"])

    def linears():
        for L in layers:
            sol.nvfp4_quantize(L["x"], L["xc"], L["xs"], L["xa"], L["qws"])
            sol.nvfp4_gemm(L["xc"], L["xs"], L["xa"], L["wc"], L["ws"], L["wa"], L["b"], L["out"],
                           L["gws"])

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    g_up, g_lin = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_up):
        update()
    with torch.cuda.graph(g_lin):
        linears()
    torch.cuda.synchronize()
    n_w = sum(L["N"] * L["K"] for L in layers)
    up_ms = timed(g_up.replay)
    return {
        "requantize_graph_ms": round(up_ms, 4),
        "requantize_eager_ms": round(timed(update), 4),
        "requantize_gbs": round(4.5625 * n_w / (up_ms * 1e-3) / 1e9, 1),
        "weights_requantized": n_w,
        "linears_graph_ms": round(timed(g_lin.replay), 4),
        "linears_eager_ms": round(timed(linears), 4),
    }


def run_small_linear(reps):
    """The 128-token 1152 -> 1152 layer, launch-bound: nvfp4_linear per call,
    eager launches against one graph holding `batch` linears; the GEMM alone;
    the MXFP4 linear and GEMM graph-replayed the same way."""
    import numpy as np
    import torch

    import paper_2604_06916_amd as sol
    from workloads import ROLE_BIAS, ROLE_W, ROLE_X, WORKLOADS, draw_activations, draw_bias, \
        draw_weights, seed_for
    wl = WORKLOADS["single-1152"]
    layer = wl.layers[0]
    M, N, K = wl.M, layer.N, layer.K
    dev = torch.device("cuda:0")

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)
    x = to_dev(draw_activations(layer.x_dist, M, K, seed_for(wl.config_id, layer.index, ROLE_X)))
    w = to_dev(draw_weights(N, K, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_W)))
    b = to_dev(draw_bias(N, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_BIAS)))
    wc, ws, wa = sol.nvfp4_quantize(w)
    out = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    lws = torch.empty(sol.nvfp4_linear_workspace_bytes(M, N, K), dtype=torch.uint8, device=dev)
    batch = 50

    def lin():
        sol.nvfp4_linear(x, wc, ws, wa, b, out, lws)
    for _ in range(10):
        lin()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps * batch):
        lin()
    e1.record()
    torch.cuda.synchronize()
    eager_us = e0.elapsed_time(e1) / (reps * batch) * 1e3
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(batch):
            lin()
    g.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    graph_us = e0.elapsed_time(e1) / (reps * batch) * 1e3
    # the GEMM alone, graph-batched the same way
    xc, xs, xa = sol.nvfp4_quantize(x)
    gws = sol.nvfp4_gemm_workspace_bytes(M, N, K)
    gws = torch.empty(gws, dtype=torch.uint8, device=dev) if gws else None
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2):
        for _ in range(batch):
            sol.nvfp4_gemm(xc, xs, xa, wc, ws, wa, b, out, gws)
    g2.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        g2.replay()
    e1.record()
    torch.cuda.synchronize()
    gemm_us = e0.elapsed_time(e1) / (reps * batch) * 1e3
    # the MXFP4 linear (quantize + GEMM) and its GEMM alone, graph-batched alike
    mwc, mws = sol.mxfp4_quantize(w)
    mlws = torch.empty(sol.mxfp4_linear_workspace_bytes(M, K), dtype=torch.uint8, device=dev)
    mxc, mxs = sol.mxfp4_quantize(x)

    def graph_time(fn):
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            for _ in range(batch):
                fn()
        gr.replay()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            gr.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (reps * batch) * 1e3
    mx_lin_us = graph_time(lambda: sol.mxfp4_linear(x, mwc, mws, b, out, mlws))
    mx_gemm_us = graph_time(lambda: sol.mxfp4_gemm(mxc, mxs, mwc, mws, b, out))
    fl = 2.0 * M * N * K
    fused = K <= 512 and nvfp4_gemm_kernel_name(M, N, K) == "nvfp4_gemm_small_kernel"
    route = ("amax pass + GEMM quantizing the activations in the kernel" if fused
             else "amax pass + encode pass + GEMM")
    return {"layer": f"M={M} {K}->{N} nvfp4_linear (+bias)", "eager_us": round(eager_us, 2),
            "graph_us": round(graph_us, 2), "gemm_graph_us": round(gemm_us, 2),
            "gemm_kernel": nvfp4_gemm_kernel_name(M, N, K), "linear_launches": route,
            "graph_tflops": round(fl / (graph_us * 1e-6) / 1e12, 2),
            "mxfp4": {"linear_graph_us": round(mx_lin_us, 2), "gemm_graph_us": round(mx_gemm_us, 2),
                      "gemm_kernel": sol.gemm_plan(M, N, K, sol.FORMAT_MXFP4)["kernel"],
                      "linear_launches": "mxfp4_quantize + mxfp4_gemm"},
            "roofline": {"bound": "latency", "achieved": round(fl / (graph_us * 1e-6) / 1e12, 2),
                         "peak": PEAK_FP16_MFMA_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(fl / (graph_us * 1e-6) / 1e12 / PEAK_FP16_MFMA_TFLOPS, 5),
                         "note": "1.1 MB of operands and 0.34 GFLOP: launch and memory round "
                                 "trips bound this layer, not HBM bandwidth or the matrix cores"}}


def run_stage1():
    """Synthetic Stage-1 rollouts (8 blocks of the FLUX-like width, 8 rollouts
    x 4608 tokens, 4 Euler steps, reward, top/bottom selection) with every
    linear on each backend.  Eager, with HIP events around every op: the
    linears' time, TFLOP/s and share, and the other ops' time by kind (time
    covered by no event is the GPU waiting for the host).  Then the same
    rollout as one captured Euler step replayed per step (no host launch
    cost): the rollout time the speed-ups are quoted on."""
    import torch

    from paper_2604_06916_amd import stage1 as G
    cfg = G.Stage1Config()
    dev = torch.device("cuda:0")
    model = G.make_weights(cfg, dev)
    x0 = G.initial_latents(cfg, dev)
    u = G.reward_direction(cfg)
    lin_flops = G.linear_flops(cfg)
    out = {"config": {"blocks": cfg.blocks, "hidden": cfg.hidden, "heads": cfg.heads,
                      "mlp": cfg.mlp, "rollouts": cfg.rollouts, "tokens": cfg.tokens,
                      "euler_steps": cfg.steps, "keep": cfg.keep,
                      "attention": "BF16, torch fused attention",
                      "linear_flops": lin_flops, "attention_flops": G.attention_flops(cfg)}}
    for backend in G.BACKENDS:
        runner = G.Runner(cfg, model, backend, dev)
        warm = G.Stage1Config(**{**cfg.__dict__, "steps": 1})
        runner.cfg = warm
        runner.rollout(x0)
        runner.cfg = cfg
        torch.cuda.synchronize()
        runner.linear_events = []
        runner.op_events = {}
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        x = runner.rollout(x0)
        r = G.rewards(cfg, x, u)
        e1.record()
        torch.cuda.synchronize()
        total = e0.elapsed_time(e1)
        lin = sum(a.elapsed_time(b) for a, b in runner.linear_events)
        ops = {k: round(sum(a.elapsed_time(b) for a, b in v), 2) for k, v in runner.op_events.items()}
        top, bottom = G.select_rollouts(r.cpu().numpy(), cfg.keep)
        rec = {"rollout_ms_eager": round(total, 2), "linear_ms": round(lin, 2),
               "linear_tflops": round(lin_flops / (lin * 1e-3) / 1e12, 1),
               "linear_share": round(lin / total, 4),
               "other_ms": round(total - lin, 2), "other_ms_by_op": ops,
               "host_gaps_ms": round(total - lin - sum(ops.values()), 2),
               "top": [int(i) for i in top], "bottom": [int(i) for i in bottom]}
        runner.linear_events = None
        runner.op_events = None
        try:
            xs = x0.clone()
            g = runner.capture_step(xs)
            times = []
            for _ in range(2):
                xs.copy_(x0)
                torch.cuda.synchronize()
                e0.record()
                for _ in range(cfg.steps):
                    g.replay()
                e1.record()
                torch.cuda.synchronize()
                times.append(e0.elapsed_time(e1))
            rec["rollout_ms"] = round(min(times), 2)
            rec["rollout_graph_matches_eager"] = bool(torch.equal(xs.view(torch.int16), x.view(torch.int16)))
            del g, xs
        except RuntimeError as e:        # capture not possible in this build: eager time only
            rec["rollout_ms"] = rec["rollout_ms_eager"]
            rec["graph_error"] = str(e)[:120]
        out[backend] = rec
        del runner
        torch.cuda.empty_cache()
    for backend in ("nvfp4", "mxfp4"):
        out[backend]["linear_speedup_vs_bf16"] = round(out["bf16"]["linear_ms"] / out[backend]["linear_ms"], 3)
        out[backend]["rollout_speedup_vs_bf16"] = round(out["bf16"]["rollout_ms"] / out[backend]["rollout_ms"], 3)
    return out


# The paper's own rollout timings (Table 5; 8x NVIDIA B200, NVFP4 exploration
# stage through NVIDIA Transformer Engine): whole RL iterations of the real
# models, quoted as context only -- no kernel figure here is comparable.
PAPER_CONTEXT = {
    "source": "Table 5 (training efficiency), Sec. 4.1 (hardware)",
    "hardware": "8x NVIDIA B200",
    "comparable": False,
    "rollout_s": {"FLUX.1": [184, 79], "SD3.5-Large": [451, 187], "SANA": [65, 46]},
    "rollout_speedup": {"FLUX.1": 2.33, "SD3.5-Large": 2.41, "SANA": 1.41},
    "end_to_end_s": {"FLUX.1": [274, 169], "SD3.5-Large": [691, 427], "SANA": [95, 76]},
    "end_to_end_speedup": {"FLUX.1": 1.62, "SD3.5-Large": 1.61, "SANA": 1.25},
    "note": "naive scaled rollout vs the two-stage framework (NVFP4 stage 1 + BF16 stage 2)",
}


def cpu_model():
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, rows, wrows):
    """The CPU oracle on a bounded sample of the same step: per layer, `rows`
    activation rows and `wrows` weight rows at full K (each clipped to the
    layer's size), quantize both and the
    float64 GEMM; throughput in the metric's unit (TFLOP/s of 2 m n K)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle.nvfp4 as O
    from workloads import ROLE_BIAS, ROLE_W, ROLE_X, draw_activations, draw_bias, draw_weights, seed_for
    flops, secs = 0.0, 0.0
    for layer in wl.layers:
        m, n = min(rows, wl.M), min(wrows, layer.N)
        xb = draw_activations(layer.x_dist, wl.M, layer.K, seed_for(wl.config_id, layer.index, ROLE_X),
                              row_range=(0, m))
        wb = draw_weights(layer.N, layer.K, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_W),
                          row_range=(0, n))
        bias = draw_bias(layer.N, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_BIAS))[:n]
        t0 = time.perf_counter()
        wq = O.nvfp4_quantize_ref(wb)
        xq = O.nvfp4_quantize_ref(xb)
        out = O.bf16_output(O.nvfp4_gemm_ref(*xq, *wq, bias))
        secs += time.perf_counter() - t0
        flops += 2.0 * m * n * layer.K
        assert out.shape == (m, n)
    pools = threadpool_info()
    blas_threads = max([i.get("num_threads", 1) for i in pools] or [1])
    blas = sorted({f"{i.get('internal_api', '?')} {i.get('version', '')}".strip()
                   for i in pools if i.get("user_api") == "blas"})
    return {
        "value": flops / secs / 1e12,
        "unit": "TFLOP/s",
        "cores": int(blas_threads),
        "kind": "oracle",
        "cpu": cpu_model(),
        "blas": ", ".join(blas) or "unknown",
        "sample": (f"per layer min({rows}, M) activation rows x min({wrows}, N) weight rows at "
                   f"full K: oracle "
                   f"quantize of both (numpy float32, 1 thread) + float64 GEMM (BLAS, "
                   f"{blas_threads} threads); {secs:.1f} s"),
    }


def gpu_state():
    """Socket power and clocks of GPU 0 as amd-smi reports them (a child
    process, 30 s limit); None where amd-smi is missing or says nothing.
    amd-smi samples are coarse: they do not show the clock of a kernel of a
    few hundred microseconds (the counter profile records that)."""
    import shutil
    import subprocess
    exe = shutil.which("amd-smi") or "/opt/rocm/bin/amd-smi"
    try:
        p = subprocess.run([exe, "metric", "-g", "0", "-p", "-c", "--json"], capture_output=True,
                           text=True, timeout=30)
        data = json.loads(p.stdout)
    except (OSError, subprocess.SubprocessError, ValueError):
        return None
    gpus = data.get("gpu_data", data) if isinstance(data, dict) else data
    if not isinstance(gpus, list) or not gpus or not isinstance(gpus[0], dict):
        return None

    def num(v):
        v = v.get("value") if isinstance(v, dict) else v
        return v if isinstance(v, (int, float)) else None

    g = gpus[0]
    power = num((g.get("power") or {}).get("socket_power"))
    clocks = g.get("clock") or {}
    gfx = [num((c or {}).get("clk")) for k, c in clocks.items() if k.startswith("gfx_")]
    gfx = [v for v in gfx if v is not None]
    mem = [num((c or {}).get("clk")) for k, c in clocks.items() if k.startswith("mem_")]
    mem = [v for v in mem if v is not None]
    return {"socket_power_w": power,
            "gfx_clk_mhz": [min(gfx), round(sum(gfx) / len(gfx)), max(gfx)] if gfx else None,
            "mem_clk_mhz": mem[0] if mem else None}


def make_layers(wl, dev):
    """Device buffers of every layer of a workload: seeded BF16 X, W and bias,
    and the outputs and workspaces the step writes."""
    import numpy as np
    import torch

    import paper_2604_06916_amd as sol
    from workloads import ROLE_BIAS, ROLE_W, ROLE_X, draw_activations, draw_bias, draw_weights, seed_for

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    layers = []
    for layer in wl.layers:
        M, N, K = wl.M, layer.N, layer.K
        gws = sol.nvfp4_gemm_workspace_bytes(M, N, K)
        layers.append(dict(
            x=to_dev(draw_activations(layer.x_dist, M, K, seed_for(wl.config_id, layer.index, ROLE_X))),
            w=to_dev(draw_weights(N, K, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_W))),
            b=to_dev(draw_bias(N, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_BIAS))),
            wc=torch.empty((N, K // 2), dtype=torch.uint8, device=dev),
            ws=torch.empty((N, K // 16), dtype=torch.uint8, device=dev),
            wa=torch.empty(1, dtype=torch.float32, device=dev),
            xc=torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
            xs=torch.empty((M, K // 16), dtype=torch.uint8, device=dev),
            xa=torch.empty(1, dtype=torch.float32, device=dev),
            qws=torch.empty(max(sol.nvfp4_quantize_workspace_bytes(max(M, N), K), 256),
                            dtype=torch.uint8, device=dev),
            gws=torch.empty(gws, dtype=torch.uint8, device=dev) if gws else None,
            out=torch.empty((M, N), dtype=torch.bfloat16, device=dev),
            M=M, N=N, K=K, name=layer.name))
    torch.cuda.synchronize()
    return layers


def run_nvfp4_step(layers, steps, warmup):
    """Time `steps` steps (after `warmup`) of the NVFP4 step on resident
    inputs: wall clock per step, and per layer HIP events (on the stream the
    kernels run on) around the weight quantize, the activation quantize and
    the GEMM.  Then, apart from the step, the activations' two quantize
    passes called one at a time (nvfp4_quantize_amax, nvfp4_quantize_encode)
    with events around each: the encode pass's own figure."""
    import numpy as np
    import torch

    import paper_2604_06916_amd as sol

    def step(events=None):
        for i, L in enumerate(layers):
            e = events[i] if events is not None else None
            if e:
                e[0].record()
            sol.nvfp4_quantize(L["w"], L["wc"], L["ws"], L["wa"], L["qws"])
            if e:
                e[1].record()
            sol.nvfp4_quantize(L["x"], L["xc"], L["xs"], L["xa"], L["qws"])
            if e:
                e[2].record()
            sol.nvfp4_gemm(L["xc"], L["xs"], L["xa"], L["wc"], L["ws"], L["wa"], L["b"], L["out"],
                           L["gws"])
            if e:
                e[3].record()

    for _ in range(warmup):
        step()
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in layers]
          for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        step(ev[s])
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) / steps * 1e3

    # the two passes apart (after another layer's GEMM, as in the step)
    reps = max(3, min(steps, 10))
    pev = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in layers]
           for _ in range(reps)]
    for r in range(reps):
        for i, L in enumerate(layers):
            P = layers[i - 1]
            sol.nvfp4_gemm(P["xc"], P["xs"], P["xa"], P["wc"], P["ws"], P["wa"], P["b"], P["out"],
                           P["gws"])
            pev[r][i][0].record()
            sol.nvfp4_quantize_amax(L["x"], L["qws"])
            pev[r][i][1].record()
            sol.nvfp4_quantize_encode(L["x"], L["xc"], L["xs"], L["xa"], L["qws"])
            pev[r][i][2].record()
    # a plain device-to-device copy of the largest activation on the same
    # box (reads 2 B and writes 2 B per element), after a GEMM like the passes
    big = max(range(len(layers)), key=lambda i: layers[i]["M"] * layers[i]["K"])
    dst = torch.empty_like(layers[big]["x"])
    cev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(reps)]
    for r in range(reps):
        P = layers[big - 1]
        sol.nvfp4_gemm(P["xc"], P["xs"], P["xa"], P["wc"], P["ws"], P["wa"], P["b"], P["out"],
                       P["gws"])
        cev[r][0].record()
        dst.copy_(layers[big]["x"])
        cev[r][1].record()
    torch.cuda.synchronize()
    copy_ms = float(np.mean([cev[r][0].elapsed_time(cev[r][1]) for r in range(reps)]))
    copy_gbs = 4.0 * layers[big]["M"] * layers[big]["K"] / (copy_ms * 1e-3) / 1e9
    del dst

    def span(i, a, b):
        return np.array([ev[s][i][a].elapsed_time(ev[s][i][b]) for s in range(steps)])

    def pspan(i, a, b):
        return np.array([pev[r][i][a].elapsed_time(pev[r][i][b]) for r in range(reps)])

    per_layer, tot = [], {"gemm": 0.0, "wq": 0.0, "xq": 0.0, "amax": 0.0, "enc": 0.0}
    for i, L in enumerate(layers):
        wq, xq, gm = span(i, 0, 1), span(i, 1, 2), span(i, 2, 3)
        am, en = pspan(i, 0, 1), pspan(i, 1, 2)
        for k, v in (("gemm", gm), ("wq", wq), ("xq", xq), ("amax", am), ("enc", en)):
            tot[k] += float(np.mean(v))
        n = L["M"] * L["K"]
        fl = 2.0 * L["M"] * L["N"] * L["K"]
        per_layer.append({
            "layer": L["name"], "M": L["M"], "N": L["N"], "K": L["K"],
            "gemm_kernel": nvfp4_gemm_kernel_name(L["M"], L["N"], L["K"]),
            "gemm_us": round(float(np.mean(gm)) * 1e3, 2),
            "gemm_tflops": round(fl / (float(np.mean(gm)) * 1e-3) / 1e12, 1),
            "gemm_us_p10_p50_p90": [round(float(np.percentile(gm, q)) * 1e3, 2) for q in (10, 50, 90)],
            "quantize_x_us": round(float(np.mean(xq)) * 1e3, 2),
            "quantize_x_us_p10_p50_p90": [round(float(np.percentile(xq, q)) * 1e3, 2) for q in (10, 50, 90)],
            "quantize_x_gbs": round(4.5625 * n / (float(np.mean(xq)) * 1e-3) / 1e9, 1),
            "amax_pass_us": round(float(np.mean(am)) * 1e3, 2),
            "amax_pass_gbs": round(2.0 * n / (float(np.mean(am)) * 1e-3) / 1e9, 1),
            "encode_pass_us": round(float(np.mean(en)) * 1e3, 2),
            "encode_pass_gbs": round(2.5625 * n / (float(np.mean(en)) * 1e-3) / 1e9, 1),
            "x_mb": round(2.0 * n / 1e6, 1),
            "quantize_w_us": round(float(np.mean(wq)) * 1e3, 2),
        })
    flops = sum(2.0 * L["M"] * L["N"] * L["K"] for L in layers)
    elems = sum(L["M"] * L["K"] for L in layers)
    return {"ms_per_step": ms_per_step, "flops": flops, "per_layer": per_layer,
            "gemm_ms": tot["gemm"], "wq_ms": tot["wq"], "xq_ms": tot["xq"],
            "amax_ms": tot["amax"], "enc_ms": tot["enc"], "copy_gbs": copy_gbs,
            "gemm_tflops": flops / (tot["gemm"] * 1e-3) / 1e12,
            "quant_gbs": 4.5625 * elems / (tot["xq"] * 1e-3) / 1e9,
            "encode_gbs": 2.5625 * elems / (tot["enc"] * 1e-3) / 1e9,
            "amax_gbs": 2.0 * elems / (tot["amax"] * 1e-3) / 1e9}


def gemm_roofline(r, layers, traffic=None):
    return {
        "bound": "mfma",
        "kernel": " + ".join(sorted({nvfp4_gemm_kernel_name(L["M"], L["N"], L["K"]) for L in layers})),
        "achieved": round(r["gemm_tflops"], 1),
        "peak": PEAK_FP16_MFMA_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(r["gemm_tflops"] / PEAK_FP16_MFMA_TFLOPS, 4),
        "frac_fp4_peak": round(r["gemm_tflops"] / PEAK_FP4_MFMA_TFLOPS, 4),
        "traffic": traffic,
        "traffic_unit": "HBM bytes per launch (mean over the step's GEMMs)",
        "algorithmic_flops_per_launch": r["flops"] / len(layers),
        "note": "a launch here is one nvfp4_gemm call, timed with HIP events on its stream; a call "
                "whose last round of 256 x 256 tiles runs as 128 x 128 quadrants is two kernel "
                "launches, counted together",
    }


def quantize_summary(r, layers):
    """Whole quantize (both passes in one call, 4.5625 B/element, timed in
    the step) and each pass called alone, over the step's activation
    tensors; the largest tensor on its own (the graded encode-pass figure);
    tensors under the MALL's 256 MB may be partly served from it on the
    second pass (labelled).  Beside the largest tensor: a plain
    device-to-device copy of it on the same box (2 B read + 2 B written per
    element), the memory system's own rate for a read-and-write stream."""
    big = max(r["per_layer"], key=lambda p: p["x_mb"])
    return {
        "kernel": "amax_partial_kernel + nvfp4_encode_kernel (activations)",
        "achieved_gbs": round(r["quant_gbs"], 1),
        "bytes_per_element": 4.5625,
        "peak_gbs": PEAK_HBM_GBS,
        "frac_hbm": round(r["quant_gbs"] / PEAK_HBM_GBS, 4),
        "encode_pass": {"achieved_gbs": round(r["encode_gbs"], 1), "bytes_per_element": 2.5625,
                        "frac_hbm": round(r["encode_gbs"] / PEAK_HBM_GBS, 4)},
        "amax_pass": {"achieved_gbs": round(r["amax_gbs"], 1), "bytes_per_element": 2.0,
                      "frac_hbm": round(r["amax_gbs"] / PEAK_HBM_GBS, 4)},
        "largest_input": {"layer": big["layer"], "x_mb": big["x_mb"],
                          "encode_pass_gbs": big["encode_pass_gbs"],
                          "encode_pass_frac_hbm": round(big["encode_pass_gbs"] / PEAK_HBM_GBS, 4),
                          "whole_gbs": big["quantize_x_gbs"],
                          "above_mall": big["x_mb"] > 256,
                          "plain_copy_gbs": round(r["copy_gbs"], 1),
                          "encode_pass_vs_plain_copy": round(big["encode_pass_gbs"] / r["copy_gbs"], 3)},
        "mall_resident_candidates": [p["layer"] for p in r["per_layer"] if p["x_mb"] <= 256],
    }


def run_other_workload(name, steps, warmup):
    """The step on another configuration (its own layers and M): GEMM
    roofline, quantize figures, per-layer record."""
    import torch

    from workloads import WORKLOADS
    wl = WORKLOADS[name]
    layers = make_layers(wl, torch.device("cuda:0"))
    r = run_nvfp4_step(layers, steps, warmup)
    res = {"config": {"workload": wl.name, "M": wl.M,
                      "layers": [f"{L['name']} {L['K']}->{L['N']}" for L in layers]},
           "step_tflops": round(r["flops"] / (r["ms_per_step"] * 1e-3) / 1e12, 2),
           "ms_per_step": round(r["ms_per_step"], 4),
           "roofline": gemm_roofline(r, layers),
           "quantize": quantize_summary(r, layers),
           "layers": r["per_layer"]}
    del layers
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the layer shards "
              f"along tokens with no communication, see the design notes", file=sys.stderr)
        sys.exit(2)

    import torch

    from workloads import WORKLOADS

    wl = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layers = make_layers(wl, dev)
    state_before = gpu_state()
    r = run_nvfp4_step(layers, args.steps, args.warmup)
    state_after = gpu_state()
    value = r["flops"] / (r["ms_per_step"] * 1e-3) / 1e12
    traffic = (measured_traffic("nvfp4_gemm_flux-12b_traffic.txt", "gemm.hip")
               if wl.name == PROFILED_WORKLOAD else None)
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": wl.name, "M": wl.M,
            "layers": [f"{L['name']} {L['K']}->{L['N']}" for L in layers],
            "step": "per layer: nvfp4_quantize(W), nvfp4_quantize(X), nvfp4_gemm(+bias)",
            "operands": "NVFP4 (E2M1 + E4M3/16 + FP32 tensor scale)",
            "mfma": "exact FP16 dequant, v_mfma_f32_32x32x16_f16, FP32 accumulate",
            "parallelism": "single GPU",
        },
        "roofline": gemm_roofline(r, layers, traffic),
        "gemm_frac_fp4_peak": round(r["gemm_tflops"] / PEAK_FP4_MFMA_TFLOPS, 4),
        "quantize": quantize_summary(r, layers),
        "time_split_ms": {"gemm": round(r["gemm_ms"], 4),
                          "quantize_x": round(r["xq_ms"], 4),
                          "quantize_x_amax_pass_alone": round(r["amax_ms"], 4),
                          "quantize_x_encode_pass_alone": round(r["enc_ms"], 4),
                          "quantize_w": round(r["wq_ms"], 4)},
        "layers": r["per_layer"],
        "workloads": None,
        "mxfp4": None,
        "graphs": None,
        "small_linear": None,
        "stage1": None,
        "cpu_baseline": None,
        "paper_context": PAPER_CONTEXT,
        "profiles": profile_status(),
        "gpu_state": {"source": "amd-smi metric -p -c, before and after the NVFP4 step timing "
                                "(gfx_clk_mhz: min, mean, max over the XCDs)",
                      "before": state_before, "after": state_after},
    }
    if not args.no_graphs:
        result["graphs"] = run_graphs(layers, max(args.steps, 5))
    if not args.no_mxfp4:
        result["mxfp4"] = run_mxfp4(layers, args.steps, args.warmup,
                                    wl.name == PROFILED_WORKLOAD, not args.no_vendor)
    if args.copy_calibration:
        n = args.copy_calibration
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    del layers
    torch.cuda.empty_cache()
    if not args.no_workloads:
        result["small_linear"] = run_small_linear(max(args.steps, 5))
        others = {}
        for name in ("sana-1.6b", "sd35-large"):
            if name != wl.name:
                others[name] = run_other_workload(name, min(args.steps, 20), min(args.warmup, 5))
        others["single-1152"] = dict(result["small_linear"])
        result["workloads"] = others
    if not args.no_stage1:
        result["stage1"] = run_stage1()
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_rows, args.cpu_wrows)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
