"""GPU parity of the synthetic Stage-1 loop against the float64 CPU oracle
of the same loop.

Stage by stage: one block runs on the GPU with every intermediate tensor
recorded, and each stage is recomputed by the oracle from the GPU's own input
to that stage.  Linears must meet the GEMM bar (2e-3 relative Frobenius);
norms, attention, GELU and residual adds one BF16 rounding (relative error
within 2^-7).  End to end the loop is not reproducible to that level: a one-
ulp BF16 difference upstream (attention and FP32 sums run in different
orders) flips the FP4 code of elements that sit next to a rounding boundary,
and the flips compound over the layers.  So the whole rollout gets a coarse
bar (the latents within 15% of the oracle's for the FP4 formats, 1% for
BF16), finite values and a valid selection."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
from gpu_util import bf16_from_dev, device, say
from oracle import stage1 as S

pytestmark = pytest.mark.gpu


def tiny(blocks=2):
    from paper_2604_06916_amd.stage1 import Stage1Config
    return Stage1Config(blocks=blocks, hidden=256, heads=2, mlp=512, rollouts=4, tokens=64,
                        steps=2, keep=2, w_sigma=0.05, seed=6100)


def f64(t):
    return O.bf16_bits_to_f32(bf16_from_dev(t)).astype(np.float64)


def rel(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


@pytest.mark.parametrize("backend", ["bf16", "nvfp4", "mxfp4"])
def test_block_stages_vs_oracle(backend):
    from paper_2604_06916_amd import stage1 as G
    cfg = tiny(blocks=1)
    dev = device()
    model = G.make_weights(cfg, dev)
    runner = G.Runner(cfg, model, backend, dev)
    runner.trace = []
    runner.blocks(G.initial_latents(cfg, dev))
    torch.cuda.synchronize()
    t = {name: f64(v) for name, v in runner.trace}
    blk = {n: (bf16_from_dev(w), bf16_from_dev(b)) for n, (w, b) in model[0].items()}
    L = {n: (S.prepare(backend, w), b) for n, (w, b) in blk.items()}
    hd = cfg.hidden // cfg.heads
    checks = [
        ("h1", S.rmsnorm(t["x"]), 2 ** -7),
        ("qkv", S.linear(backend, t["h1"], *L["qkv"]), 2e-3),
        ("a", S.attention(t["qkv"], cfg.rollouts, cfg.tokens, cfg.heads, hd), 2 ** -7),
        ("o", S.linear(backend, t["a"], *L["out"]), 2e-3),
        ("x2", S.bf16_round(t["x"] + t["o"]), 2 ** -8),
        ("h2", S.rmsnorm(t["x2"]), 2 ** -7),
        ("up", S.linear(backend, t["h2"], *L["up"]), 2e-3),
        ("g", S.bf16_round(S.gelu_tanh(t["up"])), 2 ** -7),
        ("d", S.linear(backend, t["g"], *L["down"]), 2e-3),
        ("x3", S.bf16_round(t["x2"] + t["d"]), 2 ** -8),
    ]
    for name, ref, tol in checks:
        err = rel(t[name], ref)
        say(f"{backend} {name}: rel {err:.2e}")
        assert err <= tol, (name, err)


@pytest.mark.parametrize("backend", ["bf16", "nvfp4", "mxfp4"])
def test_rollout_vs_oracle(backend):
    from paper_2604_06916_amd import stage1 as G
    cfg = tiny()
    dev = device()
    model = G.make_weights(cfg, dev)
    runner = G.Runner(cfg, model, backend, dev)
    x0 = G.initial_latents(cfg, dev)
    xg = runner.rollout(x0)
    u = G.reward_direction(cfg)
    r_gpu = G.rewards(cfg, xg, u).cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    weights = [{n: (bf16_from_dev(w), bf16_from_dev(b)) for n, (w, b) in blk.items()} for blk in model]
    x_ref = S.rollout(backend, bf16_from_dev(x0), weights, cfg)
    r_ref = S.rewards(x_ref, u, cfg)
    err = rel(f64(xg), x_ref)
    say(f"{backend}: rollout rel {err:.3e}; rewards gpu {np.round(r_gpu, 4)} oracle {np.round(r_ref, 4)}")
    assert np.isfinite(f64(xg)).all() and np.isfinite(r_gpu).all()
    assert err <= (1e-2 if backend == "bf16" else 0.15)
    top, bottom = G.select_rollouts(r_gpu, cfg.keep)
    assert r_gpu[top].min() >= r_gpu[bottom].max()


@pytest.mark.parametrize("backend", ["bf16", "nvfp4", "mxfp4"])
def test_each_euler_step_vs_oracle(backend):
    """Each Euler step of the GPU rollout, recomputed by the oracle from the
    GPU's own latents x_t and block-stack output y_t (teacher forcing: a
    difference cannot compound): x_{t+1} = bf16(x_t + (1/T)(y_t - x_t)) to
    within one BF16 ulp (the GPU evaluates it in FP32, the oracle in
    float64), bit-exact in all but a sliver of elements.  With BF16 linears
    the oracle's own block stack from x_t is also held to 1e-2; with FP4
    linears a one-ulp input difference flips codes near rounding boundaries
    and the per-linear bar applies only stage by stage
    (test_block_stages_vs_oracle)."""
    from paper_2604_06916_amd import stage1 as G
    cfg = tiny()
    dev = device()
    model = G.make_weights(cfg, dev)
    runner = G.Runner(cfg, model, backend, dev)
    runner.step_trace = []
    x0 = G.initial_latents(cfg, dev)
    runner.rollout(x0)
    torch.cuda.synchronize()
    xs = [f64(x0)] + [f64(st["x"]) for st in runner.step_trace]
    ys = [f64(st["y"]) for st in runner.step_trace]
    dt = 1.0 / cfg.steps
    for t in range(cfg.steps):
        want = S.bf16_round(xs[t] + dt * (ys[t] - xs[t]))
        diff = np.abs(xs[t + 1] - want)
        _, e = np.frexp(np.where(want != 0, np.abs(want), 1.0))
        ulp = np.exp2(e - 8.0)
        frac = float(np.mean(diff > 0))
        say(f"{backend} step {t}: Euler update differs in {frac:.2e} of elements, "
            f"worst {float((diff / ulp).max()):.2f} ulp")
        assert np.all(diff <= ulp) and frac <= 1e-3
    if backend == "bf16":
        weights = [{n: (bf16_from_dev(w), bf16_from_dev(b)) for n, (w, b) in blk.items()}
                   for blk in model]
        layers = [{n: (S.prepare(backend, w), b) for n, (w, b) in blk.items()} for blk in weights]
        for t in range(cfg.steps):
            err = rel(ys[t], S.blocks(backend, xs[t], layers, cfg))
            say(f"bf16 step {t}: blocks rel {err:.3e}")
            assert err <= 1e-2
