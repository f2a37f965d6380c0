"""Synthetic Stage-1 rollout loop around the FP4 linears.

Stage 1 of the paper's two-stage framework (Sec. 3.4) samples a large pool
of rollouts with the quantized exploration model, scores each with a reward,
and keeps the highest- and lowest-rewarded ones for the BF16 policy update.
Here a stack of diffusion-transformer blocks with random weights stands in
for the denoiser, an Euler integrator for the sampler and a fixed linear
functional for the reward; no model weights, prompts or reward models are
involved.  Every linear layer runs through one backend:

    "nvfp4"  nvfp4_linear (activations quantized on the fly, NVFP4 weights)
    "mxfp4"  mxfp4_linear
    "bf16"   a plain BF16 matmul (the unquantized baseline)

Attention is BF16 through torch's fused attention kernels only (no fallback
to the unfused path).  Norms, GELU, residual adds and the Euler update are
elementwise BF16/FP32 torch ops around the linears.

Block (pre-norm, no modulation):
    h = rmsnorm(x); qkv = linear(h); a = attention(q, k, v); x = x + linear(a)
    h = rmsnorm(x); u = gelu_tanh(linear(h)); x = x + linear(u)
Euler step with T steps: x <- x + (1/T) * (blocks(x) - x).
Reward of rollout i: mean over its tokens of <x_final[token], u> for a fixed
direction u.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch
import torch.nn.functional as F
from torch.nn.attention import SDPBackend, sdpa_kernel

from . import _binding as sol

BACKENDS = ("bf16", "nvfp4", "mxfp4")
EPS = 1e-6


@dataclass(frozen=True)
class Stage1Config:
    blocks: int = 8
    hidden: int = 3072
    heads: int = 24
    mlp: int = 12288
    rollouts: int = 8
    tokens: int = 4608
    steps: int = 4
    keep: int = 4            # K: K/2 highest- and K/2 lowest-rewarded rollouts
    w_sigma: float = 0.015
    seed: int = 5000

    @property
    def head_dim(self):
        return self.hidden // self.heads


def layer_shapes(cfg):
    """(name, N, K) of one block's linears."""
    return [("qkv", 3 * cfg.hidden, cfg.hidden), ("out", cfg.hidden, cfg.hidden),
            ("up", cfg.mlp, cfg.hidden), ("down", cfg.hidden, cfg.mlp)]


def linear_flops(cfg):
    """FLOPs of every linear of one rollout (2 M N K per linear, M = all
    rollouts' tokens, four linears per block, every block, every step)."""
    M = cfg.rollouts * cfg.tokens
    return cfg.steps * cfg.blocks * sum(2.0 * M * N * K for _, N, K in layer_shapes(cfg))


def attention_flops(cfg):
    """FLOPs of the attention products of one rollout (Q K^T and P V, each
    2 T^2 d per head and rollout)."""
    return cfg.steps * cfg.blocks * cfg.rollouts * cfg.heads * 4.0 * cfg.tokens ** 2 * cfg.head_dim


def select_rollouts(rewards, keep):
    """Indices of the keep/2 highest and keep/2 lowest rewards (host logic):
    descending rewards for the top, ascending for the bottom, ties broken by
    the lower index."""
    r = np.asarray(rewards, dtype=np.float64)
    if keep % 2 or keep > r.size:
        raise ValueError("keep must be even and at most the number of rollouts")
    order = np.lexsort((np.arange(r.size), -r))          # descending, stable by index
    top = order[: keep // 2]
    rest = order[keep // 2:]
    bottom = rest[np.lexsort((rest, r[rest]))][: keep // 2]
    return top, bottom


def make_weights(cfg, device):
    """BF16 weights and biases of every block, seeded (workloads generator)."""
    from workloads import draw_bias, draw_weights
    model = []
    for b in range(cfg.blocks):
        blk = {}
        for j, (name, N, K) in enumerate(layer_shapes(cfg)):
            seed = cfg.seed + 100 * b + 10 * j
            w = draw_weights(N, K, cfg.w_sigma, seed)
            bias = draw_bias(N, cfg.w_sigma, seed + 1)
            blk[name] = (_bf16_dev(w, device), _bf16_dev(bias, device))
        model.append(blk)
    return model


def _bf16_dev(bits, device):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


class Runner:
    """Holds the backend's weights (quantized once, as after a policy update)
    and the activation and workspace buffers of the whole loop."""

    def __init__(self, cfg, model, backend, device):
        if backend not in BACKENDS:
            raise ValueError(backend)
        self.cfg, self.backend, self.device = cfg, backend, device
        M = cfg.rollouts * cfg.tokens
        self.M = M
        self.layers = []
        for blk in model:
            L = {}
            for name, N, K in layer_shapes(cfg):
                w, b = blk[name]
                if backend == "nvfp4":
                    q = sol.nvfp4_quantize(w)
                elif backend == "mxfp4":
                    q = sol.mxfp4_quantize(w)
                else:
                    q = (w.t().contiguous(),)        # [K, N] for a plain matmul
                L[name] = (q, b, N, K)
            self.layers.append(L)
        kmax = max(K for _, _, K in layer_shapes(cfg))
        if backend == "nvfp4":
            wsb = max(sol.nvfp4_linear_workspace_bytes(M, N, K) for _, N, K in layer_shapes(cfg))
            self.ws = torch.empty(wsb, dtype=torch.uint8, device=device)
        elif backend == "mxfp4":
            self.ws = torch.empty(sol.mxfp4_linear_workspace_bytes(M, kmax), dtype=torch.uint8, device=device)
        H, D = cfg.hidden, cfg.mlp
        self.buf = {n: torch.empty((M, c), dtype=torch.bfloat16, device=device)
                    for n, c in [("qkv", 3 * H), ("a", H), ("o", H), ("u", D), ("d", H)]}
        self.linear_events = None
        self.op_events = None    # dict: op kind -> [(start, end)] of HIP events, when timing
        self.trace = None        # list: (stage name, tensor copy) of every block stage
        self.step_trace = None   # list: {"y": blocks output, "x": latents after} per Euler step

    def _op(self, kind):
        """A (start, end) event pair for one op of this kind, or None."""
        if self.op_events is None:
            return None
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record()
        self.op_events.setdefault(kind, []).append(ev)
        return ev

    def _t(self, name, t):
        if self.trace is not None:
            self.trace.append((name, t.clone()))
        return t

    def linear(self, x, layer, out):
        q, b, N, K = layer
        ev = None
        if self.linear_events is not None:
            ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            ev[0].record()
        if self.backend == "nvfp4":
            sol.nvfp4_linear(x, q[0], q[1], q[2], b, out, self.ws)
        elif self.backend == "mxfp4":
            sol.mxfp4_linear(x, q[0], q[1], b, out, self.ws)
        else:
            torch.addmm(b, x, q[0], out=out)
        if ev is not None:
            ev[1].record()
            self.linear_events.append(ev)
        return out

    def blocks(self, x):
        cfg, B = self.cfg, self.buf
        R, T, Hh, hd = cfg.rollouts, cfg.tokens, cfg.heads, cfg.head_dim
        def end(ev):
            if ev is not None:
                ev[1].record()

        for L in self.layers:
            self._t("x", x)
            ev = self._op("norm")
            h = self._t("h1", _rmsnorm(x))
            end(ev)
            qkv = self._t("qkv", self.linear(h, L["qkv"], B["qkv"])).view(R, T, 3, Hh, hd)
            q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))   # [R, heads, T, hd] views
            ev = self._op("attention")
            with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
                a = F.scaled_dot_product_attention(q, k, v)
            end(ev)
            ev = self._op("copy")
            B["a"].copy_(a.transpose(1, 2).reshape(R * T, cfg.hidden))
            end(ev)
            self._t("a", B["a"])
            o = self._t("o", self.linear(B["a"], L["out"], B["o"]))
            ev = self._op("residual")
            x = self._t("x2", x + o)
            end(ev)
            ev = self._op("norm")
            h = self._t("h2", _rmsnorm(x))
            end(ev)
            u = self._t("up", self.linear(h, L["up"], B["u"]))
            ev = self._op("gelu")
            torch.ops.aten.gelu_(u, approximate="tanh")     # in place: one kernel, no copy
            end(ev)
            self._t("g", B["u"])
            d = self._t("d", self.linear(B["u"], L["down"], B["d"]))
            ev = self._op("residual")
            x = self._t("x3", x + d)
            end(ev)
        return x

    def rollout(self, x0):
        """T Euler steps from x0 [rollouts * tokens, hidden] (BF16)."""
        x = x0
        dt = 1.0 / self.cfg.steps
        for _ in range(self.cfg.steps):
            y = self.blocks(x)
            ev = self._op("euler")
            x = (x.float() + dt * (y.float() - x.float())).to(torch.bfloat16)
            if ev is not None:
                ev[1].record()
            if self.step_trace is not None:
                self.step_trace.append({"y": y.clone(), "x": x.clone()})
        return x


    def euler_step_(self, x):
        """One Euler step on x in place (x: [rollouts * tokens, hidden] BF16)."""
        dt = 1.0 / self.cfg.steps
        y = self.blocks(x)
        x.copy_((x.float() + dt * (y.float() - x.float())).to(torch.bfloat16))
        return x

    def capture_step(self, x_static):
        """One Euler step on the static buffer x_static, captured as a HIP
        graph (warmed up once on a side stream first, which advances
        x_static by a step); replaying it T times from the initial latents
        is the rollout without any host launch cost."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.euler_step_(x_static)
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.euler_step_(x_static)
        return g


def _rmsnorm(x):
    """RMSNorm of each row (no gain) as one fused torch kernel: FP32
    statistics, BF16 result (within one BF16 ulp of the float64 definition,
    as the unfused FP32 form)."""
    return F.rms_norm(x, (x.shape[-1],), eps=EPS)


def initial_latents(cfg, device):
    from workloads import draw_activations
    return _bf16_dev(draw_activations("normal", cfg.rollouts * cfg.tokens, cfg.hidden, cfg.seed + 7), device)


def reward_direction(cfg):
    g = np.random.Generator(np.random.PCG64(cfg.seed + 9))
    return (g.standard_normal(cfg.hidden) / np.sqrt(cfg.hidden)).astype(np.float32)


def rewards(cfg, x_final, u):
    """Per-rollout mean over tokens of <x, u> (FP32)."""
    xf = x_final.float().view(cfg.rollouts, cfg.tokens, cfg.hidden)
    return (xf @ torch.from_numpy(u).to(xf.device)).mean(dim=1)
