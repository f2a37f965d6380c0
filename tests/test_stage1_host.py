"""Host logic of the synthetic Stage-1 loop and pins of its CPU oracle (no GPU):
rollout selection against brute force, the zero model, attention against its
element-by-element definition, GELU-tanh and RMSNorm against independent
routines and closed forms, the Euler step and the reward on hand-worked
cases, and planted mistakes that each make a pin fail."""
import itertools

import numpy as np
import pytest

from oracle import stage1 as S
import oracle.nvfp4 as O


class Cfg:
    blocks, hidden, heads, mlp, rollouts, tokens, steps = 1, 64, 2, 128, 3, 5, 2


def select_brute(r, keep):
    idx = list(range(len(r)))
    top = sorted(idx, key=lambda i: (-r[i], i))[: keep // 2]
    rest = [i for i in idx if i not in top]
    bottom = sorted(rest, key=lambda i: (r[i], i))[: keep // 2]
    return top, bottom


def test_select_rollouts_matches_brute_force():
    pytest.importorskip("torch")
    from paper_2604_06916_amd.stage1 import select_rollouts
    g = np.random.Generator(np.random.PCG64(3))
    for n in (2, 4, 8, 96):
        for keep in range(2, n + 1, 2):
            r = np.round(g.standard_normal(n), 1)          # ties on purpose
            top, bottom = select_rollouts(r, keep)
            bt, bb = select_brute(list(r), keep)
            assert list(top) == bt and list(bottom) == bb
            assert not set(top) & set(bottom)
    with pytest.raises(ValueError):
        select_rollouts(np.zeros(4), 3)


def test_zero_model_is_the_identity():
    """All weights and biases zero: every linear returns 0, so the residual
    stream is unchanged and each Euler step leaves x as it is, whatever the
    linear backend."""
    g = np.random.Generator(np.random.PCG64(4))
    M = Cfg.rollouts * Cfg.tokens
    x0 = O.f64_to_bf16_bits_rne(g.standard_normal((M, Cfg.hidden)))
    shapes = [("qkv", 3 * Cfg.hidden, Cfg.hidden), ("out", Cfg.hidden, Cfg.hidden),
              ("up", Cfg.mlp, Cfg.hidden), ("down", Cfg.hidden, Cfg.mlp)]
    zero = [{n: (np.zeros((N, K), np.uint16), np.zeros(N, np.uint16)) for n, N, K in shapes}]
    for backend in ("bf16", "nvfp4", "mxfp4"):
        x = S.rollout(backend, x0, zero, Cfg)
        assert np.array_equal(x, O.bf16_bits_to_f32(x0).astype(np.float64)), backend


def test_attention_matches_elementwise_definition():
    g = np.random.Generator(np.random.PCG64(5))
    R, T, H, hd = 2, 4, 2, 3
    qkv = g.standard_normal((R * T, 3 * H * hd))
    got = S.attention(qkv, R, T, H, hd)
    want = np.zeros((R * T, H * hd))
    for r, h, i in itertools.product(range(R), range(H), range(T)):
        q = qkv[r * T + i, 0 * H * hd + h * hd: 0 * H * hd + (h + 1) * hd]
        s = [np.dot(q, qkv[r * T + j, H * hd + h * hd: H * hd + (h + 1) * hd]) / np.sqrt(hd) for j in range(T)]
        p = np.exp(np.array(s) - max(s))
        p /= p.sum()
        for j in range(T):
            want[r * T + i, h * hd:(h + 1) * hd] += p[j] * qkv[r * T + j, 2 * H * hd + h * hd: 2 * H * hd + (h + 1) * hd]
    assert np.array_equal(got, S.bf16_round(want))


def test_gelu_and_rmsnorm_closed_forms():
    assert S.gelu_tanh(np.array([0.0]))[0] == 0.0
    assert abs(S.gelu_tanh(np.array([10.0]))[0] - 10.0) < 1e-12
    c = np.full((1, 16), 3.0)
    assert np.allclose(S.rmsnorm(c), S.bf16_round(3.0 / np.sqrt(9.0 + S.EPS)))


# ---------------------------------------------------------------------------
# Pins of the Stage-1 oracle's elementwise pieces, Euler step and reward
# (Sec. 3.4, Stage 1: the loop around the quantized linears).  Each is fixed
# by mathematics or by an independent library routine, never by retyping the
# oracle's formula; the planted mistakes below must each make one fail.
# ---------------------------------------------------------------------------

def pin_gelu_tanh():
    import scipy.special as sp
    x = np.linspace(-8.0, 8.0, 4001)
    g = S.gelu_tanh(x)
    # an independent implementation of the same tanh form (torch, float64, CPU)
    torch = pytest.importorskip("torch")
    t = torch.nn.functional.gelu(torch.from_numpy(x), approximate="tanh").numpy()
    assert np.max(np.abs(g - t)) <= 1e-14 * max(1.0, np.max(np.abs(t)))
    # the tanh form approximates x * Phi(x) (Phi: standard normal CDF) to
    # better than 5e-4 everywhere
    assert np.max(np.abs(g - x * sp.ndtr(x))) < 5e-4
    # odd part: gelu(x) - gelu(-x) = x for any 0.5 x (1 + odd(x)) form
    assert np.max(np.abs((g - S.gelu_tanh(-x)) - x)) <= 1e-12 * np.max(np.abs(x))
    # curvature at 0: (gelu(h) + gelu(-h)) / h^2 -> 2 Phi'(0) = sqrt(2 / pi)
    h = 1e-4
    c = (S.gelu_tanh(np.array([h]))[0] + S.gelu_tanh(np.array([-h]))[0]) / h ** 2
    assert abs(c - np.sqrt(2.0 / np.pi)) < 1e-6


def pin_rmsnorm():
    # [3, 4]: mean of squares 12.5, so x / sqrt(12.5) (EPS shifts it by 4e-8
    # relative, far below one BF16 step); worked by hand: 0.8485281, 1.1313708
    got = S.rmsnorm(np.array([[3.0, 4.0]]))
    assert np.array_equal(got, S.bf16_round(np.array([[0.84852813742, 1.13137084990]])))
    # magnitudes where EPS matters: mean x^2 = 1e-6 = EPS, so every element
    # is +-1e-3 / sqrt(2e-6) = +-1/sqrt(2) (without EPS it would be +-1)
    v = np.array([[1e-3, -1e-3, 1e-3, -1e-3]])
    assert np.array_equal(S.rmsnorm(v), S.bf16_round(np.array([[1, -1, 1, -1]]) * 0.70710678118))
    # against torch's RMSNorm (float64, CPU) on random rows of varied scale
    torch = pytest.importorskip("torch")
    g = np.random.Generator(np.random.PCG64(12))
    x = g.standard_normal((6, 48)) * np.exp2(g.integers(-12, 4, size=(6, 1)))
    t = torch.nn.functional.rms_norm(torch.from_numpy(x), (48,), eps=S.EPS).numpy()
    assert np.array_equal(S.rmsnorm(x), S.bf16_round(t))


def _bias_model(cfg, b_out, b_down, b_other):
    """Zero weights, biases given: every linear returns its bias exactly (a
    zero GEMM plus a BF16 bias in any backend)."""
    shapes = [("qkv", 3 * cfg.hidden, cfg.hidden), ("out", cfg.hidden, cfg.hidden),
              ("up", cfg.mlp, cfg.hidden), ("down", cfg.hidden, cfg.mlp)]
    blk = {}
    for name, N, K in shapes:
        bias = {"out": b_out, "down": b_down}.get(name, np.full(N, b_other))
        blk[name] = (np.zeros((N, K), np.uint16), O.f64_to_bf16_bits_rne(bias))
    return [blk]


def pin_euler_step():
    # with zero weights, one block maps x to x + b_out + b_down (attention of
    # equal scores just averages equal values; the qkv and up biases do not
    # reach the residual stream), so each Euler step x <- x + (1/T)(blocks(x) - x)
    # adds c / T with c = b_out + b_down, and T steps reach x0 + c.  Values
    # are multiples of 1/8 below 16: every BF16 rounding is exact.
    class C:
        blocks, hidden, heads, mlp, rollouts, tokens = 1, 32, 2, 64, 2, 3
    g = np.random.Generator(np.random.PCG64(13))
    M = C.rollouts * C.tokens
    x0 = g.integers(-16, 16, size=(M, C.hidden)) / 4.0
    b_out = g.integers(-8, 8, size=C.hidden) / 2.0
    b_down = g.integers(-8, 8, size=C.hidden) / 2.0
    c = b_out + b_down
    model = _bias_model(C, b_out, b_down, 0.75)
    for backend in ("bf16", "nvfp4", "mxfp4"):
        for T, halfway in ((1, None), (2, x0 + c / 2), (4, None)):
            C.steps = T
            got = S.rollout(backend, O.f64_to_bf16_bits_rne(x0), model, C)
            assert np.array_equal(got, x0 + c), (backend, T)
        # T = 2, one step by hand: x1 = x0 + (1/2)((x0 + c) - x0)
        C.steps = 2
        layers = [{n: (S.prepare(backend, w), b) for n, (w, b) in blk.items()} for blk in model]
        assert np.array_equal(S.blocks(backend, x0, layers, C), x0 + c)


def pin_rewards():
    # 2 rollouts x 3 tokens x 4 hidden, direction u = [1, 0, -1, 0.5]; by hand:
    # rollout 0 tokens give <x,u> = 1-3+2 = 0, 0-1+0 = -1, 2-0+1.5 = 3.5 -> mean 2.5/3
    # rollout 1 tokens give 4-0+0 = 4, -1-1-0.5 = -2.5, 0-0+0 = 0 -> mean 1.5/3
    class C:
        rollouts, tokens, hidden = 2, 3, 4
    x = np.array([[1, 7, 3, 4], [0, 5, 1, 0], [2, 9, 0, 3],
                  [4, 1, 0, 0], [-1, 2, 1, -1], [0, 0, 0, 0]], dtype=np.float64)
    u = np.array([1.0, 0.0, -1.0, 0.5], dtype=np.float32)
    r = S.rewards(x, u, C)
    assert r.shape == (2,)
    assert abs(r[0] - 2.5 / 3) < 1e-15 and abs(r[1] - 1.5 / 3) < 1e-15


STAGE1_PINS = [pin_gelu_tanh, pin_rmsnorm, pin_euler_step, pin_rewards]


def test_stage1_pins():
    for pin in STAGE1_PINS:
        pin()


def _any_stage1_pin_fails():
    for pin in STAGE1_PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            return True
    return False


def _mut_gelu_erf(mp):
    import scipy.special as sp
    mp.setattr(S, "gelu_tanh", lambda x: x * sp.ndtr(x))


def _mut_gelu_coefficient(mp):
    mp.setattr(S, "gelu_tanh", lambda x: 0.5 * x * (1.0 + np.tanh(0.8 * (x + 0.044715 * x ** 3))))


def _mut_gelu_no_cubic(mp):
    mp.setattr(S, "gelu_tanh", lambda x: 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * x)))


def _mut_rmsnorm_eps_outside(mp):
    mp.setattr(S, "rmsnorm", lambda x: S.bf16_round(x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + S.EPS)))


def _mut_rmsnorm_mean_abs(mp):
    mp.setattr(S, "rmsnorm", lambda x: S.bf16_round(x / np.sqrt(np.mean(np.abs(x), axis=-1, keepdims=True) ** 2 + S.EPS)))


def _mut_euler_sign(mp):
    def rollout(backend, x0_bits, weights, cfg):
        layers = [{n: (S.prepare(backend, w), b) for n, (w, b) in blk.items()} for blk in weights]
        x = O.bf16_bits_to_f32(x0_bits).astype(np.float64)
        for _ in range(cfg.steps):
            x = S.bf16_round(x - (S.blocks(backend, x, layers, cfg) - x) / cfg.steps)
        return x
    mp.setattr(S, "rollout", rollout)


def _mut_euler_dt(mp):
    def rollout(backend, x0_bits, weights, cfg):
        layers = [{n: (S.prepare(backend, w), b) for n, (w, b) in blk.items()} for blk in weights]
        x = O.bf16_bits_to_f32(x0_bits).astype(np.float64)
        for _ in range(cfg.steps):
            x = S.bf16_round(x + (S.blocks(backend, x, layers, cfg) - x) / (cfg.steps + 1))
        return x
    mp.setattr(S, "rollout", rollout)


def _mut_residual_dropped(mp):
    orig = S.blocks

    def blocks(backend, x, layers, cfg):
        return orig(backend, x, layers, cfg) - x + S.bf16_round(0 * x)
    mp.setattr(S, "blocks", blocks)


def _mut_rewards_sum(mp):
    mp.setattr(S, "rewards", lambda x, u, cfg: (x.reshape(cfg.rollouts, cfg.tokens, cfg.hidden) @ u.astype(np.float64)).sum(axis=1))


def _mut_rewards_token_major(mp):
    mp.setattr(S, "rewards", lambda x, u, cfg: (x.reshape(cfg.tokens, cfg.rollouts, cfg.hidden) @ u.astype(np.float64)).mean(axis=0))


@pytest.mark.parametrize("mutation", [_mut_gelu_erf, _mut_gelu_coefficient, _mut_gelu_no_cubic,
                                      _mut_rmsnorm_eps_outside, _mut_rmsnorm_mean_abs,
                                      _mut_euler_sign, _mut_euler_dt, _mut_residual_dropped,
                                      _mut_rewards_sum, _mut_rewards_token_major],
                         ids=lambda f: f.__name__[5:])
def test_stage1_planted_mistake_is_caught(monkeypatch, mutation):
    assert not _any_stage1_pin_fails()
    mutation(monkeypatch)
    assert _any_stage1_pin_fails()
