"""Host logic of the synthetic Stage-1 loop and pins of its CPU oracle (no GPU)."""
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
