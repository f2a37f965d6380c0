"""Full-size workloads, in the launch configuration the benchmark times.

The GPU runs each layer at its real shape; the oracle checks sampled outputs
it can afford: quantized codes/scales of sampled rows (plus the row holding
the tensor's max, which fixes alpha), bit for bit, and the linear output on a
sampled [rows x columns] block against the oracle's quantize-then-GEMM."""
import numpy as np
import pytest
import torch

import oracle.nvfp4 as O
import paper_2604_06916_amd as sol
from gpu_util import abs_products, assert_per_element, bf16_from_dev, bf16_mismatch_fraction, \
    bf16_to_dev, f32_bits, poison_bf16, rel_fro, say, u8_from_dev
from workloads import (ROLE_BIAS, ROLE_W, ROLE_X, WORKLOADS, draw_activations, draw_bias,
                       draw_weights, seed_for)

pytestmark = pytest.mark.gpu

CASES = [(w.name, l.name) for w in WORKLOADS.values() for l in w.layers]


def sample_rows(n, k, seed, xb):
    g = np.random.Generator(np.random.PCG64(seed))
    amax_row = int(np.argmax((xb & np.uint16(0x7FFF)).max(axis=1)))
    rows = np.r_[g.choice(n, size=min(k, n), replace=False), np.arange(max(0, n - 3), n), amax_row]
    return np.unique(rows)


@pytest.mark.parametrize("wname,lname", CASES)
def test_layer(wname, lname):
    wl = WORKLOADS[wname]
    layer = next(l for l in wl.layers if l.name == lname)
    M, N, K = wl.M, layer.N, layer.K
    say(f"{wname}/{lname}: M={M} N={N} K={K}")
    xb = draw_activations(layer.x_dist, M, K, seed_for(wl.config_id, layer.index, ROLE_X))
    wb = draw_weights(N, K, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_W))
    bias = draw_bias(N, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_BIAS))
    x, w, b = bf16_to_dev(xb), bf16_to_dev(wb), bf16_to_dev(bias)

    wc, ws, wa = sol.nvfp4_quantize(w)
    xc, xs, xa = sol.nvfp4_quantize(x)
    out = poison_bf16((M, N))
    sol.nvfp4_linear(x, wc, ws, wa, b, out)
    out2 = poison_bf16((M, N))
    sol.nvfp4_linear(x, wc, ws, wa, b, out2)
    torch.cuda.synchronize()
    assert not torch.isnan(out).any(), "unwritten or non-finite outputs"
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16)), "not deterministic"

    # quantizer, sampled rows, bit-exact
    rm = sample_rows(M, 256, 1, xb)
    rn = sample_rows(N, 256, 2, wb)
    rxc, rxs, rxa = O.nvfp4_quantize_ref(xb[rm])
    rwc, rws, rwa = O.nvfp4_quantize_ref(wb[rn])
    assert f32_bits(xa.cpu().numpy()[0]) == f32_bits(rxa)
    assert f32_bits(wa.cpu().numpy()[0]) == f32_bits(rwa)
    assert np.array_equal(u8_from_dev(xs[torch.as_tensor(rm, device=x.device)]), rxs)
    assert np.array_equal(u8_from_dev(xc[torch.as_tensor(rm, device=x.device)]), rxc)
    assert np.array_equal(u8_from_dev(ws[torch.as_tensor(rn, device=x.device)]), rws)
    assert np.array_equal(u8_from_dev(wc[torch.as_tensor(rn, device=x.device)]), rwc)

    # linear, sampled output block
    ref = O.nvfp4_gemm_ref(rxc, rxs, rxa, rwc, rws, rwa, bias[rn])
    got = bf16_from_dev(out)[np.ix_(rm, rn)]
    err = rel_fro(got, ref)
    mism = bf16_mismatch_fraction(got, ref)
    say(f"  rel_fro={err:.3e} mismatch={mism:.2e} on {len(rm)}x{len(rn)} sampled outputs")
    assert err <= 2e-3
    assert mism <= 0.01
    sabs = abs_products(O.nvfp4_unscaled_ref(rxc, rxs), O.nvfp4_unscaled_ref(rwc, rws))
    assert_per_element(got, ref, sabs, np.float32(rxa) * np.float32(rwa), K, bias[rn])
    del x, w, b, out, out2, xc, xs, xa, wc, ws, wa
    torch.cuda.empty_cache()


@pytest.mark.parametrize("wname,lname", CASES)
def test_layer_mxfp4(wname, lname):
    """The MXFP4 variant at full size: mxfp4_quantize of both operands and
    mxfp4_linear as the benchmark launches them; sampled rows bit-exact,
    sampled outputs within the GEMM bar.  (Each MX block is encoded on its
    own, so rows can be checked without the rest of the tensor.)"""
    wl = WORKLOADS[wname]
    layer = next(l for l in wl.layers if l.name == lname)
    M, N, K = wl.M, layer.N, layer.K
    if K % 32:
        pytest.skip("MXFP4 needs K % 32 == 0")
    say(f"{wname}/{lname} (MXFP4): M={M} N={N} K={K}")
    xb = draw_activations(layer.x_dist, M, K, seed_for(wl.config_id, layer.index, ROLE_X))
    wb = draw_weights(N, K, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_W))
    bias = draw_bias(N, wl.w_sigma, seed_for(wl.config_id, layer.index, ROLE_BIAS))
    x, w, b = bf16_to_dev(xb), bf16_to_dev(wb), bf16_to_dev(bias)
    wc, ws = sol.mxfp4_quantize(w)
    xc, xs = sol.mxfp4_quantize(x)
    out = poison_bf16((M, N))
    sol.mxfp4_linear(x, wc, ws, b, out)
    out2 = poison_bf16((M, N))
    sol.mxfp4_linear(x, wc, ws, b, out2)
    torch.cuda.synchronize()
    assert not torch.isnan(out).any(), "unwritten or non-finite outputs"
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16)), "not deterministic"

    rm = sample_rows(M, 256, 3, xb)
    rn = sample_rows(N, 256, 4, wb)
    rxc, rxs = O.mxfp4_quantize_ref(xb[rm])
    rwc, rws = O.mxfp4_quantize_ref(wb[rn])
    assert np.array_equal(u8_from_dev(xs[torch.as_tensor(rm, device=x.device)]), rxs)
    assert np.array_equal(u8_from_dev(xc[torch.as_tensor(rm, device=x.device)]), rxc)
    assert np.array_equal(u8_from_dev(ws[torch.as_tensor(rn, device=x.device)]), rws)
    assert np.array_equal(u8_from_dev(wc[torch.as_tensor(rn, device=x.device)]), rwc)

    ref = O.mxfp4_gemm_ref(rxc, rxs, rwc, rws, bias[rn])
    got = bf16_from_dev(out)[np.ix_(rm, rn)]
    err = rel_fro(got, ref)
    mism = bf16_mismatch_fraction(got, ref)
    say(f"  rel_fro={err:.3e} mismatch={mism:.2e} on {len(rm)}x{len(rn)} sampled outputs")
    assert err <= 2e-3
    assert mism <= 0.01
    sabs = abs_products(O.mxfp4_unscaled_ref(rxc, rxs), O.mxfp4_unscaled_ref(rwc, rws))
    assert_per_element(got, ref, sabs, 1.0, K, bias[rn])
    del x, w, b, out, out2, xc, xs, wc, ws
    torch.cuda.empty_cache()
