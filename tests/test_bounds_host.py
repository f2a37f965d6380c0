"""The per-element GEMM bound used by the GPU parity tests, checked on the
CPU: an FP32 evaluation of the oracle's own operands in a shuffled summation
order passes it, and the same evaluation with one 16-element block given a
wrong scale, or one block shifted by 16 elements along K, fails it (at the
longest K of the workloads, 12288, too)."""
import numpy as np
import pytest

import oracle.nvfp4 as O
from gpu_util import abs_products, assert_per_element
from workloads import draw_activations, draw_weights


def fp32_gemm(a_deq, b_deq, alpha, rng):
    """FP32 dot products in a random order per output, then the epilogue's
    FP32 multiply and the BF16 rounding."""
    M, K = a_deq.shape
    N = b_deq.shape[0]
    out = np.empty((M, N), np.float64)
    for m in range(M):
        perm = rng.permutation(K)
        prod = (a_deq[m, perm].astype(np.float32)[None, :] * b_deq[:, perm].astype(np.float32))
        acc = np.zeros(N, np.float32)
        for k in range(0, K, 64):                      # blocked FP32 sums
            acc = (acc + prod[:, k:k + 64].sum(axis=1, dtype=np.float32)).astype(np.float32)
        out[m] = (np.float32(alpha) * acc).astype(np.float32)
    return O.f64_to_bf16_bits_rne(out)


@pytest.mark.parametrize("K", [256, 3072, 12288])
def test_bound_accepts_fp32_orders_and_rejects_wrong_blocks(K):
    M, N = 6, 40
    a = O.nvfp4_quantize_ref(draw_activations("normal", M, K, seed=K + 1))
    b = O.nvfp4_quantize_ref(draw_weights(N, K, 0.02, seed=K + 2))
    ref = O.nvfp4_gemm_ref(*a, *b)
    ad, bd = O.nvfp4_unscaled_ref(a[0], a[1]), O.nvfp4_unscaled_ref(b[0], b[1])
    sabs = abs_products(ad, bd)
    alpha = np.float32(a[2]) * np.float32(b[2])
    rng = np.random.Generator(np.random.PCG64(K))
    assert_per_element(fp32_gemm(ad, bd, alpha, rng), ref, sabs, alpha, K)

    bad_scale = a[1].copy()
    bad_scale[2, 5] = np.uint8(min(int(bad_scale[2, 5]) + 8, 0x7E))   # one scale doubled
    got = fp32_gemm(O.nvfp4_unscaled_ref(a[0], bad_scale), bd, alpha, rng)
    with pytest.raises(AssertionError):
        assert_per_element(got, ref, sabs, alpha, K)

    shifted = ad.copy()
    shifted[4, 16:32] = ad[4, 32:48]                               # one block misplaced
    got = fp32_gemm(shifted, bd, alpha, rng)
    with pytest.raises(AssertionError):
        assert_per_element(got, ref, sabs, alpha, K)
