"""Helpers for the GPU parity tests: host <-> device copies of raw bit
patterns and the comparison metrics.  Inputs always come from workloads/ or
from the test itself; expected values only from oracle/."""
import sys

import numpy as np
import pytest
import torch

import oracle.nvfp4 as O


def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bf16_to_dev(bits: np.ndarray) -> torch.Tensor:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(bits.view(np.int16)).to(device()).view(torch.bfloat16)


def u8_to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).to(device())


def f32_to_dev(v) -> torch.Tensor:
    return torch.tensor([np.float32(v)], dtype=torch.float32, device=device())


def bf16_from_dev(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def u8_from_dev(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().cpu().numpy()


def f32_bits(v) -> int:
    return int(np.array([v], dtype=np.float32).view(np.uint32)[0])


def rel_fro(got_bits: np.ndarray, ref: np.ndarray) -> float:
    g = O.bf16_bits_to_f32(got_bits).astype(np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(g - ref) / den) if den > 0 else float(np.linalg.norm(g))


def bf16_mismatch_fraction(got_bits: np.ndarray, ref: np.ndarray) -> float:
    return float(np.mean(got_bits != O.bf16_output(ref)))


def poison_u8(shape, value=0xAB):
    return torch.full(shape, value, dtype=torch.uint8, device=device())


def poison_bf16(shape):
    # a NaN pattern: any element the kernel fails to write stays NaN
    return torch.full(shape, 0x7FC1, dtype=torch.int16, device=device()).view(torch.bfloat16)


def abs_products(a_deq: np.ndarray, b_deq: np.ndarray) -> np.ndarray:
    """sum_k |a[m, k]| |b[n, k]| in float64, from the oracle's dequantized
    operands (block scale times element value, per-tensor scale excluded)."""
    return np.abs(a_deq) @ np.abs(b_deq).T


def assert_per_element(got_bits: np.ndarray, ref: np.ndarray, sabs: np.ndarray, alpha, K: int,
                       bias_bits=None, label=""):
    """Every output within a bound that any FP32 summation order meets:

        |got - ref| <= ulp_bf16(max(|got|, |ref|))
                       + (K + 4) 2^-24 (|alpha| sum_k |a_k b_k| + |bias|)

    The first term covers the final rounding to BF16 (half an ulp, doubled so
    that a result rounded into the next binade still passes).  The second
    covers the FP32 arithmetic: the products are exact, a sum of K of them
    in any order rounds at most K - 1 times, each time by at most 2^-24 of a
    partial sum no larger than sum |a b|; then the product of the two tensor
    scales and the epilogue's fused multiply-add round once each.  (The
    matrix instructions add 16 or 64 products per rounding of the
    accumulator, so the count is generous.)  A wrong block scale or a
    misplaced 16-element block moves an output by far more."""
    g = O.bf16_bits_to_f32(got_bits).astype(np.float64)
    b = 0.0 if bias_bits is None else np.abs(O.bf16_bits_to_f32(bias_bits).astype(np.float64))[None, :]
    mag = np.maximum(np.abs(g), np.abs(ref))
    _, e = np.frexp(np.where(mag > 0, mag, 1.0))
    ulp = np.where(mag > 0, np.exp2(np.maximum(e - 8, -133)), 2.0 ** -133)
    bound = ulp + (K + 4) * 2.0 ** -24 * (abs(float(alpha)) * sabs + b)
    excess = np.abs(g - ref) / bound
    worst = float(excess.max()) if excess.size else 0.0
    say(f"  {label}per-element: worst |err| / bound = {worst:.3f}")
    assert np.all(np.isfinite(g))
    assert worst <= 1.0, (label, np.unravel_index(int(np.argmax(excess)), excess.shape))
