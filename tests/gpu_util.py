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
