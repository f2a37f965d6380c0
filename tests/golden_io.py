"""Reader for tests/golden/*.txt fixtures (format described in each file)."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _hexbytes(tokens):
    return np.array([int(t, 16) for t in tokens], dtype=np.uint8)


def load(name="nvfp4_hand_worked.txt"):
    cases, cur = {}, None
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *rest = line.split()
            if key in ("case", "gemm", "mxcase", "mxgemm"):
                cur = {"kind": key, "name": rest[0]}
            elif key == "end":
                cases[cur["name"]] = cur
                cur = None
            elif key == "x":
                cur["x"] = np.array([float(t) for t in rest], dtype=np.float32)
            elif key in ("alpha", "a_alpha", "b_alpha"):
                cur[key] = np.array([int(rest[0], 16)], dtype=np.uint32).view(np.float32)[0]
            elif key == "exact":
                cur[key] = float(rest[0])
            elif key == "bf16":
                cur[key] = int(rest[0], 16)
            else:
                cur[key] = _hexbytes(rest)
    return cases


def f32_to_bf16_exact(x):
    """BF16 bits of float32 values that are exactly representable in BF16."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "fixture value not exact in BF16"
    return (u >> 16).astype(np.uint16)
