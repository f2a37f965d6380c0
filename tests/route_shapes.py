"""Seeded GEMM shapes that meet every kernel route of the library: random
token counts, widths and depths in three bands (few tokens, hundreds,
thousands), K of every residue class the kernels treat apart (multiples of
128, K % 128 == 64, K % 64 == 32, K % 32 == 16).  Sized so that the float64
oracle takes each in well under a second."""
import numpy as np


def _draw(seed=2604):
    g = np.random.Generator(np.random.PCG64(seed))
    shapes = []
    # few tokens, K % 128 == 0: the 64 x 64 and wave-K kernels
    for _ in range(8):
        shapes.append((int(g.integers(1, 400)), int(g.integers(16, 2500)), int(128 * g.integers(1, 24))))
    # hundreds of tokens: 128 x 128 tiles, split last rounds, every K class
    for r in (0, 64, 32, 16, 0, 64):
        K = int(128 * g.integers(2, 16)) + r
        shapes.append((int(g.integers(300, 1100)), int(g.integers(300, 1800)), K))
    # thousands: 256 x 256 tiles, short K
    for r in (0, 64, 32, 16):
        K = int(128 * g.integers(1, 3)) + r
        shapes.append((int(g.integers(2000, 3400)), int(g.integers(2000, 3400)), K))
    # a last round split into K halves: 128 x 128 tiles (K % 128 == 0 and 64)
    shapes += [(384, 3072, 3072), (512, 2240, 2240)]
    return shapes


SHAPES = _draw()
