"""Seeded random problem sizes shared by the plan tests (CPU) and the parity
tests (GPU)."""
import numpy as np


def _single_shapes(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        Wx = int(rng.integers(1, 300))
        if i % 2 == 0:   # rows of a multiple of 4 floats: the float4 and matrix-core paths
            Wx = 4 * int(rng.integers(1, 75))
        Wy = int(rng.integers(1, 120))
        K = int(rng.integers(1, min(Wx, Wy, 13) + 1))
        M = int(rng.integers(1, 9))
        out.append((Wx, Wy, K, M))
    return out


def _multi_shapes(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        K = int(rng.integers(1, 10))
        Wx = int(rng.integers(K, 41))
        Wy = int(rng.integers(K, 41))
        C = int(rng.integers(1, 81))
        M = int(rng.integers(1, 101))
        out.append((C, M, Wx, Wy, K))
    return out


SINGLE_RANDOM = _single_shapes(40, 20221201)
MULTI_RANDOM = _multi_shapes(40, 20221202)
