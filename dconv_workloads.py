"""Seeded synthetic inputs for direct convolution.

This module only draws random arrays; it holds none of the convolution's
arithmetic.  Both sides of every parity check (the CPU oracle and the GPU
library) receive the arrays it returns, and the benchmark uses the same
recipes.

Workloads mirror the layer shapes the paper evaluates (Section 4: CNN
convolution layers with feature maps from 7 to 1K pixels, 64 to 512 channels
and filter sizes 1, 3, 5; single-channel layers with 32 to 512 filters) plus
a large single-map case with K up to 11.  The
paper used no dataset, only layer shapes, so seeded synthetic data stands in:

* single-map workloads: input and filters uniform in [-1, 1);
* multi-channel workloads: activations uniform in [0, 1) (post-ReLU-like),
  weights normal with mean 0 and variance 2 / (C * K * K) (He initialisation);
* every workload also has an integer variant with values in {-3, ..., 3}, for
  which fp32 arithmetic is exact in any summation order.

All arrays are float32, C-contiguous, in the library's layouts:
``I[C][Wy][Wx]`` (``I[Wy][Wx]`` for single-map calls), ``F[M][C][K][K]``
(``F[M][K][K]``).
"""
from __future__ import annotations

import dataclasses
import zlib

import numpy as np

SEED_BASE = 221200404


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    kind: str          # "single" or "multi"
    C: int
    M: int
    Wx: int
    Wy: int
    K: int

    @property
    def Hout(self) -> int:
        return self.Wy - self.K + 1

    @property
    def Wout(self) -> int:
        return self.Wx - self.K + 1

    @property
    def outputs(self) -> int:
        return self.M * self.Hout * self.Wout

    @property
    def flops(self) -> int:
        """2 * C * M * K^2 * Hout * Wout: one multiply and one add per term."""
        return 2 * self.C * self.M * self.K * self.K * self.Hout * self.Wout

    @property
    def compulsory_bytes(self) -> int:
        """Each input, filter and output value moved once, 4 bytes each."""
        return 4 * (self.C * self.Wy * self.Wx + self.M * self.C * self.K * self.K
                    + self.M * self.Hout * self.Wout)

    def seed(self, variant: str = "float") -> int:
        return SEED_BASE + zlib.crc32(("%s/%s" % (self.name, variant)).encode()) % 1_000_000


def _single(name, W, M, K):
    return Workload(name, "single", 1, M, W, W, K)


def _multi(name, C, W, M, K):
    return Workload(name, "multi", C, M, W, W, K)


WORKLOADS = {w.name: w for w in [
    _single("single_64x64_m1_k3", 64, 1, 3),
    *[_single("single_4096x4096_m1_k%d" % k, 4096, 1, k) for k in (3, 5, 7, 9, 11)],
    _multi("multi_c512_9x9_m512_k3", 512, 9, 512, 3),
    _multi("multi_c256_30x30_m256_k3", 256, 30, 256, 3),
    _multi("multi_c512_16x16_m512_k3", 512, 16, 512, 3),
    _multi("multi_c64_114x114_m128_k3", 64, 114, 128, 3),
    _multi("multi_c128_60x60_m128_k5", 128, 60, 128, 5),
    _multi("multi_c256_28x28_m256_k1", 256, 28, 256, 1),
    # large filters (K = 9, 11) on small maps: long inner products per
    # output, few output tiles
    _multi("multi_c64_40x40_m64_k9", 64, 40, 64, 9),
    _multi("multi_c32_42x42_m64_k11", 32, 42, 64, 11),
    # one input map, many filters: the single-channel layers the paper
    # targets (maps of 28 to 1K pixels, 32 to 512 filters, K = 1, 3, 5)
    _single("single_28x28_m512_k3", 28, 512, 3),
    _single("single_56x56_m256_k5", 56, 256, 5),
    _single("single_112x112_m128_k3", 112, 128, 3),
    _single("single_224x224_m64_k5", 224, 64, 5),
    _single("single_512x512_m128_k1", 512, 128, 1),
    _single("single_1024x1024_m32_k3", 1024, 32, 3),
    # the paper's multi-channel sweep (Section 4: maps 7 to 512, 64 to 512
    # channels, K = 1, 3, 5), as CNN-layer-like shapes with C = M
    *[_multi("layer_c%d_%dx%d_m%d_k%d" % (c, w, w, c, k), c, w, c, k) for c, w, k in (
        (64, 512, 3), (64, 224, 3), (128, 112, 3), (256, 56, 3), (512, 28, 3), (512, 14, 3),
        (512, 7, 3), (64, 56, 1), (256, 28, 1), (512, 14, 1), (64, 56, 5), (128, 28, 5),
        (256, 14, 5))],
    # 4096-wide single maps of 1, 2, 4 and 8 rounds of tiles per persistent
    # workgroup (K = 9 and 11: 1032, 2056, 4096, 8192 rows): the time per
    # round and the fixed cost of a launch
    *[Workload("single_4096x%d_m1_k%d" % (h, k), "single", 1, 1, 4096, h, k)
      for k in (9, 11) for h in (1032, 2056, 8192)],
]}

# The large single-map workload is one pass over all five filter sizes.
SINGLE_4096_SWEEP = tuple("single_4096x4096_m1_k%d" % k for k in (3, 5, 7, 9, 11))
# The multi-channel configurations.
MULTI_CONFIGS = ("multi_c512_9x9_m512_k3", "multi_c256_30x30_m256_k3", "multi_c512_16x16_m512_k3",
                 "multi_c64_114x114_m128_k3", "multi_c128_60x60_m128_k5",
                 "multi_c256_28x28_m256_k1")
# The paper's multi-channel layer sweep.
PAPER_MULTI_SWEEP = tuple(n for n in WORKLOADS if n.startswith("layer_"))
# Large filters on small multi-channel maps.
LARGE_FILTER_LAYERS = ("multi_c64_40x40_m64_k9", "multi_c32_42x42_m64_k11")
# The 4096-wide single map at 1, 2, 4 and 8 rounds of tiles per workgroup.
SINGLE_ROUNDS = tuple("single_4096x%d_m1_k%d" % (h, k) for k in (9, 11)
                      for h in (1032, 2056, 4096, 8192))
# Single map, many filters.
SINGLE_MULTI_FILTER = ("single_28x28_m512_k3", "single_56x56_m256_k5", "single_112x112_m128_k3",
                       "single_224x224_m64_k5", "single_512x512_m128_k1",
                       "single_1024x1024_m32_k3")


def make(w: Workload | str, variant: str = "float", seed: int | None = None):
    """Return ``(I, F)`` float32 arrays for workload ``w``.

    ``variant`` is ``"float"`` (the distributions above) or ``"int"`` (values in
    {-3..3}).  Single-map workloads return ``I[Wy][Wx]`` and ``F[M][K][K]``.
    """
    if isinstance(w, str):
        w = WORKLOADS[w]
    rng = np.random.default_rng(w.seed(variant) if seed is None else seed)
    ishape = (w.C, w.Wy, w.Wx)
    fshape = (w.M, w.C, w.K, w.K)
    if variant == "int":
        I = rng.integers(-3, 4, size=ishape).astype(np.float32)
        F = rng.integers(-3, 4, size=fshape).astype(np.float32)
    elif variant == "float":
        if w.kind == "single":
            I = rng.uniform(-1.0, 1.0, size=ishape).astype(np.float32)
            F = rng.uniform(-1.0, 1.0, size=fshape).astype(np.float32)
        else:
            I = rng.uniform(0.0, 1.0, size=ishape).astype(np.float32)
            std = np.sqrt(2.0 / (w.C * w.K * w.K))
            F = (rng.standard_normal(size=fshape) * std).astype(np.float32)
    else:
        raise ValueError("variant must be 'float' or 'int'")
    if w.kind == "single":
        return I[0].copy(), F[:, 0].copy()
    return I, F


def random_arrays(C, M, Wx, Wy, K, seed, variant="float"):
    """Arbitrary-shape inputs for property and edge-case tests."""
    rng = np.random.default_rng(seed)
    if variant == "int":
        I = rng.integers(-3, 4, size=(C, Wy, Wx)).astype(np.float32)
        F = rng.integers(-3, 4, size=(M, C, K, K)).astype(np.float32)
    else:
        I = rng.uniform(-1.0, 1.0, size=(C, Wy, Wx)).astype(np.float32)
        F = rng.uniform(-1.0, 1.0, size=(M, C, K, K)).astype(np.float32)
    return I, F
