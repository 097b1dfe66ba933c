"""GPU parity on seeded random shapes: many small problems with sizes drawn
at random (fixed seed), against the fp64 oracle, in every kernel family that
can run them.  Integer-valued inputs must match bit for bit; float inputs to
|O - O64| <= 1e-5 * sum|I*F| per output.
"""
import numpy as np
import pytest

from dconv_workloads import random_arrays
from gpu_util import assert_exact, assert_within, gpu_multi, gpu_single, oracle_multi, oracle_single
from random_shapes import MULTI_RANDOM, SINGLE_RANDOM

pytestmark = pytest.mark.gpu




@pytest.mark.parametrize("shape", SINGLE_RANDOM, ids=[str(s) for s in SINGLE_RANDOM])
def test_single_random(shape):
    Wx, Wy, K, M = shape
    fams = ["auto", "valu"] + (["mfma"] if 5 <= K <= 11 and Wx % 4 == 0 else [])
    I, F = random_arrays(1, M, Wx, Wy, K, seed=hash(shape) % 2**31)
    Ii, Fi = random_arrays(1, M, Wx, Wy, K, seed=hash(shape) % 2**31 + 1, variant="int")
    O64, A64 = oracle_single(I[0], F[:, 0])
    O64i, _ = oracle_single(Ii[0], Fi[:, 0])
    for fam in fams:
        assert_within(gpu_single(I[0], F[:, 0], variant=fam), O64, A64, "single %r %s" % (shape, fam))
        assert_exact(gpu_single(Ii[0], Fi[:, 0], variant=fam), O64i,
                     "single int %r %s" % (shape, fam))


@pytest.mark.parametrize("shape", MULTI_RANDOM, ids=[str(s) for s in MULTI_RANDOM])
def test_multi_random(shape):
    C, M, Wx, Wy, K = shape
    fams = ["auto", "valu"] + (["mfma"] if K <= 11 else [])
    I, F = random_arrays(C, M, Wx, Wy, K, seed=hash(shape) % 2**31)
    Ii, Fi = random_arrays(C, M, Wx, Wy, K, seed=hash(shape) % 2**31 + 1, variant="int")
    O64, A64 = oracle_multi(I, F)
    O64i, _ = oracle_multi(Ii, Fi)
    for fam in fams:
        assert_within(gpu_multi(I, F, fam), O64, A64, "multi %r %s" % (shape, fam))
        assert_exact(gpu_multi(Ii, Fi, fam), O64i, "multi int %r %s" % (shape, fam))
