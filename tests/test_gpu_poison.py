"""GPU: the LDS-poisoning debug build of the library (libdconv_poison.so,
built with -DDCONV_POISON_LDS): every kernel's LDS starts filled with NaN, so
any output computed from LDS that the kernel did not write first (a copy,
wait or barrier missing before a buffer's first use) is non-finite and
fails the comparison with the oracle.  Runs the full-size workloads in their
planned kernels, both single-map families, and every candidate plan of a few
small layers, through the debug library's C ABI."""
import ctypes
import os

import numpy as np
import pytest
import torch

import paper_2212_00404_amd as dc
from dconv_workloads import MULTI_CONFIGS, SINGLE_4096_SWEEP, WORKLOADS, make, random_arrays
from gpu_util import assert_exact, assert_within, oracle_multi, oracle_single

pytestmark = pytest.mark.gpu

POISON = os.path.join(os.path.dirname(dc.dconv.LIB_PATH), "libdconv_poison.so")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(POISON):
        pytest.fail("libdconv_poison.so is not built (paper_2212_00404_amd/build.py builds it)")
    return dc.load(POISON)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def run_multi(lib, I, F, plan=None, variant=0):
    C, Wy, Wx = I.shape
    M, _, K, _ = F.shape
    It, Ft = torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()
    O = torch.empty((M, Wy - K + 1, Wx - K + 1), device="cuda")
    if plan is None:
        rc = lib.dconv_multi_variant(It.data_ptr(), Ft.data_ptr(), O.data_ptr(), C, M, Wx, Wy, K,
                                     variant, _stream())
    else:
        rc = lib.dconv_multi_with_plan(It.data_ptr(), Ft.data_ptr(), O.data_ptr(), C, M, Wx, Wy,
                                       K, ctypes.byref(dc.Plan(**plan)), _stream())
    assert rc == 0, rc
    torch.cuda.synchronize()
    return O.cpu().numpy()


def run_single(lib, I, F, plan=None, variant=0):
    Wy, Wx = I.shape
    M, K, _ = F.shape
    It, Ft = torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()
    O = torch.empty((M, Wy - K + 1, Wx - K + 1), device="cuda")
    if plan is None:
        rc = lib.dconv_single_variant(It.data_ptr(), Ft.data_ptr(), O.data_ptr(), Wx, Wy, K, M,
                                      variant, _stream())
    else:
        rc = lib.dconv_single_with_plan(It.data_ptr(), Ft.data_ptr(), O.data_ptr(), Wx, Wy, K, M,
                                        ctypes.byref(dc.Plan(**plan)), _stream())
    assert rc == 0, rc
    torch.cuda.synchronize()
    return O.cpu().numpy()


@pytest.mark.parametrize("name", list(MULTI_CONFIGS))
def test_poisoned_multi_workloads(lib, name):
    I, F = make(name)
    O64, A64 = oracle_multi(I, F)
    for variant in (dc.dconv.VARIANT_MFMA, dc.dconv.VARIANT_VALU):
        assert_within(run_multi(lib, I, F, variant=variant), O64, A64, "%s/%d" % (name, variant))


@pytest.mark.parametrize("name", list(SINGLE_4096_SWEEP))
def test_poisoned_single_workloads(lib, name):
    w = WORKLOADS[name]
    I, F = make(name)
    O64, A64 = oracle_single(I, F)
    fams = [dc.dconv.VARIANT_VALU] + ([dc.dconv.VARIANT_MFMA] if w.K >= 5 else [])
    for variant in fams:
        assert_within(run_single(lib, I, F, variant=variant), O64, A64, "%s/%d" % (name, variant))


@pytest.mark.parametrize("layer", [(33, 70, 23, 19, 3), (130, 7, 9, 9, 3), (20, 65, 15, 13, 4),
                                   (8, 33, 12, 12, 1), (64, 64, 7, 7, 7)])
def test_poisoned_multi_every_plan(lib, layer):
    C, M, Wx, Wy, K = layer
    I, F = random_arrays(C, M, Wx, Wy, K, seed=sum(layer) * 13, variant="int")
    O64, _ = oracle_multi(I, F)
    for p in dc.plan_multi_candidates(C, M, Wx, Wy, K):
        assert_exact(run_multi(lib, I, F, plan=p), O64, "%r %r" % (layer, p))


@pytest.mark.parametrize("layer", [(40, 36, 3, 12), (70, 33, 5, 9), (132, 61, 7, 5),
                                   (64, 64, 11, 3), (301, 40, 3, 2)])
def test_poisoned_single_every_plan(lib, layer):
    Wx, Wy, K, M = layer
    I, F = random_arrays(1, M, Wx, Wy, K, seed=sum(layer) * 19, variant="int")
    I, F = I[0], F[:, 0]
    O64, _ = oracle_single(I, F)
    if Wx % 4 == 0:
        plans = dc.plan_single_candidates(Wx, Wy, K, M)
    else:  # single-float staging: the planned kernel only
        plans = [None]
    for p in plans:
        assert_exact(run_single(lib, I, F, plan=p), O64, "%r %r" % (layer, p))
