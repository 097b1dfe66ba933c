"""GPU: the stage-trace debug build of the library (libdconv_trace.so, built
with -DDCONV_STAGE_TRACE): its multi-channel matrix-core kernel computes the
same results as the ordinary build, with and without a trace buffer
registered, and writes clock records whose phases come in order."""
import ctypes
import os

import numpy as np
import pytest
import torch

import paper_2212_00404_amd as dc
from dconv_workloads import WORKLOADS, make
from gpu_util import assert_within, oracle_multi

pytestmark = pytest.mark.gpu

TRACE = os.path.join(os.path.dirname(dc.dconv.LIB_PATH), "libdconv_trace.so")
STAGES, WORDS = 64, 6 + 5 * 64


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(TRACE):
        pytest.fail("libdconv_trace.so is not built (paper_2212_00404_amd/build.py builds it)")
    lib = dc.load(TRACE)
    lib.dconv_debug_stage_trace.argtypes = [ctypes.c_void_p]
    lib.dconv_debug_stage_trace.restype = None
    return lib


def _run(lib, I, F):
    C, Wy, Wx = I.shape
    M, _, K, _ = F.shape
    It, Ft = torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()
    O = torch.empty((M, Wy - K + 1, Wx - K + 1), device="cuda")
    rc = lib.dconv_multi(ctypes.c_void_p(It.data_ptr()), ctypes.c_void_p(Ft.data_ptr()),
                         ctypes.c_void_p(O.data_ptr()), C, M, Wx, Wy, K,
                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == 0, rc
    torch.cuda.synchronize()
    return O.cpu().numpy()


@pytest.mark.parametrize("name", ["multi_c256_30x30_m256_k3", "multi_c512_9x9_m512_k3"])
def test_trace_build_results_and_records(lib, name):
    w = WORKLOADS[name]
    I, F = make(name)
    O64, A64 = oracle_multi(I, F)
    assert_within(_run(lib, I, F), O64, A64, name + " (no trace buffer)")
    p = dc.plan_multi(w.C, w.M, w.Wx, w.Wy, w.K)
    buf = torch.zeros(p["grid_x"] * 2 * WORDS, dtype=torch.int64, device="cuda")
    lib.dconv_debug_stage_trace(ctypes.c_void_p(buf.data_ptr()))
    try:
        O = _run(lib, I, F)
    finally:
        lib.dconv_debug_stage_trace(None)
    assert_within(O, O64, A64, name + " (traced)")
    rec = buf.view(p["grid_x"], 2, WORDS).cpu().numpy()[:, 0, :]   # wave 0 of each workgroup
    nst = min(-(-w.C // p["chunk_c"]), STAGES)
    order = [1, 2, 3] + [6 + 5 * s + i for s in range(nst) for i in range(5)] + [4]
    steps = np.diff(rec[:, order], axis=1)
    assert (steps >= 0).all(), "phase clocks out of order"
    assert (rec[:, 5] >= rec[:, 0]).all() and (rec[:, 0] > 0).all()
