"""GPU: every multi-channel plan the library can run (each workgroup shape
of both kernel families) against the oracle,
plans chosen by the caller, and the latency probe behind the paper's model.
Integer data, so every plan must be bit-exact (every
summation order of small integers is exact in fp32)."""
import numpy as np
import pytest
import torch

import paper_2212_00404_amd as dc
from dconv_workloads import random_arrays
from gpu_util import assert_exact, oracle_multi, oracle_single
from private_layers import PRIVATE_LAYERS

pytestmark = pytest.mark.gpu

LAYERS = [(33, 70, 23, 19, 3), (130, 7, 9, 9, 3), (64, 64, 7, 7, 7), (16, 40, 30, 30, 5),
          (8, 33, 12, 12, 1), (5, 9, 20, 17, 2), (20, 65, 15, 13, 4), (12, 70, 14, 16, 6),
          (40, 130, 40, 36, 3), (7, 40, 10, 9, 1), (67, 33, 31, 29, 1)]


@pytest.mark.parametrize("layer", LAYERS, ids=[str(l) for l in LAYERS])
def test_every_candidate_plan_is_exact(layer):
    C, M, Wx, Wy, K = layer
    I, F = random_arrays(C, M, Wx, Wy, K, seed=sum(layer) * 31 + 7, variant="int")
    O64, _ = oracle_multi(I, F)
    It, Ft = torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()
    cands = dc.plan_multi_candidates(C, M, Wx, Wy, K)
    assert len(cands) >= 2
    outs = [dc.multi(It, Ft, plan=p) for p in cands]
    torch.cuda.synchronize()
    for p, o in zip(cands, outs):
        assert_exact(o.cpu().numpy(), O64, "%r plan %r" % (layer, p))


@pytest.mark.parametrize("layer", PRIVATE_LAYERS, ids=[str(l) for l in PRIVATE_LAYERS])
def test_private_stage_copy_forms_are_exact(layer):
    """Every plan of the private-stage shapes (every wave covering the whole
    tile) on layers that reach each of their copy forms."""
    C, M, Wx, Wy, K = layer
    I, F = random_arrays(C, M, Wx, Wy, K, seed=sum(layer) * 17 + 3, variant="int")
    O64, _ = oracle_multi(I, F)
    It, Ft = torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()
    cands = [p for p in dc.plan_multi_candidates(C, M, Wx, Wy, K, "mfma")
             if p["block"] // 64 == p["waves_c"]]
    assert cands
    outs = [dc.multi(It, Ft, plan=p) for p in cands]
    torch.cuda.synchronize()
    for p, o in zip(cands, outs):
        assert_exact(o.cpu().numpy(), O64, "%r plan %r" % (layer, p))


def test_paper_rule_plan_runs():
    C, M, Wx, Wy, K = 64, 128, 40, 40, 3
    I, F = random_arrays(C, M, Wx, Wy, K, seed=4242, variant="int")
    O64, _ = oracle_multi(I, F)
    p = dc.plan_multi_paper(C, M, Wx, Wy, K, dc.MI355X)
    out = dc.multi(torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda(), plan=p)
    assert_exact(out.cpu().numpy(), O64, "paper plan")


def test_foreign_plan_is_rejected():
    C, M, Wx, Wy, K = 16, 32, 20, 20, 3
    I, F = random_arrays(C, M, Wx, Wy, K, seed=1)
    It, Ft = torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()
    p = dict(dc.plan_multi(C, M, Wx, Wy, K))
    for field, delta in (("grid_x", 1), ("waves_c", 1), ("tile_m", 32), ("kernel", 7)):
        bad = dict(p, **{field: p[field] + delta})
        with pytest.raises(RuntimeError, match="invalid"):
            dc.multi(It, Ft, plan=bad)
    other = dc.plan_multi(C, M, Wx + 40, Wy, K)   # a plan for other sizes
    if other != p:
        with pytest.raises(RuntimeError):
            dc.multi(It, Ft, plan=other)


def test_latency_probe_orders_the_hierarchy():
    """A chain that fits in the vector L1 (64 KiB, 16 hops of 4 KiB) answers
    faster than one that fits in L2 (256 KiB, 1024 hops of 256 bytes), which
    answers faster than one far beyond the last-level cache (1 GiB).  The
    probe does not warm the chain, so the cached chains are walked several
    times over (the L2 one 8 times: its first, cold pass is an eighth of the
    loads)."""
    small = dc.probe_latency(1 << 16, steps=4000, stride_bytes=4096)
    mid = dc.probe_latency(1 << 18, steps=8192, stride_bytes=256)
    large = dc.probe_latency(1 << 30, steps=4000)
    for r in (small, mid, large):
        assert r["cycles_per_load"] > 20 and r["ns_per_load"] > 10
    assert small["ns_per_load"] < mid["ns_per_load"] < large["ns_per_load"]


# (Wx, Wy, K, M): single-map layers whose candidates cover tall and short
# tiles, 16-lane narrow rows, the matrix-core kernel, and filter divisions
# from one group to one filter per group
SINGLE_LAYERS = [(40, 36, 3, 12), (70, 33, 5, 9), (132, 61, 7, 5), (64, 64, 11, 3), (300, 20, 1, 6),
                 (96, 50, 9, 4), (28, 28, 3, 40)]


@pytest.mark.parametrize("layer", SINGLE_LAYERS, ids=[str(l) for l in SINGLE_LAYERS])
def test_every_single_candidate_plan_is_exact(layer):
    Wx, Wy, K, M = layer
    I, F = random_arrays(1, M, Wx, Wy, K, seed=sum(layer) * 17 + 3, variant="int")
    I, F = I[0], F[:, 0]
    O64, _ = oracle_single(I, F)
    It, Ft = torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()
    cands = dc.plan_single_candidates(Wx, Wy, K, M)
    assert len(cands) >= 2
    assert dc.plan_single(Wx, Wy, K, M) in cands
    assert dc.plan_single_paper(Wx, Wy, K, M, dc.MI355X) in cands
    outs = [dc.single(It, Ft, plan=p) for p in cands]
    torch.cuda.synchronize()
    for p, o in zip(cands, outs):
        assert_exact(o.cpu().numpy(), O64, "%r plan %r" % (layer, p))


def test_foreign_single_plan_is_rejected():
    Wx, Wy, K, M = 64, 40, 3, 4
    I, F = random_arrays(1, M, Wx, Wy, K, seed=2)
    It, Ft = torch.from_numpy(I[0]).cuda(), torch.from_numpy(F[:, 0]).cuda()
    p = dict(dc.plan_single(Wx, Wy, K, M))
    for field, delta in (("grid_x", 1), ("tile_m", 1), ("kernel", 1), ("tile_h", 4)):
        bad = dict(p, **{field: p[field] + delta})
        with pytest.raises(RuntimeError, match="invalid"):
            dc.single(It, Ft, plan=bad)
