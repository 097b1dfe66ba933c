"""GPU parity: libdconv through its C ABI against the fp64 CPU oracle.

Bar: integer-valued inputs (every partial sum exact in fp32) are bit-exact;
floating-point inputs satisfy |O - O64| <= 1e-5 * sum|I*F| per output.
Every workload runs at full size, for both kernel families on multi-channel
shapes, and a set of ragged and degenerate shapes covers tile tails,
misaligned rows, odd channel counts and the fallback kernels.
"""
import numpy as np
import pytest
import torch

import paper_2212_00404_amd as dc
import split_shapes
from dconv_workloads import WORKLOADS, make, random_arrays
from gpu_util import (assert_exact, assert_within, gpu_multi, gpu_single, oracle_multi,
                      oracle_single)

pytestmark = pytest.mark.gpu

SINGLE = sorted(n for n, w in WORKLOADS.items() if w.kind == "single")
MULTI = sorted(n for n, w in WORKLOADS.items() if w.kind == "multi")


def single_families(Wx, K):
    """Kernel families dconv_single can run for this shape (the matrix-core
    family needs K in 5..11 and rows of a multiple of 4 floats)."""
    return ["auto", "valu"] + (["mfma"] if 5 <= K <= 11 and Wx % 4 == 0 else [])


@pytest.mark.parametrize("name", SINGLE)
@pytest.mark.parametrize("variant", ["float", "int"])
def test_single_workload(name, variant):
    w = WORKLOADS[name]
    I, F = make(name, variant)
    O64, A64 = oracle_single(I, F)
    for fam in single_families(w.Wx, w.K):
        O = gpu_single(I, F, variant=fam)
        if variant == "int":
            assert_exact(O, O64, "%s/%s" % (name, fam))
        else:
            assert_within(O, O64, A64, "%s/%s" % (name, fam))


@pytest.mark.parametrize("name", MULTI)
@pytest.mark.parametrize("family", ["auto", "mfma", "valu"])
@pytest.mark.parametrize("variant", ["float", "int"])
def test_multi_workload(name, family, variant):
    I, F = make(name, variant)
    if family == "mfma" and WORKLOADS[name].K > 11:
        with pytest.raises(RuntimeError, match="cannot run"):
            gpu_multi(I, F, family)
        return
    O = gpu_multi(I, F, family)
    O64, A64 = oracle_multi(I, F)
    if variant == "int":
        assert_exact(O, O64, "%s/%s" % (name, family))
    else:
        assert_within(O, O64, A64, "%s/%s" % (name, family))


# (Wx, Wy, K, M): tails in both directions, Wx % 4 != 0 (unaligned rows), K up
# to the generic kernel (K > 11), one output, one pixel, several filters.
SINGLE_SHAPES = [
    (1, 1, 1, 1), (5, 5, 5, 2), (7, 3, 3, 1), (300, 17, 5, 3), (257, 33, 3, 1),
    (258, 70, 2, 4), (520, 65, 7, 2), (61, 200, 9, 1), (130, 45, 11, 3), (100, 80, 13, 2),
    (64, 64, 16, 1), (33, 40, 1, 5), (1030, 9, 4, 1), (96, 96, 6, 37), (80, 81, 8, 1),
    (90, 91, 10, 2),
    # matrix-core kernel: tails of its 16 x 256 tiles and 4 x 64 patches, K = 5..11
    (300, 70, 11, 2), (516, 41, 9, 1), (264, 100, 7, 3), (12, 12, 11, 1), (20, 37, 5, 4),
    (68, 9, 8, 2), (1028, 35, 10, 1), (256, 256, 6, 1),
    # large maps with K >= 8: ragged last tile column and row, unequal tile
    # runs per persistent workgroup, two filters, an even K
    (4100, 2100, 9, 1), (2052, 4000, 11, 2), (1024, 8192, 10, 1),
    # persistent workgroups with two or three tiles each (the matrix-core
    # kernel walks tiles in pairs; an odd count ends on a single tile)
    (4096, 1300, 7, 1), (4096, 1300, 11, 1),
    # rows of O off 16-byte boundaries, four filters per workgroup, output
    # above 32 MB: the vector kernel with ordinary (not non-temporal) stores
    (1024, 1024, 3, 16), (1030, 1000, 5, 16),
]


@pytest.mark.parametrize("shape", SINGLE_SHAPES, ids=[str(s) for s in SINGLE_SHAPES])
def test_single_shapes(shape):
    Wx, Wy, K, M = shape
    I, F = random_arrays(1, M, Wx, Wy, K, seed=sum(shape) * 7919)
    O64, A64 = oracle_single(I[0], F[:, 0])
    Ii, Fi = random_arrays(1, M, Wx, Wy, K, seed=sum(shape) * 7919 + 1, variant="int")
    O64i, _ = oracle_single(Ii[0], Fi[:, 0])
    for fam in single_families(Wx, K):
        assert_within(gpu_single(I[0], F[:, 0], variant=fam), O64, A64,
                      "single %r %s" % (shape, fam))
        assert_exact(gpu_single(Ii[0], Fi[:, 0], variant=fam), O64i,
                     "single int %r %s" % (shape, fam))


# (C, M, Wx, Wy, K): odd channel counts (the MFMA path pairs channels), M not a
# multiple of any filter tile, K from 1 to beyond the MFMA kernels, tiny and
# non-square maps, a filter too large for any LDS tile, and deep channel
# sums over tiny maps.
MULTI_SHAPES = [
    (1, 1, 1, 1, 1), (3, 5, 9, 7, 3), (5, 33, 12, 12, 1), (7, 40, 10, 13, 2), (2, 3, 20, 20, 4),
    (17, 70, 23, 19, 5), (9, 31, 16, 30, 6), (4, 65, 25, 25, 7), (6, 9, 20, 20, 9),
    (3, 4, 17, 21, 11), (2, 3, 40, 40, 31), (33, 129, 15, 15, 3), (64, 64, 7, 7, 7),
    (3, 64, 70, 70, 7), (130, 7, 9, 9, 3), (1, 96, 100, 3, 3),
    # one or a few outputs per filter and many channels: long channel sums
    # inside one workgroup, split over its waves (a channel count that is
    # not a multiple of any stage leaves a partial last stage)
    (1024, 32, 3, 3, 3), (1536, 32, 4, 5, 3), (1025, 33, 3, 3, 3),
]


@pytest.mark.parametrize("shape", MULTI_SHAPES, ids=[str(s) for s in MULTI_SHAPES])
def test_multi_shapes(shape):
    C, M, Wx, Wy, K = shape
    families = ["auto", "valu"] + (["mfma"] if K <= 11 else [])
    I, F = random_arrays(C, M, Wx, Wy, K, seed=sum(shape) * 104729)
    O64, A64 = oracle_multi(I, F)
    Ii, Fi = random_arrays(C, M, Wx, Wy, K, seed=sum(shape) * 104729 + 1, variant="int")
    O64i, _ = oracle_multi(Ii, Fi)
    for fam in families:
        assert_within(gpu_multi(I, F, fam), O64, A64, "multi %r %s" % (shape, fam))
        assert_exact(gpu_multi(Ii, Fi, fam), O64i, "multi int %r %s" % (shape, fam))


def test_delta_filter_is_bit_exact_on_random_floats():
    """A one-hot filter copies the shifted input exactly (x * 1 + 0 is exact)."""
    rng = np.random.default_rng(5)
    I = rng.uniform(-1, 1, (3, 40, 50)).astype(np.float32)
    F = np.zeros((4, 3, 5, 5), np.float32)
    picks = [(0, 1, 3), (2, 4, 0), (1, 0, 2), (2, 3, 4)]
    for m, (c, r, s) in enumerate(picks):
        F[m, c, r, s] = 1.0
    for fam in ("mfma", "valu"):
        O = gpu_multi(I, F, fam)
        for m, (c, r, s) in enumerate(picks):
            assert np.array_equal(O[m], I[c, r:r + 36, s:s + 46]), fam
    Fs = np.zeros((2, 7, 7), np.float32)
    Fs[0, 2, 5] = 1.0
    Fs[1, 6, 0] = 1.0
    O = gpu_single(I[0], Fs)
    assert np.array_equal(O[0], I[0, 2:36, 5:49])
    assert np.array_equal(O[1], I[0, 6:40, 0:44])


@pytest.mark.parametrize("name", ["multi_c512_9x9_m512_k3", "multi_c512_16x16_m512_k3",
                                  "single_64x64_m1_k3", "single_4096x4096_m1_k7"])
def test_repeated_calls_are_bitwise_identical(name):
    """Fixed summation order: twenty calls give the same bits (the 7x7 and
    14x14 layers split every stage's channels over the waves of a workgroup
    and add them through LDS)."""
    w = WORKLOADS[name]
    if w.kind == "multi":
        assert dc.plan_multi(w.C, w.M, w.Wx, w.Wy, w.K)["waves_c"] > 1
    I, F = make(name)
    dev = torch.device("cuda:0")
    It, Ft = torch.from_numpy(I).to(dev), torch.from_numpy(F).to(dev)
    run = (lambda: dc.single(It, Ft)) if w.kind == "single" else (lambda: dc.multi(It, Ft))
    first = run()
    outs = [run() for _ in range(19)]
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o, first)


def test_every_wave_split_plan_is_deterministic():
    """Every candidate plan with several wave groups on the channel sum,
    twenty times on the same float data: identical bits each time."""
    C, M, Wx, Wy, K = 256, 48, 9, 9, 3
    I, F = random_arrays(C, M, Wx, Wy, K, seed=777)
    dev = torch.device("cuda:0")
    It, Ft = torch.from_numpy(I).to(dev), torch.from_numpy(F).to(dev)
    plans = [p for p in dc.plan_multi_candidates(C, M, Wx, Wy, K) if p["waves_c"] > 1]
    assert len(plans) >= 4
    for p in plans:
        first = dc.multi(It, Ft, plan=p)
        outs = [dc.multi(It, Ft, plan=p) for _ in range(19)]
        torch.cuda.synchronize()
        for o in outs:
            assert torch.equal(o, first), p


def test_every_output_written_on_a_side_stream():
    """Output buffer pre-filled with NaN, work enqueued on a non-default stream."""
    I, F = make("multi_c256_28x28_m256_k1")
    It = torch.from_numpy(I).cuda()
    Ft = torch.from_numpy(F).cuda()
    out = torch.full((256, 28, 28), float("nan"), device="cuda")
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        dc.multi(It, Ft, out=out)
    s.synchronize()
    O64, A64 = oracle_multi(I, F)
    assert_within(out.cpu().numpy(), O64, A64, "side stream")
    Is, Fs = make("single_64x64_m1_k3")
    outs = torch.full((1, 62, 62), float("nan"), device="cuda")
    with torch.cuda.stream(s):
        dc.single(torch.from_numpy(Is).cuda(), torch.from_numpy(Fs).cuda(), out=outs)
    s.synchronize()
    O64, A64 = oracle_single(Is, Fs)
    assert_within(outs.cpu().numpy(), O64, A64, "side stream single")


def test_wave_split_plans_back_to_back():
    """Calls with different plans (with and without the in-workgroup split of
    the channel sum) queued back to back on one stream: each leaves nothing
    behind that the next one reads."""
    shapes = split_shapes.REUSE
    splits = [dc.plan_multi(*s)["waves_c"] for s in shapes]
    assert sum(sp > 1 for sp in splits) >= 3, splits
    cases = []
    for i, (C, M, Wx, Wy, K) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, K, seed=9000 + i, variant="int")
        cases.append((I, F, torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()))
    torch.cuda.synchronize()
    outs = [dc.multi(It, Ft) for _, _, It, Ft in cases]
    torch.cuda.synchronize()
    for (I, F, _, _), out, s in zip(cases, outs, shapes):
        O64, _ = oracle_multi(I, F)
        assert_exact(out.cpu().numpy(), O64, "reuse %r" % (s,))


def test_wave_split_calls_on_two_streams():
    """Wave-split calls on two streams at once share nothing but the device."""
    shapes = split_shapes.TWO_STREAMS
    assert all(dc.plan_multi(*s)["waves_c"] > 1 for s in shapes)
    data = [random_arrays(*s, seed=9100 + i, variant="int") for i, s in enumerate(shapes)]
    dev = [(torch.from_numpy(I).cuda(), torch.from_numpy(F).cuda()) for I, F in data]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    outs = [[], []]
    for _ in range(3):
        for k in range(2):
            with torch.cuda.stream(streams[k]):
                outs[k].append(dc.multi(*dev[k]))
    torch.cuda.synchronize()
    for k in range(2):
        O64, _ = oracle_multi(*data[k])
        for o in outs[k]:
            assert_exact(o.cpu().numpy(), O64, "stream %d" % k)


def test_calls_from_several_host_threads():
    """Four host threads, each with its own stream, issue wave-split
    multi-channel and single-map calls at once (the C calls run without the
    Python lock): the property cache and the planners are shared, and every
    result must still be exact."""
    import threading

    shapes = split_shapes.THREADS
    assert all(dc.plan_multi(*s)["waves_c"] > 1 for s in shapes)
    data = [random_arrays(*s, seed=9200 + i, variant="int") for i, s in enumerate(shapes)]
    Is, Fs = random_arrays(1, 3, 300, 200, 5, seed=9300, variant="int")
    dev = torch.device("cuda:0")
    inputs = [(torch.from_numpy(I).to(dev), torch.from_numpy(F).to(dev)) for I, F in data]
    single_in = (torch.from_numpy(Is[0]).to(dev), torch.from_numpy(Fs[:, 0]).to(dev))
    torch.cuda.synchronize()
    outs = [[] for _ in shapes]
    errors = []

    def worker(k):
        try:
            torch.cuda.set_device(dev)
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for _ in range(8):
                    outs[k].append((dc.multi(*inputs[k]), dc.single(*single_in)))
            s.synchronize()
        except Exception as e:  # reported below, on the main thread
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(len(shapes))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    O64s, _ = oracle_single(Is[0], Fs[:, 0])
    for k, (I, F) in enumerate(data):
        O64, _ = oracle_multi(I, F)
        assert len(outs[k]) == 8
        for om, osg in outs[k]:
            assert_exact(om.cpu().numpy(), O64, "thread %d multi" % k)
            assert_exact(osg.cpu().numpy(), O64s, "thread %d single" % k)


def _offset_view(host, offset, dev, guard=4):
    """A contiguous device view of `host` whose first element sits `offset`
    floats past a fresh allocation (so 4 * offset bytes off its alignment),
    with NaN in the `offset` floats before it and `guard` floats after it."""
    flat = torch.full((offset + host.size + guard,), float("nan"), dtype=torch.float32, device=dev)
    view = flat[offset:offset + host.size].view(host.shape)
    view.copy_(torch.from_numpy(np.ascontiguousarray(host)))
    return flat, view


def _guards_intact(flat, offset, n):
    f = flat.cpu().numpy()
    return np.isnan(f[:offset]).all() and np.isnan(f[offset + n:]).all()


# (offset of I, of F, of O) in floats: every base address off 16-byte
# alignment in turn, and all three at once
OFFSETS = [(1, 2, 3), (0, 0, 1), (0, 0, 2), (2, 0, 0), (3, 1, 0), (1, 1, 1)]


@pytest.mark.parametrize("offsets", OFFSETS, ids=[str(o) for o in OFFSETS])
def test_misaligned_base_pointers(offsets):
    """I, F and O passed as views whose base pointers are 4, 8 or 12 bytes
    off a 16-byte boundary (the planners choose float4 staging, the
    matrix-core single-map kernel and the store kind from the pointers'
    alignment): results match the oracle and nothing outside O is written."""
    oi, of, oo = offsets
    dev = torch.device("cuda:0")
    # single map: float4 and single-float staging, non-temporal and ordinary
    # stores (four filters per workgroup and 64 MB of output), matrix cores
    for (Wx, Wy, K, M) in [(300, 70, 5, 3), (1024, 1024, 3, 16), (260, 40, 7, 2)]:
        I, F = random_arrays(1, M, Wx, Wy, K, seed=Wx * 31 + K + 17 * oi + of, variant="int")
        I, F = I[0], F[:, 0]
        O64, _ = oracle_single(I, F)
        _, It = _offset_view(I, oi, dev)
        _, Ft = _offset_view(F, of, dev)
        for fam in single_families(Wx, K):
            flat, Ot = _offset_view(np.zeros(O64.shape, np.float32), oo, dev)
            if fam == "mfma" and oi % 4:
                # the matrix-core kernel stages whole 16-byte rows
                with pytest.raises(RuntimeError, match="cannot run"):
                    dc.single(It, Ft, out=Ot, variant=fam)
                continue
            dc.single(It, Ft, out=Ot, variant=fam)
            torch.cuda.synchronize()
            assert_exact(Ot.cpu().numpy(), O64, "single %r %s %r" % ((Wx, Wy, K, M), fam, offsets))
            assert _guards_intact(flat, oo, O64.size), "single wrote outside O"
    for (C, M, Wx, Wy, K) in [(33, 70, 23, 19, 3), (256, 40, 9, 9, 3), (20, 24, 14, 13, 1),
                              (6, 9, 20, 20, 9)]:
        I, F = random_arrays(C, M, Wx, Wy, K, seed=C * 131 + K + 7 * oo, variant="int")
        O64, _ = oracle_multi(I, F)
        _, It = _offset_view(I, oi, dev)
        _, Ft = _offset_view(F, of, dev)
        for fam in ["auto", "valu"] + (["mfma"] if K <= 11 else []):
            flat, Ot = _offset_view(np.zeros(O64.shape, np.float32), oo, dev)
            dc.multi(It, Ft, out=Ot, variant=fam)
            torch.cuda.synchronize()
            assert_exact(Ot.cpu().numpy(), O64, "multi %r %s %r" % ((C, M, Wx, Wy, K), fam, offsets))
            assert _guards_intact(flat, oo, O64.size), "multi wrote outside O"
