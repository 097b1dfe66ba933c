"""The C ABI without a GPU: the library loads, exports what include/dconv.h
declares, validates arguments before any HIP call, and plans launches whose
grids cover every output and fit the gfx950 limits (host logic only)."""
import ctypes
import os
import re

import pytest

import paper_2212_00404_amd as dc
from dconv_workloads import WORKLOADS
from random_shapes import MULTI_RANDOM, SINGLE_RANDOM

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dconv.h")
LDS_MAX = 160 * 1024

# non-NULL placeholders: validation rejects before anything is dereferenced
P = ctypes.c_void_p(0x1000)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dconv_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = dc.load()
    names = declared_functions()
    assert set(names) == set(dc.EXPORTED), names
    for name in names:
        assert hasattr(lib, name), name


def test_only_api_symbols_are_exported():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", dc.dconv.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    text_syms = [l.split()[-1] for l in out.splitlines() if " T " in l]
    assert sorted(text_syms) == sorted(dc.EXPORTED)


def test_null_pointers():
    lib = dc.load()
    assert lib.dconv_single(None, P, P, 8, 8, 3, 1, None) == dc.dconv.ENULL
    assert lib.dconv_single(P, None, P, 8, 8, 3, 1, None) == dc.dconv.ENULL
    assert lib.dconv_single(P, P, None, 8, 8, 3, 1, None) == dc.dconv.ENULL
    assert lib.dconv_multi(None, P, P, 2, 2, 8, 8, 3, None) == dc.dconv.ENULL
    assert lib.dconv_multi_variant(P, P, None, 2, 2, 8, 8, 3, 0, None) == dc.dconv.ENULL


@pytest.mark.parametrize("args", [
    (8, 8, 0, 1),     # K < 1
    (8, 8, 9, 1),     # K > Wx
    (9, 4, 5, 1),     # K > Wy (argument order Wx, Wy, K, M)
    (8, 8, 3, 0),     # M < 1
    (0, 8, 1, 1),     # Wx < 1
])
def test_single_invalid_sizes(args):
    Wx, Wy, K, M = args
    assert dc.load().dconv_single(P, P, P, Wx, Wy, K, M, None) == dc.dconv.EINVAL


@pytest.mark.parametrize("args", [
    (0, 2, 8, 8, 3),   # C < 1
    (2, 0, 8, 8, 3),   # M < 1
    (2, 2, 8, 8, 0),   # K < 1
    (2, 2, 4, 9, 5),   # K > Wx (order C, M, Wx, Wy, K)
    (2, 2, 9, 4, 5),   # K > Wy
])
def test_multi_invalid_sizes(args):
    C, M, Wx, Wy, K = args
    assert dc.load().dconv_multi(P, P, P, C, M, Wx, Wy, K, None) == dc.dconv.EINVAL


def test_bad_variant():
    assert dc.load().dconv_multi_variant(P, P, P, 2, 2, 8, 8, 3, 7, None) == dc.dconv.EINVAL


def test_range_limits():
    lib = dc.load()
    # input 65536 x 65536 = 2^32 elements
    assert lib.dconv_single(P, P, P, 65536, 65536, 3, 1, None) == dc.dconv.ERANGE
    # filters: M*C*K*K = 2^31
    assert lib.dconv_multi(P, P, P, 65536, 32768, 1, 1, 1, None) == dc.dconv.ERANGE
    # output M*Hout*Wout > 2^31-1
    assert lib.dconv_single(P, P, P, 40000, 40000, 1, 2, None) == dc.dconv.ERANGE


def test_library_allocates_no_device_memory():
    """The ABI promises no device allocation: the library imports no HIP
    allocator (hipMalloc*, hipFree*, hipExtMalloc*, memory pools)."""
    import subprocess
    out = subprocess.run(["nm", "-D", "--undefined-only", dc.dconv.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    imported = [l.split()[-1] for l in out.splitlines() if l.strip()]
    assert imported, "no imported symbols found"
    bad = [s for s in imported if re.match(r"hip(Ext)?(Malloc|Free|MemPool|HostAlloc|MallocAsync)", s)]
    assert bad == [], bad


def test_strerror():
    for code in (0, -1, -2, -3, -4, -5):
        assert dc.strerror(code) and dc.strerror(code) != "unknown status"
    assert dc.strerror(12345) == "unknown status"


def _check_single_plan(Wx, Wy, K, M, variant="auto"):
    p = dc.plan_single(Wx, Wy, K, M, variant=variant)
    Hout, Wout = Wy - K + 1, Wx - K + 1
    assert p["lds_bytes"] <= LDS_MAX
    assert p["block"] in (64, 128, 256, 512, 1024)
    if p["kernel"] in (0, 2, 3):   # persistent tiled kernels: each workgroup walks a run of tiles
        tiles_x = -(-Wout // p["tile_w"])
        tiles_y = -(-Hout // p["tile_h"])
        assert 1 <= p["grid_x"] <= tiles_x * tiles_y
        assert p["grid_x"] * p["grid_y"] <= 4 * 256
        assert (p["kernel"] == 3) == (p["variant"] == dc.dconv.VARIANT_MFMA)
        assert p["grid_y"] * p["tile_m"] >= M
        assert (p["grid_y"] - 1) * p["tile_m"] < M
    else:
        assert p["grid_x"] * p["block"] >= M * Hout * Wout
    return p


def _check_multi_plan(C, M, Wx, Wy, K, variant="auto"):
    p = dc.plan_multi(C, M, Wx, Wy, K, variant)
    Hout, Wout = Wy - K + 1, Wx - K + 1
    assert p["lds_bytes"] <= LDS_MAX
    if p["kernel"] == 99:   # one output per thread
        assert p["grid_x"] * p["block"] >= M * Hout * Wout
        return p
    tiles = -(-Hout // p["tile_h"]) * -(-Wout // p["tile_w"])
    mtiles = -(-M // p["tile_m"])
    # one workgroup per (output tile, filter tile): the channel sum is never
    # divided among workgroups, only among the waves of one
    assert p["grid_x"] == tiles * mtiles
    assert p["waves_c"] >= 1 and p["block"] % (64 * p["waves_c"]) == 0
    assert p["block"] <= 1024
    if variant == "mfma":
        assert p["variant"] == dc.dconv.VARIANT_MFMA
        assert p["tile_h"] * p["tile_w"] <= 128
    if variant == "valu":
        assert p["variant"] == dc.dconv.VARIANT_VALU
    return p


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_plans_for_workloads(name):
    w = WORKLOADS[name]
    if w.kind == "single":
        p = _check_single_plan(w.Wx, w.Wy, w.K, w.M)
        # persistent workgroups on every one of the 256 compute units at the
        # large size
        if w.Wx >= 1024:
            assert p["grid_x"] * p["grid_y"] >= 256
    else:
        for v in ("auto", "valu") + (("mfma",) if w.K <= 11 else ()):
            _check_multi_plan(w.C, w.M, w.Wx, w.Wy, w.K, v)
        p = dc.plan_multi(w.C, w.M, w.Wx, w.Wy, w.K)
        # the matrix cores wherever a kernel exists (K <= 11)
        assert p["variant"] == (dc.dconv.VARIANT_MFMA if w.K <= 11 else dc.dconv.VARIANT_VALU)


@pytest.mark.parametrize("shape", [
    (1, 1, 1, 1), (5, 7, 3, 2), (300, 17, 5, 3), (64, 64, 11, 1), (100, 80, 13, 2),
    (4096, 4096, 11, 1), (28, 28, 5, 512), (1024, 1024, 3, 32), (37, 1000, 9, 4),
    (4100, 2100, 9, 1), (2052, 4000, 11, 2), (1024, 8192, 10, 1), (4096, 4096, 8, 100)])
def test_single_plan_shapes(shape):
    _check_single_plan(*shape)
    _check_single_plan(*shape, variant="valu")
    Wx, Wy, K, M = shape
    if 5 <= K <= 11 and Wx % 4 == 0:
        assert _check_single_plan(*shape, variant="mfma")["kernel"] == 3
    else:
        with pytest.raises(RuntimeError):
            dc.plan_single(*shape, variant="mfma")


def test_single_auto_takes_the_matrix_cores_at_k7_only():
    """The automatic single-map plan runs the matrix-core kernel at K = 7,
    where it measured faster than the vector kernel on a 4096 x 4096 map, and
    the vector kernel for every other K (and for rows that are not whole
    float4, which the matrix-core kernel cannot stage)."""
    for K in range(1, 12):
        assert dc.plan_single(4096, 4096, K, 1)["kernel"] == (3 if K == 7 else 0), K
        if K >= 5:
            assert dc.plan_single(4096, 4096, K, 1, variant="mfma")["kernel"] == 3
    # rows of 4097 floats: the vector kernel's unaligned-row form
    assert dc.plan_single(4097, 4096, 7, 1)["kernel"] == 2


@pytest.mark.parametrize("shape", [
    (1, 1, 1, 1, 1), (3, 5, 9, 7, 3), (512, 512, 9, 9, 3), (7, 33, 40, 23, 5), (2, 3, 20, 20, 9),
    (16, 16, 64, 64, 31), (64, 130, 57, 31, 7), (3, 64, 224, 224, 7), (1, 1, 4096, 2, 2)])
def test_multi_plan_shapes(shape):
    C, M, Wx, Wy, K = shape
    for v in ("auto", "valu") + (("mfma",) if K <= 11 else ()):
        _check_multi_plan(C, M, Wx, Wy, K, v)


def test_mfma_refuses_large_filters():
    with pytest.raises(RuntimeError):
        dc.plan_multi(4, 4, 20, 20, 12, "mfma")


def test_wave_split_test_shapes_split_inside_the_workgroup():
    """The GPU tests of the in-workgroup channel split (several waves summing
    one output, added through LDS) need plans that take it."""
    import split_shapes
    for s in split_shapes.THREADS + split_shapes.TWO_STREAMS:
        assert dc.plan_multi(*s)["waves_c"] > 1, s
    assert sum(dc.plan_multi(*s)["waves_c"] > 1 for s in split_shapes.REUSE) >= 3


def test_private_layers_reach_every_copy_form():
    """The layers of the private-stage GPU test still reach each copy form.
    The form a plan takes follows the kernel's rule: a plan is privately
    staged when every wave covers the whole tile (block / 64 == waves_c); its
    input planes go 16 bytes per lane when the map is at least one padded row
    (IW rounded up to 4) wide and the padded plane fits the plane slot
    (64 * ceil(K * (PT + K - 1) / 64), +16 for 16-wide instructions; 32 where a
    32-pixel tile's plane fits 32 floats), PT being the shape's pixels per
    tile."""
    from private_layers import PRIVATE_LAYERS
    pt = {5: 64, 8: 32, 9: 32, 10: 16, 11: 16, 12: 16, 15: 32}   # private shapes
    seen = set()
    for C, M, Wx, Wy, K in PRIVATE_LAYERS:
        for p in dc.plan_multi_candidates(C, M, Wx, Wy, K, "mfma"):
            if p["block"] // 64 != p["waves_c"]:
                continue
            mf = 32 if p["kernel"] in (5, 8, 9) else 16
            PT = pt[p["kernel"]]
            ics = 32 if mf == 32 and K * (PT + K - 1) <= 32 else \
                64 * -(-K * (PT + K - 1) // 64) + (16 if mf == 16 else 0)
            iw, ih = p["tile_w"] + K - 1, p["tile_h"] + K - 1
            iwp = (iw + 3) // 4 * 4
            in4 = Wx >= iwp and ih * iwp <= ics
            tx = -(-(Wx - K + 1) // p["tile_w"])
            rem = C % p["chunk_c"]
            idle = rem != 0 and rem <= (p["waves_c"] - 1) * (p["chunk_c"] // p["waves_c"])
            seen |= {"in4" if in4 else "fallback"}
            if in4 and ics == 32:
                seen.add("in4 paired planes")
            if in4 and (tx - 1) * p["tile_w"] + iwp > Wx:
                seen.add("in4 window moved left")
            if idle:
                seen.add("in4 idle waves" if in4 else "fallback idle waves")
            if p["kernel"] == 15:
                seen.add("16 x 32 eight waves")
            if K % 2 == 0:
                seen.add("even K")
    assert seen >= {"in4", "fallback", "in4 paired planes", "in4 window moved left",
                    "in4 idle waves", "fallback idle waves", "16 x 32 eight waves",
                    "even K"}, seen


def test_small_maps_take_small_tiles_and_many_waves():
    """7x7 outputs with 512 channels and filters: without dividing the
    channel sum among workgroups, filling the chip takes small tiles (at most
    16 filters x 16 pixels) and many waves per workgroup on the channel sum."""
    p = dc.plan_multi(512, 512, 9, 9, 3)
    assert p["tile_m"] * p["tile_h"] * p["tile_w"] <= 256
    assert p["waves_c"] >= 8
    assert p["grid_x"] >= 128


@pytest.mark.parametrize("shape", SINGLE_RANDOM, ids=[str(s) for s in SINGLE_RANDOM])
def test_single_plan_random(shape):
    for v in ("auto", "valu"):
        _check_single_plan(*shape, variant=v)


@pytest.mark.parametrize("shape", MULTI_RANDOM, ids=[str(s) for s in MULTI_RANDOM])
def test_multi_plan_random(shape):
    for v in ("auto", "valu") + (("mfma",) if shape[4] <= 11 else ()):
        _check_multi_plan(*shape, variant=v)



def test_source_digest_ignores_comments_only():
    """The digest that ties recorded HBM counters to a kernel build covers the
    code, not its comments."""
    from paper_2212_00404_amd.build import _code_only
    a = "int f(int x) { return x + 1; }  // one\n/* two */\n"
    b = "/* header */\nint f(int x) { return x + 1; }\n\n"
    assert _code_only(a) == _code_only(b)
    assert _code_only('s = "//kept";') == 's = "//kept";'
    assert _code_only("x = 1;") != _code_only("x = 2;")


def test_debug_builds_export_the_api():
    """The LDS-poisoning and stage-trace twins export the same entry points,
    the trace build one more (its buffer registration), which the ordinary
    library does not have."""
    import subprocess
    for lib, extra in (("libdconv_poison.so", set()),
                       ("libdconv_trace.so", {"dconv_debug_stage_trace"})):
        path = os.path.join(os.path.dirname(dc.dconv.LIB_PATH), lib)
        out = subprocess.run(["nm", "-D", "--defined-only", path],
                             capture_output=True, text=True, check=True).stdout
        syms = {l.split()[-1] for l in out.splitlines() if " T " in l}
        assert syms == set(dc.EXPORTED) | extra, (lib, syms ^ (set(dc.EXPORTED) | extra))
