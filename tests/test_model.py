"""The paper's partition model (Section 2.2, Table 1; Sections 3.1, 3.2) and
the plan enumeration it is compared against (host logic, no GPU).

Pins: Table 1's printed figures for the GTX 1080 Ti (tests/golden), and the
defining inequalities of P, Q and M' (each chosen factor meets its bounds and
is the smallest that does)."""
import json
import math
import os

import pytest

import paper_2212_00404_amd as dc

HERE = os.path.dirname(os.path.abspath(__file__))
TABLE1 = json.load(open(os.path.join(HERE, "golden", "table1_gtx1080ti.json")))


def test_table1_reproduced():
    t = TABLE1["inputs"]
    assert dc.GTX_1080TI == dict(
        latency_clk=t["global_memory_latency_clk"], bandwidth_gbs=t["bandwidth_gbs"],
        clock_mhz=t["base_clock_mhz"], num_cu=t["sm"], lanes_per_cu=t["cores_per_sm"],
        ops_per_clk_lane=t["flops_per_clock_per_core"], wave_size=t["warp_size"],
        word_bytes=t["word_bytes"], onchip_bytes=t["shared_memory_bytes"])
    m = dc.model_latency(dc.GTX_1080TI)
    d = TABLE1["derived"]
    assert m["n_fma"] == d["n_fma"]
    assert m["bytes_per_clk"] == d["transmission_rate_bytes_per_clk"]
    assert m["data_bytes"] == d["data_requirement_bytes"]
    assert m["threads_per_cu"] == d["thread_requirement_per_sm"]
    assert m["threads_total"] == d["threads_total"]
    assert m["waves_per_cu"] == d["warp_requirement_per_sm"]
    assert m["bytes_per_cu"] == d["data_requirement_per_sm_bytes"]
    assert m["v_s"] == d["v_s_bytes"]
    assert m["v_s"] >= m["data_bytes"]


def test_latency_model_scales():
    base = dict(dc.GTX_1080TI)
    m1 = dc.model_latency(base)
    m2 = dc.model_latency(dict(base, latency_clk=2 * base["latency_clk"]))
    assert m2["n_fma"] == 2 * m1["n_fma"]
    assert m2["data_bytes"] == 2 * m1["data_bytes"]
    assert dc.model_latency(dict(base, num_cu=56))["threads_per_cu"] <= m1["threads_per_cu"]


def test_mi355x_figures():
    with pytest.raises(ValueError):
        dc.model_latency(dict(dc.MI355X, latency_clk=None))
    m = dc.model_latency(dc.MI355X)
    assert m["bytes_per_clk"] == 3333                  # 8 TB/s / 2.4 GHz
    assert m["n_fma"] == 900 * 64 * 2
    assert m["data_bytes"] == 3333 * 900
    assert m["threads_per_cu"] % 64 == 0
    assert m["v_s"] >= m["data_bytes"]


def _d1(dev, Wx, Wy, K, M, P):
    return (K * K * math.ceil(M / dev["num_cu"]) + (math.ceil(Wy / P) + K - 1) * Wx) * 4


def _d2(dev, Wx, Wy, K, M, Q):
    return (K * K * math.ceil(M / Q) + (math.ceil(Wy / dev["num_cu"]) + K - 1) * Wx) * 4


def _th1(dev, Wx, Wy, K, M, P):
    return K * K * math.ceil(M / dev["num_cu"]) * math.ceil(Wy / P) * Wx


def _th2(dev, Wx, Wy, K, M, Q):
    return K * K * math.ceil(M / Q) * math.ceil(Wy / dev["num_cu"]) * Wx


SINGLE_LAYERS = [(4096, 4096, 3, 1), (4096, 4096, 11, 1), (224, 224, 3, 64), (28, 28, 5, 512),
                 (1024, 1024, 1, 32), (112, 112, 5, 256), (56, 56, 3, 128)]


@pytest.mark.parametrize("dev", ["gtx", "mi355x"])
@pytest.mark.parametrize("layer", SINGLE_LAYERS)
def test_single_division_meets_its_bounds(dev, layer):
    d = dc.GTX_1080TI if dev == "gtx" else dc.MI355X
    Wx, Wy, K, M = layer
    n_fma = dc.model_latency(d)["n_fma"]
    r = dc.model_single(d, Wx, Wy, K, M)
    S = d["onchip_bytes"]
    # the reported footprints and work are the formulas at the chosen factors
    P = r["P"] if r["method"] == 1 else (r["p_lo"] if r["p_admissible"] else 1)
    Q = r["Q"] if r["method"] == 2 else (r["q_lo"] if r["q_admissible"] else 1)
    assert r["D1"] == _d1(d, Wx, Wy, K, M, P) and r["Th1"] == _th1(d, Wx, Wy, K, M, P)
    assert r["D2"] == _d2(d, Wx, Wy, K, M, Q) and r["Th2"] == _th2(d, Wx, Wy, K, M, Q)
    # admissible factors fit on chip, keep N_FMA of work, and are the smallest that fit
    if r["p_admissible"]:
        p = r["p_lo"]
        assert 1 <= p <= min(Wy, r["p_hi"])
        assert _d1(d, Wx, Wy, K, M, p) <= S and _th1(d, Wx, Wy, K, M, p) >= n_fma
        assert p == 1 or _d1(d, Wx, Wy, K, M, p - 1) > S
    if r["q_admissible"]:
        q = r["q_lo"]
        assert 1 <= q <= min(M, r["q_hi"])
        assert _d2(d, Wx, Wy, K, M, q) <= S and _th2(d, Wx, Wy, K, M, q) >= n_fma
        assert q == 1 or _d2(d, Wx, Wy, K, M, q - 1) > S
    # the method with the smaller footprint is kept, the other factor reset
    if r["D1"] < r["D2"]:
        assert (r["method"], r["Q"]) == (1, 1)
    else:
        assert (r["method"], r["P"]) == (2, 1)


@pytest.mark.parametrize("K", [1, 3, 5, 7])
@pytest.mark.parametrize("S", [32, 64, 128])
@pytest.mark.parametrize("Wxp", [32, 64, 128, 256])
def test_multi_block_is_the_smallest_busy_set(K, S, Wxp):
    d = dc.GTX_1080TI
    n_fma = dc.model_latency(d)["n_fma"]
    b = dc.model_multi(d, K, S, Wxp)
    assert b["Wy_p"] == math.ceil(S / (4 * K))
    assert b["M_p"] * (S // 4) * Wxp >= n_fma
    assert b["M_p"] == 1 or (b["M_p"] - 1) * (S // 4) * Wxp < n_fma
    assert b["set_bytes"] == S * b["M_p"] + b["Wy_p"] * Wxp * 4
    assert b["fits"] == (2 * b["set_bytes"] <= d["onchip_bytes"])


def test_model_rejects_bad_input():
    with pytest.raises(RuntimeError):
        dc.model_latency(dict(dc.GTX_1080TI, num_cu=0))
    with pytest.raises(RuntimeError):
        dc.model_single(dc.GTX_1080TI, 4, 4, 5, 1)
    with pytest.raises(RuntimeError):
        dc.model_multi(dc.GTX_1080TI, 3, 30, 64)   # S not a multiple of the word


MULTI_LAYERS = [(512, 512, 9, 9, 3), (256, 256, 30, 30, 3), (64, 128, 114, 114, 3),
                (128, 128, 60, 60, 5), (256, 256, 28, 28, 1), (3, 64, 224, 224, 7),
                (7, 40, 10, 13, 2), (2, 3, 40, 40, 31)]


@pytest.mark.parametrize("layer", MULTI_LAYERS)
def test_candidates_cover_the_planner_and_fit(layer):
    C, M, Wx, Wy, K = layer
    cands = dc.plan_multi_candidates(C, M, Wx, Wy, K)
    assert cands
    assert dc.plan_multi(C, M, Wx, Wy, K) in cands
    for v in ("valu", "mfma"):
        if v == "mfma" and K > 11:
            continue
        sub = dc.plan_multi_candidates(C, M, Wx, Wy, K, v)
        assert dc.plan_multi(C, M, Wx, Wy, K, v) in sub
        assert all(p in cands for p in sub)
    Hout, Wout = Wy - K + 1, Wx - K + 1
    seen = set()
    for p in cands:
        key = (p["variant"], p["kernel"])
        assert key not in seen
        seen.add(key)
        assert p["lds_bytes"] <= 160 * 1024
        if p["kernel"] == 99:
            assert p["grid_x"] * p["block"] >= M * Hout * Wout
            continue
        tiles = -(-Hout // p["tile_h"]) * -(-Wout // p["tile_w"])
        assert p["grid_x"] == tiles * -(-M // p["tile_m"])


# Pixel lanes per workgroup tile of each matrix-core shape (MF x NB x WN).
MFMA_TILE_PIXELS = [32, 128, 64, 128, 128, 64, 64, 128, 32, 32, 16, 16, 16, 16, 32, 32]


@pytest.mark.parametrize("layer", MULTI_LAYERS + [(512, 512, 16, 16, 3), (512, 512, 7, 7, 3),
                                                  (512, 512, 14, 14, 1), (37, 40, 33, 20, 3)])
def test_tile_choice(layer):
    """Each matrix-core candidate's output tile wastes the fewest pixel lanes
    over the map; among such tiles it takes (K > 1) one whose input row,
    padded to whole float4s, fits in the map width, then the widest."""
    C, M, Wx, Wy, K = layer
    if K > 11:
        return
    Hout, Wout = Wy - K + 1, Wx - K + 1
    for p in dc.plan_multi_candidates(C, M, Wx, Wy, K, "mfma"):
        cap = MFMA_TILE_PIXELS[p["kernel"]]
        tiles = []
        for tpx in range(1, min(cap, Wout) + 1):
            tpy = min(cap // tpx, Hout)
            lanes = -(-Wout // tpx) * -(-Hout // tpy) * cap
            fits = K > 1 and (tpx + K - 1 + 3) // 4 * 4 <= Wx
            tiles.append((lanes, not fits, -tpx, tpy, tpx))
        best = min(tiles)
        assert (p["tile_h"], p["tile_w"]) == (best[3], best[4]), (p, best)


def test_tile_choice_examples():
    """A 7x7 output of a 9x9 map takes 4x4 tiles of 16 pixels (rows of 6
    floats, padded to 8, fit the map's 9; the equally wasteful 2x7 tile's 9,
    padded to 12, do not); a 28x28 output, 2x16 tiles of 32 pixels rather
    than 1x28; K = 1 keeps the widest tile."""
    plans = {p["kernel"]: p for p in dc.plan_multi_candidates(512, 512, 9, 9, 3, "mfma")}
    assert (plans[10]["tile_h"], plans[10]["tile_w"]) == (4, 4)
    plans = {p["kernel"]: p for p in dc.plan_multi_candidates(256, 256, 30, 30, 3, "mfma")}
    assert (plans[9]["tile_h"], plans[9]["tile_w"]) == (2, 16)
    plans = {p["kernel"]: p for p in dc.plan_multi_candidates(256, 256, 28, 28, 1, "mfma")}
    assert (plans[8]["tile_h"], plans[8]["tile_w"]) == (1, 28)


def test_planner_avoids_idle_waves():
    """With 64 channels, the deep 128-channel private shapes leave half their
    waves without channels; the planner prices that and takes another
    shape on the 56x56 1x1 layer."""
    p = dc.plan_multi(64, 64, 56, 56, 1)
    assert p["kernel"] not in (8, 9), p


@pytest.mark.parametrize("layer", MULTI_LAYERS)
def test_paper_rule_plan(layer):
    C, M, Wx, Wy, K = layer
    dev = dc.MI355X
    p = dc.plan_multi_paper(C, M, Wx, Wy, K, dev)
    cands = dc.plan_multi_candidates(C, M, Wx, Wy, K)
    assert p in cands
    n_fma = dc.model_latency(dev)["n_fma"]
    unsplit = cands   # no plan divides the channel sum among workgroups

    def work(c):
        if c["kernel"] == 99:
            return 0
        per_wg = c["tile_m"] * c["chunk_c"] * K * K * c["tile_h"] * c["tile_w"]
        max_wg = 2048 // c["block"]
        occ = min(max_wg, dev["onchip_bytes"] // c["lds_bytes"] if c["lds_bytes"] else max_wg,
                  -(-c["grid_x"] // dev["num_cu"]))
        return per_wg * max(occ, 1)

    busy = [c for c in unsplit if work(c) >= n_fma]
    if busy:
        assert work(p) >= n_fma
        assert p["tile_m"] == min(c["tile_m"] for c in busy)
        same_m = [c for c in busy if c["tile_m"] == p["tile_m"]]
        assert p["tile_h"] * p["tile_w"] == max(c["tile_h"] * c["tile_w"] for c in same_m)
    else:
        assert work(p) == max(work(c) for c in unsplit)


SINGLE_LAYERS = [(4096, 4096, 3, 1), (4096, 4096, 11, 1), (28, 28, 3, 512), (56, 56, 5, 256),
                 (112, 112, 3, 128), (224, 224, 5, 64), (512, 512, 1, 128), (1024, 1024, 3, 32),
                 (64, 64, 3, 1), (300, 70, 7, 9), (4097, 100, 9, 3)]


@pytest.mark.parametrize("layer", SINGLE_LAYERS, ids=[str(l) for l in SINGLE_LAYERS])
def test_single_candidates(layer):
    """Every single-map candidate covers the output and the filters, fits
    the LDS, and the planner's and the paper rule's plans are among them."""
    Wx, Wy, K, M = layer
    cands = dc.plan_single_candidates(Wx, Wy, K, M)
    assert cands
    assert dc.plan_single(Wx, Wy, K, M) in cands
    assert dc.plan_single_paper(Wx, Wy, K, M, dc.MI355X) in cands
    Hout, Wout = Wy - K + 1, Wx - K + 1
    seen = set()
    for p in cands:
        key = (p["kernel"], p["tile_h"], p["tile_w"], p["tile_m"], p["grid_x"], p["grid_y"])
        assert key not in seen
        seen.add(key)
        assert p["lds_bytes"] <= 160 * 1024
        if p["kernel"] == 1:
            assert p["grid_x"] * p["block"] >= M * Hout * Wout
            continue
        tiles = -(-Hout // p["tile_h"]) * -(-Wout // p["tile_w"])
        assert 1 <= p["grid_x"] <= tiles
        assert p["grid_y"] * p["tile_m"] >= M > (p["grid_y"] - 1) * p["tile_m"]
    for v in ("valu", "mfma"):
        if v == "mfma" and not (5 <= K <= 11 and Wx % 4 == 0):
            continue
        sub = dc.plan_single_candidates(Wx, Wy, K, M, v)
        assert all(p in cands for p in sub)
        assert all(p["variant"] == (2 if v == "mfma" else 1) for p in sub)


@pytest.mark.parametrize("layer", SINGLE_LAYERS, ids=[str(l) for l in SINGLE_LAYERS])
def test_single_paper_rule_plan(layer):
    """The Section 3.1 rule: method 1 takes the vector candidate whose filter
    groups are closest to min(M, N); method 2 keeps all filters in one group
    where a candidate does."""
    Wx, Wy, K, M = layer
    dev = dc.MI355X
    p = dc.plan_single_paper(Wx, Wy, K, M, dev)
    split = dc.model_single(dev, Wx, Wy, K, M)
    vec = dc.plan_single_candidates(Wx, Wy, K, M, "valu")
    assert p in vec
    if split["method"] == 1:
        target = min(M, dev["num_cu"])
        assert abs(p["grid_y"] - target) == min(abs(c["grid_y"] - target) for c in vec)
    else:
        if any(c["grid_y"] == 1 for c in vec):
            assert p["grid_y"] == 1
