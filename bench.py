#!/usr/bin/env python3
"""Throughput of libdconv on one MI355X.

A step is one pass of the direct-convolution hot path over one batch of
synthetic input.  The default step ("dconv_configs") is eleven launches, each
with its own input and output buffers: dconv_single on the 4096 x 4096 map
with one filter for K = 3, 5, 7, 9, 11 (670 MB per pass, more than the 256 MB
Infinity Cache, so every one of these launches reads its input from HBM),
then dconv_multi on the six multi-channel layers (C = 512 at 9 x 9; C = 256
at 30 x 30; C = 512 at 16 x 16; C = 64 at 114 x 114; C = 128 at 60 x 60,
K = 5; C = 256 at 28 x 28, K = 1).  ``--workload`` selects another named
step or a single workload (one launch per step).

Prints ONE JSON line: GFLOP/s over the timed steps (2*C*M*K^2*Hout*Wout
flops per launch; the steps run back to back with HIP events only around the
whole timed region), the per-launch durations with each launch's roofline
(attainable = min(157.3 TFLOP/s, flop/byte x 8 TB/s)) from a second pass of
the same steps with a HIP event pair around every launch on the launch
stream, the roofline of the dominant launch, and the CPU oracle timed on the
host cores.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

METRIC = "GFLOP/s and % fp32 roofline for dconv_single/dconv_multi (fp32, 1 MI355X)"
PEAK_FP32_VECTOR_TFLOPS = 157.3      # 256 CU x 2.4 GHz x 256 flop/clk (packed FMA)
PEAK_FP32_UNPACKED_TFLOPS = 78.6     # one fp32 FMA per lane per clock
PEAK_FP32_MFMA_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
SWEEP = "single_4096x4096_m1_k3-11"
DEFAULT_STEP = "dconv_configs"
# Named multi-launch steps: the default (the single-map sweep and the six
# multi-channel layers), the single-map sweep alone, single-map layers with
# many filters, the multi-channel layers alone, the paper's layer sweep, two
# large-filter multi-channel layers, and 4096-wide maps of 1 to 8 rounds of
# tiles per workgroup.
SWEEPS = (DEFAULT_STEP, SWEEP, "single_multi_filter", "multi_layers", "paper_multi_sweep",
          "large_filter_layers", "single_rounds")


def step_names(workload):
    """The workloads of a named step, or [workload] for a single one."""
    import dconv_workloads as dw
    steps = {DEFAULT_STEP: list(dw.SINGLE_4096_SWEEP) + list(dw.MULTI_CONFIGS),
             SWEEP: list(dw.SINGLE_4096_SWEEP), "single_multi_filter": list(dw.SINGLE_MULTI_FILTER),
             "multi_layers": list(dw.MULTI_CONFIGS), "paper_multi_sweep": list(dw.PAPER_MULTI_SWEEP),
             "large_filter_layers": list(dw.LARGE_FILTER_LAYERS),
             "single_rounds": list(dw.SINGLE_ROUNDS)}
    return steps.get(workload, [workload])
# Sources each kernel family is built from: recorded HBM traffic stays valid
# while these are unchanged.
SINGLE_SOURCES = ("single.hip", "xcd.h")
MULTI_SOURCES = ("multi.hip", "multi_kernels.h", "multi_mfma_k1_3.hip", "multi_mfma_k4_6.hip",
                 "multi_mfma_k7_9.hip", "multi_mfma_k10_11.hip", "xcd.h")


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_STEP,
                    help="%s (default), %s, or a name from dconv_workloads.WORKLOADS"
                         % (SWEEPS[0], ", ".join(SWEEPS[1:])))
    ap.add_argument("--variant", default="auto", choices=["auto", "mfma", "valu"],
                    help="kernel family: multi-channel workloads; for the single map, "
                         "mfma runs the matrix-core kernel where it exists (K = 5 ... 11)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-reps", type=int, default=2)
    ap.add_argument("--collect-counters", metavar="DIR",
                    help="run rocprofv3 (kernel trace, SQ counters of both kernel families, "
                         "FETCH_SIZE, WRITE_SIZE) over every launch of the step, one child "
                         "process per workload and pass, results under DIR; this process "
                         "never touches the GPU")
    ap.add_argument("--counter-report", metavar="DIR",
                    help="turn the rocprofv3 results under DIR (from --collect-counters) into "
                         "the markdown tables of --report-out and update profiles/traffic.json")
    ap.add_argument("--trace-report", metavar="DIR",
                    help="turn a rocprofv3 --kernel-trace --stats run of this benchmark under "
                         "DIR into a per-launch table (kernel, calls, average us, TFLOP/s, "
                         "roofline fraction); --report-out names the file")
    ap.add_argument("--report-out", metavar="FILE",
                    help="where --counter-report writes its tables (default: stdout)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="instead of convolving, copy a MIB-sized device buffer --steps "
                         "times (reference kernel for scaling HBM byte counters)")
    ap.add_argument("--stage-trace", action="store_true",
                    help="run each multi-channel workload of the step on the stage-trace build "
                         "(libdconv_trace.so) and report where a stage's clocks go (copy wait, "
                         "barrier, issuing the next stage's copies, MFMAs) for the first and "
                         "the last wave of every workgroup; --report-out names the file")
    ap.add_argument("--peaks", action="store_true",
                    help="instead of convolving, run the peak microbenchmarks (HBM read, write "
                         "and copy streams, fp32 FMA, fp32 MFMA 32x32x2 and 16x16x4, global->LDS "
                         "copies of 4 and 16 bytes per lane); one JSON line")
    ap.add_argument("--latency-probe", action="store_true",
                    help="instead of convolving, measure dependent-load latency over chains of "
                         "64 KiB to 4 GiB (the latency input of the paper's partition model); "
                         "one JSON line per footprint and stride")
    ap.add_argument("--miopen", action="store_true",
                    help="also time torch.nn.functional.conv2d (MIOpen on ROCm, fp32 with "
                         "TF32 disabled) on each workload of the step, as "
                         "context beside each kernel's time")
    ap.add_argument("--heldout", type=int, default=0, metavar="N",
                    help="time every matrix-core candidate plan of N seeded random layer shapes "
                         "and the planner's choice; one JSON line per shape (the default seed's "
                         "shapes were not used to fit the planner's time model)")
    ap.add_argument("--heldout-seed", type=int, default=7,
                    help="seed of the --heldout shape generator (the time model was fitted on "
                         "the first 24 shapes of seeds 20221230 and 11)")
    ap.add_argument("--autotune", action="store_true",
                    help="for the multi-channel workload(s), time every candidate plan, the "
                         "planner's choice and the paper-rule choice; one JSON line per workload")
    return ap.parse_args()


def latency_probe():
    """dconv_probe_latency over random cyclic chains of growing footprint."""
    import paper_2212_00404_amd as dc
    for fp in (1 << 16, 1 << 20, 1 << 22, 1 << 24, 1 << 26, 1 << 28, 1 << 30, 1 << 32):
        for stride in (256, 4096):
            print(json.dumps(dc.probe_latency(fp, steps=20000, stride_bytes=stride)), flush=True)


def autotune(names, steps, warmup, report_out=None):
    """Per multi-channel workload: the time of every candidate plan (both
    kernel families, every workgroup shape), of the
    planner's choice and of the plan the paper's Section 3.2 rules pick for
    an MI355X.  Each plan is timed over `steps` back-to-back launches."""
    import torch
    import paper_2212_00404_amd as dc
    from dconv_workloads import WORKLOADS, make
    dev = torch.device("cuda:0")
    results = []
    for n in names:
        w = WORKLOADS[n]
        I, F = make(w)
        It, Ft = torch.from_numpy(I).to(dev), torch.from_numpy(F).to(dev)
        Ot = torch.empty((w.M, w.Hout, w.Wout), device=dev)
        single = w.kind == "single"
        args = (w.Wx, w.Wy, w.K, w.M) if single else (w.C, w.M, w.Wx, w.Wy, w.K)
        run = dc.single if single else dc.multi

        def timed(plan):
            for _ in range(warmup):
                run(It, Ft, out=Ot, plan=plan)
            torch.cuda.synchronize()
            try:
                torch.cuda._sleep(int(min(0.2, 6e-5 * steps) * 2.0e9))
            except (AttributeError, RuntimeError):
                pass
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(steps):
                run(It, Ft, out=Ot, plan=plan)
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / steps * 1e3

        def tag(p):
            fam = "mfma" if p["variant"] == 2 else "valu"
            if single:   # tile, filters per group, workgroups x filter groups
                return "%s/k%d/%dx%d/m%d/g%dx%d" % (fam, p["kernel"], p["tile_h"], p["tile_w"],
                                                    p["tile_m"], p["grid_x"], p["grid_y"])
            return "%s/k%d/m%d/%dx%d/c%d/w%d" % (fam, p["kernel"], p["tile_m"], p["tile_h"],
                                                p["tile_w"], p["chunk_c"], p["waves_c"])

        if single:
            cands = dc.plan_single_candidates(*args)
            planner = tag(dc.plan_single(*args))
            paper = tag(dc.plan_single_paper(*args, dc.MI355X))
        else:
            cands = dc.plan_multi_candidates(*args)
            planner = tag(dc.plan_multi(*args))
            paper = tag(dc.plan_multi_paper(*args, dc.MI355X))
        times = {tag(p): round(timed(p), 2) for p in cands}
        best = min(times, key=times.get)
        us = lambda t: times[t]
        res = {"workload": n, "flops": w.flops, "candidates": len(cands),
               "best": best, "best_us": us(best),
               "planner": planner, "planner_us": us(planner),
               "paper_rule": paper, "paper_rule_us": us(paper),
               "model": dc.model_latency(dc.MI355X), "us": times}
        results.append(res)
        print(json.dumps(res), flush=True)
    if report_out:
        write_autotune_report(results, report_out)


def heldout(n, steps, warmup, seed=7, report_out=None):
    """The planner on seeded random layer shapes (seed 7: shapes it was not
    fitted on): C, M in 32..512,
    outputs 7..112 square, K in {1, 3, 5, 7} (at most 3 GFLOP each), drawn
    from a seeded generator; every matrix-core candidate plan timed over
    `steps` back-to-back launches behind a GPU-side delay."""
    import torch
    import paper_2212_00404_amd as dc
    rng = np.random.default_rng(seed)
    dev = torch.device("cuda:0")
    shapes = []
    while len(shapes) < n:
        K = int(rng.choice([1, 3, 5, 7]))
        hout = int(rng.choice([7, 12, 14, 20, 28, 40, 56, 80, 112]))
        C = int(rng.choice([32, 64, 96, 128, 192, 256, 384, 512]))
        M = int(rng.choice([32, 64, 96, 128, 192, 256, 384, 512]))
        if 2 * C * M * K * K * hout * hout <= 6e9:
            shapes.append((C, M, hout + K - 1, hout + K - 1, K))

    def tag(p):
        return "k%d/m%d/%dx%d/c%d/w%d" % (p["kernel"], p["tile_m"], p["tile_h"], p["tile_w"],
                                         p["chunk_c"], p["waves_c"])

    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    results = []
    for (C, M, Wx, Wy, K) in shapes:
        I = torch.rand((C, Wy, Wx), device=dev, generator=g)
        F = torch.randn((M, C, K, K), device=dev, generator=g) * (2.0 / (C * K * K)) ** 0.5
        O = torch.empty((M, Wy - K + 1, Wx - K + 1), device=dev)
        times = {}
        for p in dc.plan_multi_candidates(C, M, Wx, Wy, K, "mfma"):
            for _ in range(max(1, warmup)):
                dc.multi(I, F, out=O, plan=p)
            torch.cuda.synchronize()
            try:
                torch.cuda._sleep(int(min(0.2, 6e-5 * steps) * 2.0e9))
            except (AttributeError, RuntimeError):
                pass
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(steps):
                dc.multi(I, F, out=O, plan=p)
            b.record()
            torch.cuda.synchronize()
            times[tag(p)] = a.elapsed_time(b) / steps * 1e3
        planner = tag(dc.plan_multi(C, M, Wx, Wy, K))
        best = min(times, key=times.get)
        res = {"shape": {"C": C, "M": M, "Wx": Wx, "Wy": Wy, "K": K},
               "candidates": len(times), "best": best, "best_us": round(times[best], 2),
               "planner": planner, "planner_us": round(times[planner], 2),
               "planner_over_best": round(times[planner] / times[best], 3),
               "us": {t: round(v, 2) for t, v in times.items()}}
        results.append(res)
        print(json.dumps(res), flush=True)
    if report_out:
        write_heldout_report(results, report_out, seed)


def copy_probe(mib, steps):
    """A plain device-to-device copy of known size: its FETCH_SIZE/WRITE_SIZE
    counters per dispatch calibrate the counters of the convolution kernels."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.rand(n, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4,
                      "steps": steps, "gbs": round(2 * n * 4 / dt / 1e9, 1)}), flush=True)


# rocprofv3 passes of --collect-counters: (name, rocprofv3 arguments).  One
# run per pass (counter blocks are not split over passes; at most 8 SQ and 4
# TCC counters per run).
COUNTER_PASSES = (
    ("trace", ["--kernel-trace", "--stats"]),
    ("sq_mfma", ["--kernel-trace", "--pmc", "SQ_WAVES", "SQ_INSTS_VALU_MFMA_F32",
                 "SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_LDS",
                 "SQ_LDS_BANK_CONFLICT", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE"]),
    ("sq_valu", ["--kernel-trace", "--pmc", "SQ_WAVES", "SQ_INSTS_VALU", "SQ_INSTS_VALU_FMA_F32",
                 "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE"]),
    ("fetch", ["--kernel-trace", "--pmc", "FETCH_SIZE"]),
    ("write", ["--kernel-trace", "--pmc", "WRITE_SIZE"]),
)
COPY_PROBE_MIB = 512
CLOCK_GHZ = 2.4
SIMDS = 1024


def _rocprof_cmd(pass_args, out_dir, name, prog):
    return (["rocprofv3"] + pass_args + ["-d", out_dir, "-o", name, "--output-format", "csv", "--"]
            + prog)


def collect_counters(out_dir, workload, variant):
    """rocprofv3 over each launch of the step, one child process per workload
    and pass (each under a 120 s limit), plus the plain-copy calibration of
    FETCH_SIZE / WRITE_SIZE.  Never touches the GPU itself."""
    import subprocess
    names = step_names(workload)
    here = os.path.abspath(__file__)
    runs = []
    for n in names:
        prog = [sys.executable, here, "--workload", n, "--variant", variant, "--steps", "5",
                "--warmup", "1", "--no-cpu-baseline"]
        for pname, pargs in COUNTER_PASSES:
            runs.append((os.path.join(out_dir, n, pname), pname, pargs, prog))
    for pname, pargs in COUNTER_PASSES[3:]:
        prog = [sys.executable, here, "--copy-probe", str(COPY_PROBE_MIB), "--steps", "5"]
        runs.append((os.path.join(out_dir, "_copy_probe", pname), pname, pargs, prog))
    for d, pname, pargs, prog in runs:
        os.makedirs(d, exist_ok=True)
        cmd = _rocprof_cmd(pargs, d, pname, prog)
        print("counters: %s" % " ".join(cmd), flush=True)
        r = subprocess.run(cmd, stdout=subprocess.DEVNULL, stderr=subprocess.PIPE, text=True,
                           timeout=120)
        if r.returncode != 0 and not _found(d, "_kernel_stats.csv" if pname == "trace"
                                            else "_counter_collection.csv"):
            sys.exit("rocprofv3 failed (%d) for %s:\n%s" % (r.returncode, d, r.stderr[-2000:]))


def _found(d, suffix):
    for root, _, files in os.walk(d):
        for f in files:
            if f.endswith(suffix):
                return os.path.join(root, f)
    return None


def _counters_by_kernel(path):
    """{kernel name: {counter: mean value per dispatch}} of a rocprofv3
    counter_collection.csv (each counter summed over its dimension instances
    within a dispatch, then averaged over dispatches)."""
    import csv
    from collections import defaultdict
    per = defaultdict(lambda: defaultdict(float))   # (kernel, dispatch) -> counter -> sum
    for row in csv.DictReader(open(path)):
        key = (row["Kernel_Name"], row.get("Dispatch_Id", ""))
        per[key][row["Counter_Name"]] += float(row["Counter_Value"])
    out = defaultdict(lambda: defaultdict(list))
    for (k, _), cs in per.items():
        for c, v in cs.items():
            out[k][c].append(v)
    return {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in out.items()}


def _kernel_stats(path):
    """{kernel name: (calls, average ns)} of a rocprofv3 kernel_stats.csv."""
    import csv
    return {row["Name"]: (int(row["Calls"]), float(row["AverageNs"]))
            for row in csv.DictReader(open(path))}


def _short(name):
    import re
    m = re.search(r"(single_\w+|multi_\w+)<[^>]*>", name)
    return m.group(0) if m else name[:60]


def trace_report(root, workload=DEFAULT_STEP, out_path=None, command=None):
    """Per-launch table of a rocprofv3 kernel trace of this benchmark: each
    libdconv dispatch is matched to the step's workload whose plan has the
    same filter size (the kernel's first template argument), grid and
    workgroup size, with the kernel-trace average and median duration and the
    roofline of kernel_roofline()."""
    import csv
    import re
    from collections import defaultdict
    import paper_2212_00404_amd as dc
    from dconv_workloads import WORKLOADS
    names = step_names(workload)
    key = {}
    for n in names:
        w = WORKLOADS[n]
        p = launch_plan(dc, w, "auto", "auto")
        # (multi-channel kernels: filters per workgroup and wave groups too,
        # as two workloads may share a grid)
        extra = () if w.kind == "single" else (p["tile_m"], p["waves_c"])
        key[(w.kind, w.K, p["grid_x"] * p["grid_y"] * p["block"], p["block"]) + extra] = n
    tr = _found(root, "_kernel_trace.csv")
    durs = defaultdict(list)
    kname = {}
    for r in csv.DictReader(open(tr)):
        m = re.search(r"dconv::\(anonymous namespace\)::(single|multi)_\w+<([\d, a-z]+)>",
                      r["Kernel_Name"])
        if not m:
            continue
        targs = [a.strip() for a in m.group(2).split(",")]
        grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
        extra = ()
        if m.group(1) == "multi" and "multi_mfma" in r["Kernel_Name"]:
            mf, mb, wm, wc = int(targs[1]), int(targs[2]), int(targs[4]), int(targs[6])
            extra = (mf * mb * wm, wc)
        n = key.get((m.group(1), int(targs[0]), grid, int(r["Workgroup_Size_X"])) + extra)
        if n is None:
            continue
        durs[n].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
        kname.setdefault(n, r["Kernel_Name"])
    lines = ["# Kernel trace: every launch of the bench step `%s`" % workload, ""]
    if command:
        lines += ["Command:", "", "```", command, "```", ""]
    lines += ["Per launch: rocprofv3 kernel-trace durations of the libdconv kernel (all dispatches "
              "of the run: warm-up, the timed steps, the event-timed pass and the back-to-back "
              "repeats).  Roofline: attainable = min(157.3 TFLOP/s, flop/byte x 8 TB/s); `frac` = "
              "achieved / attainable at the average.", "",
              "| workload | kernel | dispatches | avg us | median us | TFLOP/s | bound | frac |",
              "|---|---|---|---|---|---|---|---|"]
    for n in names:
        if n not in durs:
            continue
        w = WORKLOADS[n]
        d = sorted(durs[n])
        avg = sum(d) / len(d)
        rf = kernel_roofline(w, avg, "multi_mfma" in kname[n])
        lines.append("| %s | `%s` | %d | %.2f | %.2f | %.2f | %s | %.3f |" % (
            n, _short(kname[n]), len(d), avg * 1e6, d[len(d) // 2] * 1e6, rf["tflops"],
            rf["bound"], rf["frac"]))
    text = "\n".join(lines) + "\n"
    if out_path:
        with open(out_path, "w") as fh:
            fh.write(text)
    else:
        print(text)


def counter_report(root, out_path=None):
    """Tables from the results of collect_counters: per workload, the main
    kernel's duration and its MFMA / VALU / LDS / HBM counters against the
    chip's peaks.  Also records the HBM bytes per launch of every kernel in
    profiles/traffic.json (tagged with the kernel sources' digest)."""
    from dconv_workloads import WORKLOADS
    from paper_2212_00404_amd.build import source_digest
    cal = {}
    for pname in ("fetch", "write"):
        f = _found(os.path.join(root, "_copy_probe", pname), "_counter_collection.csv")
        if f:
            ck = _counters_by_kernel(f)
            copy_kernel = max(ck, key=lambda k: sum(ck[k].values()))
            cnt = "FETCH_SIZE" if pname == "fetch" else "WRITE_SIZE"
            cal[pname] = (copy_kernel, ck[copy_kernel][cnt])
    copy_bytes = COPY_PROBE_MIB * (1 << 20)
    fscale = copy_bytes / (cal["fetch"][1] * 1024.0) if "fetch" in cal else None
    wscale = copy_bytes / (cal["write"][1] * 1024.0) if "write" in cal else None
    from dconv_workloads import MULTI_CONFIGS, SINGLE_4096_SWEEP, PAPER_MULTI_SWEEP
    order = list(SINGLE_4096_SWEEP) + list(MULTI_CONFIGS) + list(PAPER_MULTI_SWEEP)
    present = [n for n in os.listdir(root) if n in WORKLOADS]
    rows = []
    for n in sorted(present, key=lambda n: (order.index(n) if n in order else len(order), n)):
        w = WORKLOADS[n]
        ts = _found(os.path.join(root, n, "trace"), "_kernel_stats.csv")
        if not ts:
            continue
        stats = _kernel_stats(ts)
        main = max((k for k in stats if "dconv" in k), key=lambda k: stats[k][0] * stats[k][1])
        dur_s = stats[main][1] * 1e-9
        r = {"workload": n, "kernel": _short(main), "avg_us": dur_s * 1e6,
             "tflops": w.flops / dur_s / 1e12}
        for pname in ("sq_mfma", "sq_valu", "fetch", "write"):
            f = _found(os.path.join(root, n, pname), "_counter_collection.csv")
            if f:
                r.update(_counters_by_kernel(f).get(main, {}))
        rows.append((w, r))
    lines = ["# Counters of every launch of the default bench step", "",
             "Collected with `python3 bench.py --collect-counters <dir>` (rocprofv3 over each "
             "workload, one pass per counter set: kernel trace, "
             + "; ".join("`%s`" % " ".join(a[a.index("--pmc") + 1:]) for _, a in COUNTER_PASSES
                         if "--pmc" in a)
             + "), reported by `python3 bench.py --counter-report <dir> --report-out <file>`.",
             "Duration: rocprofv3 kernel-trace average of the main kernel.  Peaks: 157.3 TFLOP/s "
             "(fp32 matrix, and packed fp32 vector), 78.6 (one fp32 FMA per lane per clock), "
             "8 TB/s HBM; %d SIMDs at %.1f GHz." % (SIMDS, CLOCK_GHZ), ""]
    lines += ["| workload | kernel | avg us | TFLOP/s | MFMA busy | issued / algorithmic | "
              "FMA TFLOP/s | VALU busy | LDS instr | conflict cycles / LDS instr | HBM read MB | "
              "HBM write MB | HBM / algorithmic | HBM GB/s |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    traffic = {}

    def fmt(v, spec):
        return "-" if v is None else spec % v
    for w, r in rows:
        dur = r["avg_us"] * 1e-6
        busy = r.get("SQ_VALU_MFMA_BUSY_CYCLES")
        busy = busy / SIMDS / (dur * CLOCK_GHZ * 1e9) if busy else None
        mops = r.get("SQ_INSTS_VALU_MFMA_MOPS_F32")
        issued = mops * 512 / w.flops if mops else None
        fma = r.get("SQ_INSTS_VALU_FMA_F32")
        fma_tf = fma * 64 * 2 / dur / 1e12 if fma else None
        valu = r.get("SQ_INSTS_VALU")
        valu_busy = valu * 4 / SIMDS / (dur * CLOCK_GHZ * 1e9) if valu else None
        lds = r.get("SQ_INSTS_LDS")
        conf = r.get("SQ_LDS_BANK_CONFLICT")
        cpl = conf / lds if lds and conf is not None else None
        rb = r["FETCH_SIZE"] * 1024 * fscale if "FETCH_SIZE" in r and fscale else None
        wb = r["WRITE_SIZE"] * 1024 * wscale if "WRITE_SIZE" in r and wscale else None
        tot = rb + wb if rb is not None and wb is not None else None
        lines.append("| %s | `%s` | %.2f | %.1f | %s | %s | %s | %s | %s | %s | %s | %s | %s | %s |" % (
            w.name, r["kernel"], r["avg_us"], r["tflops"], fmt(busy, "%.2f"), fmt(issued, "%.3f"),
            fmt(fma_tf, "%.1f"), fmt(valu_busy, "%.2f"), fmt(lds, "%.0f"), fmt(cpl, "%.2f"),
            fmt(rb and rb / 1e6, "%.1f"), fmt(wb and wb / 1e6, "%.1f"),
            fmt(tot and tot / w.compulsory_bytes, "%.2f"), fmt(tot and tot / dur / 1e9, "%.0f")))
        if tot is not None:
            traffic[w.name] = {"kernel": r["kernel"], "fetch_kib": round(r["FETCH_SIZE"], 1),
                               "write_kib": round(r["WRITE_SIZE"], 1), "fetch_bytes": round(rb),
                               "write_bytes": round(wb), "bytes_per_launch": round(tot),
                               "source_digest": source_digest(
                                   SINGLE_SOURCES if w.kind == "single" else MULTI_SOURCES)}
    lines += ["", "HBM bytes: FETCH_SIZE and WRITE_SIZE (KiB per dispatch, what leaves the L2s: "
              "Infinity Cache hits count too) scaled so that a %d MiB device copy reads and "
              "writes %d MiB (factors %s and %s, copy kernel `%s`).  Algorithmic bytes = "
              "4 * (C*Wy*Wx + M*C*K*K + M*Hout*Wout)." % (
                  COPY_PROBE_MIB, COPY_PROBE_MIB, fmt(fscale, "%.4f"), fmt(wscale, "%.4f"),
                  cal.get("fetch", ("-",))[0][:60]),
              "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / SIMDs / (duration x clock); issued / "
              "algorithmic = SQ_INSTS_VALU_MFMA_MOPS_F32 x 512 / (2*C*M*K*K*outputs); FMA "
              "TFLOP/s = SQ_INSTS_VALU_FMA_F32 x 64 lanes x 2 / duration; VALU busy = "
              "SQ_INSTS_VALU x 4 clocks / SIMDs / (duration x clock); conflict cycles per LDS "
              "instruction = SQ_LDS_BANK_CONFLICT / SQ_INSTS_LDS."]
    text = "\n".join(lines) + "\n"
    if out_path:
        with open(out_path, "w") as fh:
            fh.write(text)
    else:
        print(text)
    if traffic:
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
        data = {"_calibration": {"copy_kernel": cal["fetch"][0], "copy_bytes": copy_bytes,
                                 "fetch_kib_per_copy": cal["fetch"][1],
                                 "write_kib_per_copy": cal["write"][1],
                                 "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4)}}
        data.update(traffic)
        with open(path, "w") as fh:
            json.dump(data, fh, indent=1, sort_keys=True)
    return rows


def traffic_for(kernel_tag, kind="single"):
    """HBM bytes per launch measured with rocprofv3 counters, if recorded
    for the current kernel sources (profiles/traffic.json); else None."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        data = json.load(open(path))
    except (OSError, ValueError):
        return None
    ent = data.get(kernel_tag)
    if not ent:
        return None
    from paper_2212_00404_amd.build import source_digest
    if ent.get("source_digest") != source_digest(SINGLE_SOURCES if kind == "single"
                                                 else MULTI_SOURCES):
        return None
    return ent.get("bytes_per_launch")


def launch_plan(dc, w, variant, single_variant):
    """The plan the library uses for workload w (host logic)."""
    if w.kind == "multi":
        return dc.plan_multi(w.C, w.M, w.Wx, w.Wy, w.K, variant)
    return dc.plan_single(w.Wx, w.Wy, w.K, w.M, variant=single_variant)


def kernel_roofline(w, avg_s, uses_mfma, measured=None):
    """Roofline of one launch of workload w taking avg_s seconds.

    Attainable = min(P, AI x 8 TB/s) with AI = flops / compulsory bytes and
    P = 157.3 TFLOP/s (the fp32 matrix peak for the matrix-core kernels, the
    packed fp32 vector peak for the vector kernels); the bound is HBM where
    AI x 8 TB/s is the smaller.  `frac` = achieved / attainable in the bound's
    unit.  With measured peaks (bench.py --peaks, recorded in
    profiles/peaks.json) the same launch is also given against them."""
    tf = w.flops / avg_s / 1e12
    gbs = w.compulsory_bytes / avg_s / 1e9
    ai = w.flops / w.compulsory_bytes
    peak = PEAK_FP32_MFMA_TFLOPS if uses_mfma else PEAK_FP32_VECTOR_TFLOPS
    hbm_roof = ai * PEAK_HBM_GBS / 1e3
    attainable = min(peak, hbm_roof)
    out = {"tflops": round(tf, 2), "gbs": round(gbs, 1), "flop_per_byte": round(ai, 2),
           "bound": "hbm" if hbm_roof < peak else ("mfma" if uses_mfma else "alu"),
           "attainable_tflops": round(attainable, 2), "frac": round(tf / attainable, 4),
           "frac_fp32_peak": round(tf / peak, 4), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}
    if not uses_mfma:
        out["frac_unpacked_fp32"] = round(tf / PEAK_FP32_UNPACKED_TFLOPS, 4)
    if measured:
        mp = measured.get("mfma_f32_32x32_tflops" if uses_mfma else "fma_fp32_tflops")
        bw = measured.get("hbm_copy_gbs")
        if mp and bw:
            att_m = min(mp, ai * bw / 1e3)
            out["frac_measured_peaks"] = round(tf / att_m, 4)
    return out


def load_measured_peaks():
    """The peaks bench.py --peaks measured, if recorded (profiles/peaks.json)."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "peaks.json")
    try:
        with open(path) as fh:
            return json.load(fh).get("peaks")
    except (OSError, ValueError):
        return None


def cpu_baseline(launches, reps, min_seconds=10.0):
    """The fp64 oracle on the host cores over the same launches: whole steps,
    repeated at least `reps` times and until `min_seconds` of CPU work have
    run; the rate of the fastest step is reported."""
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS") or 0) or oracle.default_threads()
    flops = sum(w.flops for w, _, _ in launches)
    times = []
    t_start = time.perf_counter()
    while len(times) < max(1, reps) or time.perf_counter() - t_start < min_seconds:
        t0 = time.perf_counter()
        for w, I, F in launches:
            if w.kind == "single":
                oracle.conv_single(I, F, threads=threads)
            else:
                oracle.conv_multi(I, F, threads=threads)
        times.append(time.perf_counter() - t0)
    best = min(times)
    # the same step on one thread, once (context: the oracle's per-core rate)
    t0 = time.perf_counter()
    for w, I, F in launches:
        if w.kind == "single":
            oracle.conv_single(I, F, threads=1)
        else:
            oracle.conv_multi(I, F, threads=1)
    one = time.perf_counter() - t0
    return {"value": round(flops / best / 1e9, 3), "unit": "GFLOP/s", "cores": threads,
            "kind": "oracle",
            "sample": "whole steps (%d launch%s, %.2f GFLOP each), %d repetitions in %.1f s, "
                      "fastest reported, fp64 C oracle"
                      % (len(launches), "es" if len(launches) > 1 else "", flops / 1e9,
                         len(times), sum(times)),
            "single_thread_value": round(flops / one / 1e9, 3),
            "affinity_cpus": len(os.sched_getaffinity(0)),
            "cpu_model": _cpu_model()}


def _cpu_model():
    """The host CPU's model name (what lscpu prints), or None."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def miopen_context(bufs, per_kernel, steps, warmup):
    """torch's own convolution (MIOpen) on the same inputs: a context figure
    for each workload, not a parity reference.  Eq. 1 is what conv2d computes
    with no padding, stride 1 and weights [M][C][K][K] (Eq. 2: C = 1)."""
    import torch
    import paper_2212_00404_amd as dc
    torch.backends.cudnn.allow_tf32 = False
    torch.backends.cuda.matmul.allow_tf32 = False

    def back_to_back(fn):
        for _ in range(max(warmup, 3)):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        # a GPU-side delay first, so that the launches queue up behind it and
        # short kernels are timed back to back, not at the host's launch rate
        try:
            torch.cuda._sleep(int(min(0.2, 5e-5 * steps) * 2.0e9))
        except (AttributeError, RuntimeError):
            pass
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps * 1e3

    for i, (w, It, Ft, Ot) in enumerate(bufs):
        if w.kind == "multi":
            x, wt = It[None], Ft
            run = lambda: dc.multi(It, Ft, out=Ot)
        else:
            x, wt = It[None, None], Ft[:, None]
            run = lambda: dc.single(It, Ft, out=Ot)
        ref = torch.nn.functional.conv2d(x, wt)
        us = back_to_back(lambda: torch.nn.functional.conv2d(x, wt))
        # libdconv timed the same way (the same layer back to back, events
        # only around the run), so the two figures are comparable
        ours = back_to_back(run)
        diff = (ref[0] - Ot).abs().max().item()
        scale = Ot.abs().max().item() or 1.0
        per_kernel[i]["miopen_us"] = round(us, 2)
        per_kernel[i]["miopen_tflops"] = round(w.flops / (us * 1e-6) / 1e12, 2)
        per_kernel[i]["dconv_back_to_back_us"] = round(ours, 2)
        per_kernel[i]["dconv_speedup_vs_miopen"] = round(us / ours, 3)
        per_kernel[i]["miopen_max_rel_diff"] = float("%.3g" % (diff / scale))


class KernelEvents:
    """HIP event pairs around each launch of the instrumented pass.

    Created through the HIP runtime that torch has loaded (same soname, so
    the same instance) with hipEventDisableSystemFence: the events only
    time, and the device is synchronised before they are read.  Falls back
    to torch events (default flags) if that entry point is unavailable."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, stream, steps, per_step):
        import ctypes
        import torch
        self.stream = stream
        self.kind = "hip_no_system_fence"
        try:
            hip = ctypes.CDLL("libamdhip64.so.7")
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
            hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

            def make():
                e = ctypes.c_void_p()
                if hip.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE) != 0:
                    raise OSError("hipEventCreateWithFlags failed")
                return e
            self.hip, self.ct = hip, ctypes
            self.ev = [[(make(), make()) for _ in range(per_step)] for _ in range(steps)]
            self.ends = (make(), make())
        except (OSError, AttributeError):
            self.hip = None
            self.kind = "torch_default"
            mk = lambda: torch.cuda.Event(enable_timing=True)
            self.ev = [[(mk(), mk()) for _ in range(per_step)] for _ in range(steps)]
            self.ends = (mk(), mk())
        self.sp = None if self.hip is None else self.ct.c_void_p(stream.cuda_stream)

    def _rec(self, e):
        if self.hip is None:
            e.record(self.stream)
        elif self.hip.hipEventRecord(e, self.sp) != 0:
            raise RuntimeError("hipEventRecord failed")

    def _el(self, a, b):
        if self.hip is None:
            return a.elapsed_time(b)
        f = self.ct.c_float()
        if self.hip.hipEventElapsedTime(self.ct.byref(f), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return f.value

    def record(self, s, i, which):
        self._rec(self.ev[s][i][which])

    def record_start(self):
        self._rec(self.ends[0])

    def record_stop(self):
        self._rec(self.ends[1])

    def elapsed_ms(self, s, i):
        return self._el(*self.ev[s][i])

    def total_ms(self):
        return self._el(*self.ends)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: libdconv has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.copy_probe:
        copy_probe(args.copy_probe, args.steps)
        return
    if args.latency_probe:
        latency_probe()
        return
    if args.stage_trace:
        stage_trace(args.workload if args.workload != DEFAULT_STEP else "multi_layers",
                    args.warmup, args.report_out)
        return
    if args.peaks:
        from paper_2212_00404_amd import peaks
        print(json.dumps({"peaks": peaks.run()}), flush=True)
        return
    if args.heldout:
        heldout(args.heldout, args.steps, args.warmup, seed=args.heldout_seed,
                report_out=args.report_out)
        return
    if args.autotune:
        autotune(step_names(args.workload), args.steps, args.warmup, args.report_out)
        return
    if args.collect_counters:
        collect_counters(args.collect_counters, args.workload, args.variant)
        return
    if args.trace_report:
        trace_report(args.trace_report, args.workload, args.report_out,
                     command="rocprofv3 --kernel-trace --stats -d <dir> -o bench --output-format csv "
                             "-- python3 bench.py --workload %s --steps 20 --warmup 3 "
                             "--no-cpu-baseline" % args.workload)
        return
    if args.counter_report:
        counter_report(args.counter_report, args.report_out)
        return

    import torch
    import paper_2212_00404_amd as dc
    from dconv_workloads import WORKLOADS, make

    names = step_names(args.workload)
    for n in names:
        if n not in WORKLOADS:
            sys.exit("unknown workload %s" % n)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dc.load()

    launches = []   # (workload, host I, host F)
    bufs = []       # (workload, I, F, O) on the device
    for n in names:
        w = WORKLOADS[n]
        I, F = make(w)
        launches.append((w, I, F))
        It = torch.from_numpy(I).to(dev)
        Ft = torch.from_numpy(F).to(dev)
        Ot = torch.empty((w.M, w.Hout, w.Wout), dtype=torch.float32, device=dev)
        bufs.append((w, It, Ft, Ot))
    torch.cuda.synchronize()

    def single_variant(w):
        # the matrix-core single-map kernel exists for K = 5 ... 11
        return args.variant if args.variant != "mfma" or 5 <= w.K <= 11 else "auto"

    def launch(b):
        w, It, Ft, Ot = b
        if w.kind == "single":
            dc.single(It, Ft, out=Ot, variant=single_variant(w))
        else:
            dc.multi(It, Ft, out=Ot, variant=args.variant)

    for _ in range(args.warmup):
        for b in bufs:
            launch(b)
    torch.cuda.synchronize()

    # Timed region: the K steps back to back, HIP events only at its two
    # ends, on the launch stream.  A GPU-side delay queued first lets the
    # host enqueue the timed launches ahead of the GPU, so short kernels run
    # back to back rather than at the pace of the Python launch path (the
    # delay ends before `start`).
    stream = torch.cuda.current_stream(dev)
    launches_total = args.steps * len(bufs)
    delay_cycles = int(min(0.2, 6e-5 * launches_total) * 2.0e9)

    def gpu_delay():
        try:
            torch.cuda._sleep(delay_cycles)
        except (AttributeError, RuntimeError):
            pass

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    gpu_delay()
    start.record(stream)
    for s in range(args.steps):
        for b in bufs:
            launch(b)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start.elapsed_time(stop)
    ms_per_step = total_ms / args.steps

    # Per-kernel durations: the same K steps again with a HIP event pair
    # around every launch.  An event with the default system-scope fence
    # adds about 3 us per launch (cache write-back), so these events are
    # created without it (timing only); they still add about 1.5 us per
    # launch, which is why the step time above is measured without them.
    ev = KernelEvents(stream, args.steps, len(bufs))
    torch.cuda.synchronize()
    gpu_delay()
    ev.record_start()
    for s in range(args.steps):
        for i, b in enumerate(bufs):
            ev.record(s, i, 0)
            launch(b)
            ev.record(s, i, 1)
    ev.record_stop()
    torch.cuda.synchronize()
    ms_per_step_instr = ev.total_ms() / args.steps

    step_flops = sum(w.flops for w, _, _, _ in bufs)
    value_gflops = step_flops / (ms_per_step * 1e-3) / 1e9

    measured_peaks = load_measured_peaks()
    per_kernel = []
    for i, (w, _, _, _) in enumerate(bufs):
        d = np.array([ev.elapsed_ms(s, i) for s in range(args.steps)])
        avg_s = float(d.mean()) * 1e-3
        plan = launch_plan(dc, w, args.variant, single_variant(w))
        ent = {"workload": w.name, "kernel_family": "mfma" if plan["variant"] == 2 else "valu",
               "avg_us": round(avg_s * 1e6, 2),
               "median_us": round(float(np.median(d)) * 1e3, 2)}
        ent.update(kernel_roofline(w, avg_s, plan["variant"] == 2, measured_peaks))
        per_kernel.append(ent)

    # Warm figures: each launch repeated back to back on the same buffers
    # (working sets up to the 256 MB Infinity Cache stay resident), events
    # only around the repeats.  The step above rotates through separate
    # buffers and measures the cold case.
    reps = max(1, min(args.steps, 20))
    for i, b in enumerate(bufs):
        launch(b)
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gpu_delay()
        a.record(stream)
        for _ in range(reps):
            launch(b)
        z.record(stream)
        torch.cuda.synchronize()
        per_kernel[i]["back_to_back_us"] = round(a.elapsed_time(z) / reps * 1e3, 2)

    if args.miopen:
        miopen_context(bufs, per_kernel, args.steps, args.warmup)

    # The dominant launch (the longest on average) carries the headline
    # roofline: its bound, the achieved rate in that bound's unit against the
    # datasheet peak, and the HBM bytes its counters measured.
    dom = max(range(len(bufs)), key=lambda i: per_kernel[i]["avg_us"])
    w = bufs[dom][0]
    pk = per_kernel[dom]
    uses_mfma = pk["kernel_family"] == "mfma"
    traffic = traffic_for(w.name, w.kind) if args.variant == "auto" else None
    if pk["bound"] == "hbm":
        achieved = w.compulsory_bytes / (pk["avg_us"] * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                "traffic": traffic, "kernel": w.name,
                "bytes_per_launch": w.compulsory_bytes}
    else:
        achieved = w.flops / (pk["avg_us"] * 1e-6) / 1e12
        peak = PEAK_FP32_MFMA_TFLOPS if uses_mfma else PEAK_FP32_VECTOR_TFLOPS
        roof = {"bound": pk["bound"], "achieved": round(achieved, 2),
                "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "traffic": traffic, "kernel": w.name,
                "flops_per_launch": w.flops,
                "peak_unpacked_fp32": None if uses_mfma else PEAK_FP32_UNPACKED_TFLOPS}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(launches, args.cpu_reps)

    if args.workload == DEFAULT_STEP:
        config = {"workload": DEFAULT_STEP,
                  "description": "dconv_single on a 4096x4096 map with one filter for K = 3, 5, "
                                 "7, 9, 11, then dconv_multi on six layers: C=M=512 9x9 K=3; "
                                 "C=M=256 30x30 K=3; C=M=512 16x16 K=3; C=64 M=128 114x114 K=3; "
                                 "C=M=128 60x60 K=5; C=M=256 28x28 K=1",
                  "workloads": [b[0].name for b in bufs], "variant": args.variant,
                  "launches_per_step": len(bufs),
                  "buffers": "separate I/O per launch (670 MB for the single map)"}
    elif args.workload == SWEEP:
        config = {"workload": SWEEP, "kind": "single", "Wx": 4096, "Wy": 4096, "M": 1, "C": 1,
                  "K": [3, 5, 7, 9, 11], "launches_per_step": 5, "variant": args.variant,
                  "buffers": "separate I/O per K (670 MB per step)"}
    elif args.workload in SWEEPS:
        config = {"workload": args.workload, "kind": bufs[0][0].kind,
                  "workloads": [b[0].name for b in bufs], "variant": args.variant,
                  "launches_per_step": len(bufs)}
    else:
        config = {"workload": w.name, "kind": w.kind, "C": w.C, "M": w.M, "Wx": w.Wx,
                  "Wy": w.Wy, "K": w.K, "variant": args.variant, "launches_per_step": 1}
    out = {
        "metric": METRIC, "value": round(value_gflops, 2), "unit": "GFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_with_kernel_events": round(ms_per_step_instr, 5),
        "kernel_events": ev.kind,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic", "config": config, "roofline": roof, "cpu_baseline": cpu,
        "per_kernel": per_kernel, "wall_s_timed": round(wall, 4),
        # The paper's own speedups over cuDNN v7.1 on a Pascal GPU (Section 4):
        # context only, another library on another machine.
        "paper_context": {"speedup_vs_cudnn_pascal": {
            "single_channel": {"average": 2.6, "range": [1.5, 5.6]},
            "multi_channel": {"average": 1.39, "range": [1.05, 2.0]}}},
    }
    print(json.dumps(out), flush=True)
    if args.report_out:
        write_step_report(out, args.report_out)


def stage_trace(workload, warmup, report_out=None):
    """Stage-loop timeline of the multi-channel matrix-core kernel from the
    stage-trace build (libdconv_trace.so, -DDCONV_STAGE_TRACE): per workload
    of the step, the planner's plan launched warmup + 1 times with a trace
    buffer registered; the last launch's records (two per workgroup: wave 0
    and the last wave) are summarised as medians over workgroups, in shader
    clocks and microseconds.  The trace's own global stores add a little to
    every phase."""
    import ctypes
    import torch
    import paper_2212_00404_amd as dc
    from paper_2212_00404_amd import build as pb
    from dconv_workloads import WORKLOADS, make
    stages_max, words = 64, 6 + 5 * 64
    lib = dc.load(pb.TRACE_LIB)
    lib.dconv_debug_stage_trace.argtypes = [ctypes.c_void_p]
    lib.dconv_debug_stage_trace.restype = None
    dev = torch.device("cuda:0")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    results = []
    for n in step_names(workload):
        w = WORKLOADS[n]
        if w.kind != "multi":
            continue
        p = dc.plan_multi(w.C, w.M, w.Wx, w.Wy, w.K)
        if p["variant"] != 2:
            continue
        I, F = make(w)
        It, Ft = torch.from_numpy(I).to(dev), torch.from_numpy(F).to(dev)
        Ot = torch.empty((w.M, w.Hout, w.Wout), device=dev)
        buf = torch.zeros(p["grid_x"] * 2 * words, dtype=torch.int64, device=dev)
        lib.dconv_debug_stage_trace(ctypes.c_void_p(buf.data_ptr()))
        for _ in range(warmup + 1):
            rc = lib.dconv_multi(ctypes.c_void_p(It.data_ptr()), ctypes.c_void_p(Ft.data_ptr()),
                                 ctypes.c_void_p(Ot.data_ptr()), w.C, w.M, w.Wx, w.Wy, w.K,
                                 stream)
            if rc != 0:
                sys.exit("dconv_multi (trace build) failed: %d" % rc)
        torch.cuda.synchronize()
        lib.dconv_debug_stage_trace(None)
        t = buf.cpu().numpy().reshape(p["grid_x"], 2, words).astype(np.float64)
        first = t[:, 0, :]
        ok = (first[:, 5] > first[:, 0]) & (first[:, 4] > first[:, 1])
        ghz = float(np.median((first[ok, 4] - first[ok, 1]) / (first[ok, 5] - first[ok, 0]))) / 10.0
        nst = min(-(-w.C // p["chunk_c"]), stages_max)
        med = lambda x: float(np.median(x))

        def phases(rec):
            out = []
            for k in range(4):   # wait, barrier, issue, compute
                vals = [rec[:, 6 + 5 * s + k + 1] - rec[:, 6 + 5 * s + k] for s in range(nst)]
                out.append(med(np.concatenate(vals)))
            return out
        res = {"workload": n, "plan": "k%d/m%d/%dx%d/c%d/w%d/%dwaves" % (
                   p["kernel"], p["tile_m"], p["tile_h"], p["tile_w"], p["chunk_c"], p["waves_c"],
                   p["block"] // 64),
               "workgroups": p["grid_x"], "stages": -(-w.C // p["chunk_c"]),
               "clock_ghz": round(ghz, 2),
               "setup": med(first[:, 2] - first[:, 1]), "first_copies": med(first[:, 3] - first[:, 2]),
               "wave0": phases(first), "last_wave": phases(t[:, 1, :]),
               "span_us": med(first[:, 5] - first[:, 0]) / 100.0}
        results.append(res)
        print(json.dumps(res), flush=True)
    if report_out:
        lines = ["# Stage timeline of the multi-channel matrix-core kernel", "", "Command:", "",
                 "```", _command_line(), "```", "",
                 "The stage-trace build (`libdconv_trace.so`, `-DDCONV_STAGE_TRACE`) records the "
                 "shader clock around each phase of the stage loop in wave 0 and in the last "
                 "wave of every workgroup; medians over workgroups and stages, in clocks (the "
                 "trace's own stores add a little to each phase).  Per stage: wait = this wave's "
                 "copies of the stage landing, barrier = every wave arriving, issue = issuing "
                 "the next stage's copies, MFMAs = the stage's matrix instructions (plans whose "
                 "waves stage their own channels, `w` equal to the wave count: no barrier, and "
                 "the copies are issued halfway through the MFMAs, so the MFMA phase holds "
                 "them).  Setup = "
                 "kernel start to the first copies; first copies = issuing stage 0; span = "
                 "kernel start to end of wave 0 (wall clock).", "",
                 "| workload | plan | workgroups | stages | clock GHz | setup | first copies | "
                 "wave 0: wait / barrier / issue / MFMAs | last wave: wait / barrier / issue / "
                 "MFMAs | span us |",
                 "|---|---|---|---|---|---|---|---|---|---|"]
        for r in results:
            lines.append("| %s | `%s` | %d | %d | %.2f | %d | %d | %s | %s | %.2f |" % (
                r["workload"], r["plan"], r["workgroups"], r["stages"], r["clock_ghz"],
                r["setup"], r["first_copies"], " / ".join("%d" % v for v in r["wave0"]),
                " / ".join("%d" % v for v in r["last_wave"]), r["span_us"]))
        with open(report_out, "w") as fh:
            fh.write("\n".join(lines) + "\n")


def _command_line():
    """This run's command, with the report and result paths shown as <file> and
    <dir> (any path works there)."""
    out, skip = [], None
    for a in sys.argv[1:]:
        if skip:
            out.append(skip)
            skip = None
            continue
        out.append(a)
        if a == "--report-out":
            skip = "<file>"
        elif a in ("--collect-counters", "--counter-report", "--trace-report"):
            skip = "<dir>"
    return "python3 bench.py " + " ".join(out)


def write_step_report(out, path):
    """The bench line as a markdown table (one row per launch of the step),
    with the command that produced it."""
    pk = out["per_kernel"]
    mi = any("miopen_us" in r for r in pk)
    lines = ["# bench: %s" % out["config"]["workload"], "", "Command:", "", "```",
             _command_line(), "```", "",
             "Step: %.2f GFLOP/s (%.4f ms per step over %d steps; `value` of the bench line).  "
             "Per launch: HIP events around every launch of a second pass of the same steps "
             "(avg), and the same launch repeated on its own buffers (back to back).  Roofline: "
             "attainable = min(157.3 TFLOP/s, flop/byte x 8 TB/s), `frac` = achieved / attainable."
             % (out["value"], out["ms_per_step"], out["steps"]), ""]
    head = "| workload | family | avg us | back to back us | TFLOP/s | bound | frac |"
    sep = "|---|---|---|---|---|---|---|"
    if mi:
        head += " MIOpen us | MIOpen TFLOP/s | libdconv back to back us | speedup vs MIOpen |"
        sep += "---|---|---|---|"
    lines += [head, sep]
    for r in pk:
        row = "| %s | %s | %.2f | %s | %.2f | %s | %.3f |" % (
            r["workload"], r["kernel_family"], r["avg_us"], r.get("back_to_back_us", "-"),
            r["tflops"], r["bound"], r["frac"])
        if mi:
            row += " %s | %s | %s | %s |" % (r.get("miopen_us", "-"), r.get("miopen_tflops", "-"),
                                             r.get("dconv_back_to_back_us", "-"),
                                             r.get("dconv_speedup_vs_miopen", "-"))
        lines.append(row)
    if out.get("cpu_baseline"):
        cb = out["cpu_baseline"]
        lines += ["", "CPU oracle (fp64, %d threads, %s): %.2f GFLOP/s; one thread: %.2f." % (
            cb["cores"], cb.get("cpu_model"), cb["value"], cb.get("single_thread_value", 0))]
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def write_autotune_report(results, path):
    """--autotune results (one dict per workload) as a markdown table."""
    lines = ["# Plans: exhaustive search vs the library planner vs the paper's rules",
             "", "Command:", "", "```", _command_line(), "```", "",
             "Every candidate plan timed over back-to-back launches behind a GPU-side delay (HIP "
             "events around the run).  Multi-channel (`dconv_plan_multi_candidates`: each "
             "workgroup shape of both kernel families): tags family / shape / filters per "
             "workgroup / output tile / channels per stage / wave groups on the channel sum; "
             "`paper rule` = `dconv_plan_multi_paper` (Section 3.2) with the MI355X description "
             "(N_FMA from the measured 900-clock latency): at least N_FMA multiply-adds per "
             "compute unit per stage, the fewest filters per workgroup, then the largest tile.  "
             "Single map (`dconv_plan_single_candidates`: each tile shape crossed with the "
             "division of the filters into groups): tags family / kernel / tile / filters per "
             "group / workgroups x filter groups; `paper rule` = `dconv_plan_single_paper` "
             "(Section 3.1: method 1 divides the filters over the compute units and walks the map "
             "in P pieces, method 2 divides the map and applies every filter).", "",
             "| workload | candidates | best plan | best us | planner plan | planner us | "
             "planner / best | paper-rule plan | paper-rule us | paper / best |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for d in results:
        lines.append("| %s | %d | `%s` | %.2f | `%s` | %.2f | %.3f | `%s` | %.2f | %.2f |" % (
            d["workload"], d["candidates"], d["best"], d["best_us"], d["planner"], d["planner_us"],
            d["planner_us"] / d["best_us"], d["paper_rule"], d["paper_rule_us"],
            d["paper_rule_us"] / d["best_us"]))
    r = [d["planner_us"] / d["best_us"] for d in results]
    lines += ["", "Planner / best: %.3f on average, %.3f at worst over %d workloads." % (
        sum(r) / len(r), max(r), len(r))]
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")


def write_heldout_report(results, path, seed):
    lines = ["# The multi-channel planner on seeded random layer shapes", "", "Command:", "",
             "```", _command_line(), "```", "",
             "Layer shapes drawn from a seeded generator (seed %d; C, M in 32..512, outputs "
             "7..112 square, K in {1, 3, 5, 7}); every matrix-core candidate plan timed over "
             "back-to-back launches, and the planner's choice.  %s" % (
                 seed, "The planner's time model was not fitted on these shapes." if seed == 7
                 else "The planner's time model was fitted on the 24 first shapes of this seed."
                 if seed in (20221230, 11) else ""), "",
             "| C | M | map | K | candidates | best plan | best us | planner plan | planner us | "
             "planner / best |", "|---|---|---|---|---|---|---|---|---|---|"]
    for d in results:
        s = d["shape"]
        lines.append("| %d | %d | %dx%d | %d | %d | `%s` | %.2f | `%s` | %.2f | %.3f |" % (
            s["C"], s["M"], s["Wx"], s["Wy"], s["K"], d["candidates"], d["best"], d["best_us"],
            d["planner"], d["planner_us"], d["planner_over_best"]))
    r = [d["planner_over_best"] for d in results]
    lines += ["", "Planner / best: %.3f on average, %.3f at worst over %d shapes." % (
        sum(r) / len(r), max(r), len(r))]
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
