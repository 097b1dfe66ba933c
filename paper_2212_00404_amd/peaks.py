"""Peak-rate microbenchmarks on the current HIP device (libdconv_peaks.so).

Each function launches one kernel of ``peaks/peaks.hip`` a few times on the
current torch stream, times the launches with HIP events and returns the
rate.  These are the measured ceilings the roofline fractions of bench.py
are reported against beside the datasheet peaks: HBM read, write and copy
streams, one fp32 FMA per lane per clock (packed fp32 is disabled in this
build), the two fp32 matrix instructions the convolution kernels use, and
the global-to-LDS copy path their stages go through.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdconv_peaks.so")
_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libdconv_peaks.so is not built; run paper_2212_00404_amd/build.py")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i, ll = ctypes.c_void_p, ctypes.c_int, ctypes.c_longlong
        lib.peaks_hbm_read.argtypes = [vp, ll, vp, i, vp]
        lib.peaks_hbm_write.argtypes = [vp, ll, i, vp]
        lib.peaks_hbm_copy.argtypes = [vp, vp, ll, i, vp]
        lib.peaks_fma.argtypes = [vp, i, i, vp]
        lib.peaks_mfma.argtypes = [vp, i, i, i, vp]
        lib.peaks_lds_dma.argtypes = [vp, ll, i, i, i, vp, i, vp]
        lib.peaks_lds_dma_layout.argtypes = [vp, i, i, vp, vp]
        lib.peaks_vgpr_load.argtypes = [vp, ll, i, vp, i, vp]
        lib.peaks_mfma_chains.argtypes = [vp, i, i, i, vp]
        for f in ("peaks_hbm_read", "peaks_hbm_write", "peaks_hbm_copy", "peaks_fma",
                  "peaks_mfma", "peaks_lds_dma", "peaks_lds_dma_layout", "peaks_vgpr_load",
                  "peaks_mfma_chains"):
            getattr(lib, f).restype = i
        _lib = lib
    return _lib


def _time(launch, reps):
    """Median of `reps` event-timed launches (ms), after one warm-up."""
    s = torch.cuda.current_stream()
    launch(s)
    torch.cuda.synchronize()
    out = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        launch(s)
        b.record(s)
        torch.cuda.synchronize()
        out.append(a.elapsed_time(b))
    out.sort()
    return out[len(out) // 2]


def _rc(rc):
    if rc != 0:
        raise RuntimeError("peaks launch failed (%d)" % rc)


def run(reps: int = 10, hbm_mib: int = 2048) -> dict:
    """Every microbenchmark once; returns a dict of rates."""
    lib = load()
    dev = torch.device("cuda", torch.cuda.current_device())
    cu = torch.cuda.get_device_properties(dev).multi_processor_count
    sp = lambda s: ctypes.c_void_p(s.cuda_stream)
    res = {"compute_units": cu}
    nbytes = hbm_mib << 20
    a = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).uniform_()
    b = torch.empty_like(a)
    grid = cu * 8
    sink = torch.empty(grid * 256, dtype=torch.float32, device=dev)
    ms = _time(lambda s: _rc(lib.peaks_hbm_read(a.data_ptr(), nbytes, sink.data_ptr(), grid, sp(s))), reps)
    res["hbm_read_gbs"] = round(nbytes / ms / 1e6, 1)
    ms = _time(lambda s: _rc(lib.peaks_hbm_write(b.data_ptr(), nbytes, grid, sp(s))), reps)
    res["hbm_write_gbs"] = round(nbytes / ms / 1e6, 1)
    ms = _time(lambda s: _rc(lib.peaks_hbm_copy(a.data_ptr(), b.data_ptr(), nbytes, grid, sp(s))), reps)
    res["hbm_copy_gbs"] = round(2 * nbytes / ms / 1e6, 1)
    res["hbm_bytes"] = nbytes
    del a, b
    # fp32 FMA: grid x 256 lanes x iters x 8 FMAs x 2 flops
    iters = 20000
    grid = cu * 8
    out = torch.empty(grid * 256, dtype=torch.float32, device=dev)
    ms = _time(lambda s: _rc(lib.peaks_fma(out.data_ptr(), iters, grid, sp(s))), reps)
    res["fma_fp32_tflops"] = round(grid * 256 * iters * 8 * 2 / ms / 1e9, 2)
    # fp32 MFMA: grid x 4 waves x iters x 4 instructions x (4096, 2048 or 512)
    # flops
    for shape, fl in ((32, 4096), (16, 2048), (4, 512)):
        it = 4000 * 4096 // fl
        ms = _time(lambda s: _rc(lib.peaks_mfma(out.data_ptr(), it, grid, shape, sp(s))), reps)
        res["mfma_f32_%dx%d_tflops" % (shape, shape)] = round(grid * 4 * it * 4 * fl / ms / 1e9, 2)
    # dependent v_mfma_f32_4x4x1f32: clocks (at 2.4 GHz) per instruction with
    # one wave per SIMD and 1, 2, 4 or 8 independent accumulation chains
    chains = {}
    for na in (1, 2, 4, 8):
        it = 32000 // na
        ms = _time(lambda s: _rc(lib.peaks_mfma_chains(out.data_ptr(), na, it, cu, sp(s))), reps)
        chains[str(na)] = round(ms * 1e-3 * 2.4e9 / (it * na), 1)
    res["mfma_f32_4x4_clk_per_instr_by_chains"] = chains
    # global -> LDS copies from a 2 MiB region (L2-resident): bytes per
    # second in total and per compute unit per clock at 2.4 GHz
    # (16-byte copies also from sources one float off their alignment)
    region = 1 << 19
    src = torch.rand(region + 4, dtype=torch.float32, device=dev)
    g = cu * 2
    o = torch.empty(g * 256, dtype=torch.float32, device=dev)
    for width, shift in ((4, 0), (16, 0), (16, 1)):
        bursts = 400
        ms = _time(lambda s: _rc(lib.peaks_lds_dma(src.data_ptr(), region, shift, width, bursts,
                                                   o.data_ptr(), g, sp(s))), reps)
        total = g * 4 * bursts * 16 * 64 * width
        key = "lds_dma_b%d%s" % (width * 8, "_unaligned" if shift else "")
        res[key + "_gbs"] = round(total / ms / 1e6, 1)
        res[key + "_bytes_per_cu_clk"] = round(total / ms / 1e-3 / cu / 2.4e9, 1)
    # the copy rate per compute unit against the number of waves issuing
    # copies (4 per workgroup; at most 8 fit for 16-byte copies, whose
    # workgroups hold 64 KB of LDS)
    by_waves = {"b32": {}, "b128": {}}
    for width, waves in ((4, 4), (4, 8), (4, 16), (4, 32), (16, 4), (16, 8)):
        gw = cu * waves // 4
        ow = torch.empty(gw * 256, dtype=torch.float32, device=dev)
        ms = _time(lambda s: _rc(lib.peaks_lds_dma(src.data_ptr(), region, 0, width, 200,
                                                   ow.data_ptr(), gw, sp(s))), reps)
        total = gw * 4 * 200 * 16 * 64 * width
        by_waves["b%d" % (width * 8)][str(waves)] = round(total / ms / 1e-3 / cu / 2.4e9, 1)
        del ow
    res["lds_dma_bytes_per_cu_clk_by_waves_per_cu"] = by_waves
    # the same walk into registers (float4 loads)
    bursts = 400
    ms = _time(lambda s: _rc(lib.peaks_vgpr_load(src.data_ptr(), region, bursts, o.data_ptr(),
                                                 g, sp(s))), reps)
    total = g * 4 * bursts * 16 * 64 * 16
    res["l2_vgpr_b128_gbs"] = round(total / ms / 1e6, 1)
    res["l2_vgpr_b128_bytes_per_cu_clk"] = round(total / ms / 1e-3 / cu / 2.4e9, 1)
    return res


def lds_dma_layout(shift: int, active: int = 64):
    """The 264-float LDS array after one wave's 16-byte-per-lane direct copy
    of 256 floats (1, 2, ..., 256) to float offset `shift`, issued by lanes
    0 .. active-1 only (see peaks.hip)."""
    lib = load()
    dev = torch.device("cuda", torch.cuda.current_device())
    src = torch.arange(256, dtype=torch.float32, device=dev) + 1.0
    out = torch.full((264,), -1.0, dtype=torch.float32, device=dev)
    _rc(lib.peaks_lds_dma_layout(src.data_ptr(), shift, active, out.data_ptr(),
                                 ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)))
    torch.cuda.synchronize()
    return out.cpu()
