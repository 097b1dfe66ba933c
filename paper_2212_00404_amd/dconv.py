"""Python binding of libdconv (argument marshalling only).

Every computation runs in the HIP kernels of ``libdconv.so`` through its C
ABI (``include/dconv.h``); this module only checks tensor properties, builds
the output tensor and passes device pointers and the current torch stream.
There is no fallback: if the library is missing or was not built for this
machine, the calls raise.

Paper: Chang, Onishi, Maruyama, "Fast convolution kernels on Pascal GPU with
high memory efficiency", Section 2.1 (Eq. 1 multi-channel, Eq. 2 single map).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdconv.so")

OK = 0
ENULL = -1
EINVAL = -2
ERANGE = -3
EHIP = -4
EUNSUPPORTED = -5

VARIANT_AUTO = 0
VARIANT_VALU = 1
VARIANT_MFMA = 2
_VARIANTS = {"auto": VARIANT_AUTO, "valu": VARIANT_VALU, "mfma": VARIANT_MFMA}

EXPORTED = ("dconv_single", "dconv_single_variant", "dconv_multi", "dconv_multi_variant",
            "dconv_strerror", "dconv_plan_single", "dconv_plan_single_variant",
            "dconv_plan_single_candidates", "dconv_single_with_plan", "dconv_plan_multi",
            "dconv_plan_multi_candidates", "dconv_multi_with_plan", "dconv_model_latency",
            "dconv_model_single", "dconv_model_multi", "dconv_plan_multi_paper",
            "dconv_plan_single_paper", "dconv_probe_latency")


class Plan(ctypes.Structure):
    """Mirror of ``dconv_plan`` in ``include/dconv.h``."""
    _fields_ = [(n, ctypes.c_int) for n in (
        "variant", "kernel", "tile_m", "tile_h", "tile_w", "chunk_c", "waves_c",
        "grid_x", "grid_y", "grid_z", "block", "lds_bytes")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class DeviceParams(ctypes.Structure):
    """Mirror of ``dconv_device_params``."""
    _fields_ = [("latency_clk", ctypes.c_double), ("bandwidth_gbs", ctypes.c_double),
                ("clock_mhz", ctypes.c_double)] + [(n, ctypes.c_int) for n in (
                    "num_cu", "lanes_per_cu", "ops_per_clk_lane", "wave_size", "word_bytes",
                    "onchip_bytes")]


class LatencyModel(ctypes.Structure):
    """Mirror of ``dconv_latency_model``."""
    _fields_ = [("n_fma", ctypes.c_longlong), ("bytes_per_clk", ctypes.c_int),
                ("data_bytes", ctypes.c_longlong), ("threads_total", ctypes.c_longlong),
                ("threads_per_cu", ctypes.c_int),
                ("waves_per_cu", ctypes.c_int), ("bytes_per_cu", ctypes.c_int),
                ("v_s", ctypes.c_longlong)]


class SingleSplit(ctypes.Structure):
    """Mirror of ``dconv_single_split``."""
    _fields_ = [(n, ctypes.c_int) for n in ("method", "P", "Q")] + [
        (n, ctypes.c_longlong) for n in ("D1", "D2", "Th1", "Th2", "p_lo", "p_hi", "q_lo",
                                         "q_hi")] + [
        ("p_admissible", ctypes.c_int), ("q_admissible", ctypes.c_int)]


class MultiBlock(ctypes.Structure):
    """Mirror of ``dconv_multi_block``."""
    _fields_ = [(n, ctypes.c_int) for n in ("S", "Wx_p", "Wy_p", "M_p")] + [
        ("set_bytes", ctypes.c_longlong), ("fma_per_set", ctypes.c_longlong), ("fits", ctypes.c_int)]


def _as_dict(st):
    return {n: getattr(st, n) for n, _ in st._fields_}


# Device descriptions for the partition model.  GTX_1080TI is the paper's
# Table 1 (latency 258 clocks from its pointer-chasing reference, 484 GB/s,
# 1480 MHz base clock, 28 SMs x 128 cores, 2 per core per clock, warps of 32,
# 4-byte words, 96 KB shared memory per SM).  MI355X: 8 TB/s, 2.4 GHz, 256
# CUs x 64 fp32 FMA lanes per clock, 2 flops per FMA, wavefronts of 64,
# 160 KB LDS, and a latency of 900 clocks: what probe_latency measured for a
# dependent-load chain whose footprint (256 MiB to 4 GiB, random hops) is
# beyond the caches (about 375 ns; ~350 clocks when the chain fits in the
# 4 MiB L2, ~130 in the 32 KiB vector L1).
GTX_1080TI = dict(latency_clk=258.0, bandwidth_gbs=484.0, clock_mhz=1480.0, num_cu=28,
                  lanes_per_cu=128, ops_per_clk_lane=2, wave_size=32, word_bytes=4,
                  onchip_bytes=96 * 1024)
MI355X = dict(latency_clk=900.0, bandwidth_gbs=8000.0, clock_mhz=2400.0, num_cu=256,
              lanes_per_cu=64, ops_per_clk_lane=2, wave_size=64, word_bytes=4,
              onchip_bytes=160 * 1024)


def _device(dev: dict) -> DeviceParams:
    missing = [k for k, v in dev.items() if v is None]
    if missing:
        raise ValueError("device parameters not set: %s" % missing)
    return DeviceParams(**dev)


_lib = None


def load(path: str | None = None):
    """Load libdconv.so (built by ``paper_2212_00404_amd/build.py``)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError("libdconv.so is not built (%s); run "
                           "`python paper_2212_00404_amd/build.py` first" % p)
    lib = ctypes.CDLL(p)
    vp, i = ctypes.c_void_p, ctypes.c_int
    lib.dconv_single.argtypes = [vp, vp, vp, i, i, i, i, vp]
    lib.dconv_single.restype = i
    lib.dconv_single_variant.argtypes = [vp, vp, vp, i, i, i, i, i, vp]
    lib.dconv_single_variant.restype = i
    lib.dconv_plan_single_variant.argtypes = [i, i, i, i, i, i, ctypes.POINTER(Plan)]
    lib.dconv_plan_single_variant.restype = i
    lib.dconv_plan_single_candidates.argtypes = [i, i, i, i, i, i, ctypes.POINTER(Plan), i,
                                                 ctypes.POINTER(i)]
    lib.dconv_plan_single_candidates.restype = i
    lib.dconv_single_with_plan.argtypes = [vp, vp, vp, i, i, i, i, ctypes.POINTER(Plan), vp]
    lib.dconv_single_with_plan.restype = i
    lib.dconv_multi.argtypes = [vp, vp, vp, i, i, i, i, i, vp]
    lib.dconv_multi.restype = i
    lib.dconv_multi_variant.argtypes = [vp, vp, vp, i, i, i, i, i, i, vp]
    lib.dconv_multi_variant.restype = i
    lib.dconv_strerror.argtypes = [i]
    lib.dconv_strerror.restype = ctypes.c_char_p
    lib.dconv_plan_single.argtypes = [i, i, i, i, i, ctypes.POINTER(Plan)]
    lib.dconv_plan_single.restype = i
    lib.dconv_plan_multi.argtypes = [i, i, i, i, i, i, i, ctypes.POINTER(Plan)]
    lib.dconv_plan_multi.restype = i
    lib.dconv_plan_multi_candidates.argtypes = [i, i, i, i, i, i, i, ctypes.POINTER(Plan), i,
                                                ctypes.POINTER(i)]
    lib.dconv_plan_multi_candidates.restype = i
    lib.dconv_multi_with_plan.argtypes = [vp, vp, vp, i, i, i, i, i, ctypes.POINTER(Plan), vp]
    lib.dconv_multi_with_plan.restype = i
    dp, lm = ctypes.POINTER(DeviceParams), ctypes.POINTER(LatencyModel)
    lib.dconv_model_latency.argtypes = [dp, lm]
    lib.dconv_model_latency.restype = i
    lib.dconv_model_single.argtypes = [dp, lm, i, i, i, i, ctypes.POINTER(SingleSplit)]
    lib.dconv_model_single.restype = i
    lib.dconv_model_multi.argtypes = [dp, lm, i, i, i, ctypes.POINTER(MultiBlock)]
    lib.dconv_model_multi.restype = i
    lib.dconv_plan_multi_paper.argtypes = [i, i, i, i, i, dp, ctypes.POINTER(Plan)]
    lib.dconv_plan_multi_paper.restype = i
    lib.dconv_plan_single_paper.argtypes = [i, i, i, i, dp, ctypes.POINTER(Plan)]
    lib.dconv_plan_single_paper.restype = i
    lib.dconv_probe_latency.argtypes = [vp, i, vp, vp]
    lib.dconv_probe_latency.restype = i
    if path is None:
        _lib = lib
    return lib


def strerror(status: int) -> str:
    return load().dconv_strerror(int(status)).decode()


def _check(rc: int):
    if rc != OK:
        raise RuntimeError("libdconv: %s (status %d)" % (strerror(rc), rc))


def _require(t: torch.Tensor, name: str, ndim: int):
    if not isinstance(t, torch.Tensor):
        raise ValueError("%s must be a torch.Tensor" % name)
    if t.dtype != torch.float32:
        raise ValueError("%s must be float32, got %s" % (name, t.dtype))
    if t.device.type != "cuda":
        raise ValueError("%s must be on a HIP device, got %s" % (name, t.device))
    if t.dim() != ndim:
        raise ValueError("%s must have %d dimensions, got %d" % (name, ndim, t.dim()))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


class _OnDevice:
    """Make ``device`` current for the C call (the library launches on the
    current HIP device); a no-op when it already is."""

    def __init__(self, device):
        self.index = device.index if device.index is not None else torch.cuda.current_device()
        self.prev = None

    def __enter__(self):
        cur = torch.cuda.current_device()
        if cur != self.index:
            self.prev = cur
            torch.cuda.set_device(self.index)

    def __exit__(self, *exc):
        if self.prev is not None:
            torch.cuda.set_device(self.prev)


def single(I: torch.Tensor, F: torch.Tensor, out: torch.Tensor | None = None,
           variant: str = "auto", plan: dict | None = None) -> torch.Tensor:
    """Eq. 2: ``I[Wy, Wx]``, ``F[M, K, K]`` -> ``O[M, Wy-K+1, Wx-K+1]`` (fp32).

    ``variant`` forces the kernel family: ``"auto"``, ``"valu"`` or ``"mfma"``.
    ``plan``: one of ``plan_single_candidates(...)`` for these sizes
    (overrides ``variant``).
    """
    _require(I, "I", 2)
    _require(F, "F", 3)
    Wy, Wx = I.shape
    M, K, K2 = F.shape
    if K != K2:
        raise ValueError("filters must be square, got %r" % (tuple(F.shape),))
    if F.device != I.device:
        raise ValueError("I and F must be on the same device")
    if not (1 <= K <= min(Wx, Wy)):
        raise ValueError("need 1 <= K <= min(Wx, Wy)")
    if variant not in _VARIANTS:
        raise ValueError("variant must be one of %s" % sorted(_VARIANTS))
    shape = (M, Wy - K + 1, Wx - K + 1)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=I.device)
    else:
        _require(out, "out", 3)
        if tuple(out.shape) != shape or out.device != I.device:
            raise ValueError("out must be %r on %s" % (shape, I.device))
    with _OnDevice(I.device):
        if plan is not None:
            rc = load().dconv_single_with_plan(I.data_ptr(), F.data_ptr(), out.data_ptr(), Wx, Wy,
                                               K, M, ctypes.byref(Plan(**plan)), _stream(I.device))
        else:
            rc = load().dconv_single_variant(I.data_ptr(), F.data_ptr(), out.data_ptr(), Wx, Wy,
                                             K, M, _VARIANTS[variant], _stream(I.device))
    _check(rc)
    return out


def multi(I: torch.Tensor, F: torch.Tensor, out: torch.Tensor | None = None,
          variant: str = "auto", plan: dict | None = None) -> torch.Tensor:
    """Eq. 1: ``I[C, Wy, Wx]``, ``F[M, C, K, K]`` -> ``O[M, Wy-K+1, Wx-K+1]`` (fp32).

    ``variant`` forces the kernel family: ``"auto"``, ``"valu"`` or ``"mfma"``.
    ``plan``: one of ``plan_multi_candidates(...)`` for these sizes (overrides
    ``variant``).
    """
    _require(I, "I", 3)
    _require(F, "F", 4)
    C, Wy, Wx = I.shape
    M, C2, K, K2 = F.shape
    if C2 != C or K != K2:
        raise ValueError("filter shape %r does not match input %r" % (tuple(F.shape), tuple(I.shape)))
    if F.device != I.device:
        raise ValueError("I and F must be on the same device")
    if not (1 <= K <= min(Wx, Wy)):
        raise ValueError("need 1 <= K <= min(Wx, Wy)")
    if variant not in _VARIANTS:
        raise ValueError("variant must be one of %s" % sorted(_VARIANTS))
    shape = (M, Wy - K + 1, Wx - K + 1)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=I.device)
    else:
        _require(out, "out", 3)
        if tuple(out.shape) != shape or out.device != I.device:
            raise ValueError("out must be %r on %s" % (shape, I.device))
    with _OnDevice(I.device):
        if plan is not None:
            rc = load().dconv_multi_with_plan(I.data_ptr(), F.data_ptr(), out.data_ptr(), C, M,
                                              Wx, Wy, K, ctypes.byref(Plan(**plan)),
                                              _stream(I.device))
        else:
            rc = load().dconv_multi_variant(I.data_ptr(), F.data_ptr(), out.data_ptr(), C, M, Wx,
                                            Wy, K, _VARIANTS[variant], _stream(I.device))
    _check(rc)
    return out


def plan_single(Wx: int, Wy: int, K: int, M: int, num_cu: int = 256,
                variant: str = "auto") -> dict:
    """The launch plan ``dconv_single_variant`` would use (host logic, no device)."""
    p = Plan()
    _check(load().dconv_plan_single_variant(Wx, Wy, K, M, _VARIANTS[variant], num_cu,
                                            ctypes.byref(p)))
    return p.as_dict()


def plan_single_candidates(Wx: int, Wy: int, K: int, M: int, variant: str = "auto",
                           num_cu: int = 256) -> list:
    """Every plan ``dconv_single_with_plan`` accepts for these sizes (a
    16-byte-aligned input with Wx % 4 == 0; host logic)."""
    n = ctypes.c_int(0)
    lib = load()
    _check(lib.dconv_plan_single_candidates(Wx, Wy, K, M, _VARIANTS[variant], num_cu, None, 0,
                                            ctypes.byref(n)))
    arr = (Plan * max(n.value, 1))()
    _check(lib.dconv_plan_single_candidates(Wx, Wy, K, M, _VARIANTS[variant], num_cu, arr,
                                            n.value, ctypes.byref(n)))
    return [arr[k].as_dict() for k in range(n.value)]


def plan_single_paper(Wx: int, Wy: int, K: int, M: int, dev: dict) -> dict:
    """The single-map candidate the Section 3.1 division picks for a device."""
    p = Plan()
    _check(load().dconv_plan_single_paper(Wx, Wy, K, M, ctypes.byref(_device(dev)),
                                          ctypes.byref(p)))
    return p.as_dict()


def plan_multi(C: int, M: int, Wx: int, Wy: int, K: int, variant: str = "auto",
               num_cu: int = 256) -> dict:
    """The launch plan ``dconv_multi_variant`` would use (host logic, no device)."""
    p = Plan()
    _check(load().dconv_plan_multi(C, M, Wx, Wy, K, _VARIANTS[variant], num_cu, ctypes.byref(p)))
    return p.as_dict()


def plan_multi_candidates(C: int, M: int, Wx: int, Wy: int, K: int, variant: str = "auto",
                          num_cu: int = 256) -> list:
    """Every plan ``dconv_multi_with_plan`` accepts for these sizes (host logic)."""
    n = ctypes.c_int(0)
    lib = load()
    _check(lib.dconv_plan_multi_candidates(C, M, Wx, Wy, K, _VARIANTS[variant], num_cu, None, 0,
                                           ctypes.byref(n)))
    arr = (Plan * max(n.value, 1))()
    _check(lib.dconv_plan_multi_candidates(C, M, Wx, Wy, K, _VARIANTS[variant], num_cu, arr,
                                           n.value, ctypes.byref(n)))
    return [arr[k].as_dict() for k in range(n.value)]


def model_latency(dev: dict) -> dict:
    """Section 2.2 / Table 1 figures (N_FMA, V_s, ...) for a device description."""
    out = LatencyModel()
    _check(load().dconv_model_latency(ctypes.byref(_device(dev)), ctypes.byref(out)))
    return _as_dict(out)


def model_single(dev: dict, Wx: int, Wy: int, K: int, M: int) -> dict:
    """Section 3.1 division (method, P, Q, D1, D2, Th1, Th2) for a single-channel layer."""
    d, lm, out = _device(dev), LatencyModel(), SingleSplit()
    lib = load()
    _check(lib.dconv_model_latency(ctypes.byref(d), ctypes.byref(lm)))
    _check(lib.dconv_model_single(ctypes.byref(d), ctypes.byref(lm), Wx, Wy, K, M,
                                  ctypes.byref(out)))
    return _as_dict(out)


def model_multi(dev: dict, K: int, S: int, Wxp: int) -> dict:
    """Section 3.2 stride-fixed block (W'y, M', data-set bytes) for segment S, W'x."""
    d, lm, out = _device(dev), LatencyModel(), MultiBlock()
    lib = load()
    _check(lib.dconv_model_latency(ctypes.byref(d), ctypes.byref(lm)))
    _check(lib.dconv_model_multi(ctypes.byref(d), ctypes.byref(lm), K, S, Wxp, ctypes.byref(out)))
    return _as_dict(out)


def plan_multi_paper(C: int, M: int, Wx: int, Wy: int, K: int, dev: dict) -> dict:
    """The candidate the Section 3.2 rules pick for a device description."""
    p = Plan()
    _check(load().dconv_plan_multi_paper(C, M, Wx, Wy, K, ctypes.byref(_device(dev)),
                                         ctypes.byref(p)))
    return p.as_dict()


def probe_latency(footprint_bytes: int, steps: int = 20000, stride_bytes: int = 256,
                  seed: int = 0, device=None) -> dict:
    """Dependent-load latency over a random cyclic chain of ``footprint_bytes``
    (one hop per ``stride_bytes``), measured by dconv_probe_latency.  Returns
    shader-clock cycles and nanoseconds per load."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else device
    slot = stride_bytes // 4
    n = footprint_bytes // stride_bytes
    if n < 2 or slot < 1:
        raise ValueError("footprint must hold at least two strides")
    g = torch.Generator().manual_seed(seed)
    order = torch.randperm(n, generator=g)
    nxt = torch.empty(n, dtype=torch.int64)
    nxt[order] = torch.roll(order, -1)
    chain = torch.zeros(n * slot, dtype=torch.int32)
    chain[torch.arange(n) * slot] = (nxt * slot).to(torch.int32)
    # start the walk at index 0, which is slot 0 of the cycle
    chain_d = chain.to(dev)
    out = torch.zeros(3, dtype=torch.int64, device=dev)
    with _OnDevice(dev):
        _check(load().dconv_probe_latency(chain_d.data_ptr(), steps, out.data_ptr(),
                                          _stream(dev)))
    torch.cuda.synchronize(dev)
    cyc, ticks, _ = out.tolist()
    return {"footprint_bytes": footprint_bytes, "steps": steps, "stride_bytes": stride_bytes,
            "cycles_per_load": cyc / steps, "ns_per_load": ticks * 10.0 / steps}
