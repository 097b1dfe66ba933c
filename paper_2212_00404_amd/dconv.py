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
ENOMEM = -6

VARIANT_AUTO = 0
VARIANT_VALU = 1
VARIANT_MFMA = 2
_VARIANTS = {"auto": VARIANT_AUTO, "valu": VARIANT_VALU, "mfma": VARIANT_MFMA}

EXPORTED = ("dconv_single", "dconv_multi", "dconv_multi_variant", "dconv_strerror",
            "dconv_plan_single", "dconv_plan_multi")


class Plan(ctypes.Structure):
    """Mirror of ``dconv_plan`` in ``include/dconv.h``."""
    _fields_ = [(n, ctypes.c_int) for n in (
        "variant", "kernel", "tile_m", "tile_h", "tile_w", "chunk_c", "split_c",
        "grid_x", "grid_y", "grid_z", "block", "lds_bytes")] + [("workspace_bytes", ctypes.c_longlong)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


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


def single(I: torch.Tensor, F: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """Eq. 2: ``I[Wy, Wx]``, ``F[M, K, K]`` -> ``O[M, Wy-K+1, Wx-K+1]`` (fp32)."""
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
    shape = (M, Wy - K + 1, Wx - K + 1)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=I.device)
    else:
        _require(out, "out", 3)
        if tuple(out.shape) != shape or out.device != I.device:
            raise ValueError("out must be %r on %s" % (shape, I.device))
    with _OnDevice(I.device):
        rc = load().dconv_single(I.data_ptr(), F.data_ptr(), out.data_ptr(), Wx, Wy, K, M,
                                 _stream(I.device))
    _check(rc)
    return out


def multi(I: torch.Tensor, F: torch.Tensor, out: torch.Tensor | None = None,
          variant: str = "auto") -> torch.Tensor:
    """Eq. 1: ``I[C, Wy, Wx]``, ``F[M, C, K, K]`` -> ``O[M, Wy-K+1, Wx-K+1]`` (fp32).

    ``variant`` forces the kernel family: ``"auto"``, ``"valu"`` or ``"mfma"``.
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
        rc = load().dconv_multi_variant(I.data_ptr(), F.data_ptr(), out.data_ptr(), C, M, Wx, Wy,
                                        K, _VARIANTS[variant], _stream(I.device))
    _check(rc)
    return out


def plan_single(Wx: int, Wy: int, K: int, M: int, num_cu: int = 256) -> dict:
    """The launch plan ``dconv_single`` would use (host logic, no device)."""
    p = Plan()
    _check(load().dconv_plan_single(Wx, Wy, K, M, num_cu, ctypes.byref(p)))
    return p.as_dict()


def plan_multi(C: int, M: int, Wx: int, Wy: int, K: int, variant: str = "auto",
               num_cu: int = 256) -> dict:
    """The launch plan ``dconv_multi_variant`` would use (host logic, no device)."""
    p = Plan()
    _check(load().dconv_plan_multi(C, M, Wx, Wy, K, _VARIANTS[variant], num_cu, ctypes.byref(p)))
    return p.as_dict()
