"""CPU oracle for direct valid-mode stride-1 2-D convolution.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, fp64 definition of
what the GPU library computes.  Only ``tests/``, the smoke check in
``__graft_entry__.py`` and the CPU-baseline leg of ``bench.py`` may import it.
It imports nothing from the GPU library, and the GPU library imports nothing
from it.

Definition followed (paper, Section 2.1, Eq. 1 for C input maps; Eq. 2 is the
single-map case C = 1): for every filter m and every valid output position,
the output is the sum over channels ch and filter offsets (i along x, j along
y) of input(x+i, y+j) times filter(i, j).  The storage conventions chosen where
the paper is silent are documented in ``dconv_oracle.c``: maps are
``[C][Wy][Wx]`` with x fastest, filters ``[M][C][K][K]`` with the row index
paired with the y offset, outputs ``[M][Wy-K+1][Wx-K+1]``; no flip.

Each function returns the fp64 value and ``A = sum |I * F|`` per output.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is None:
        path = _build.build(force=False)
        lib = ctypes.CDLL(path)
        lib.oracle_conv_f64.restype = ctypes.c_int
        lib.oracle_conv_f64.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
            ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_int]
        lib.oracle_max_threads.restype = ctypes.c_int
        lib.oracle_max_threads.argtypes = []
        _lib = lib
    return _lib


def max_threads() -> int:
    """Threads the OpenMP runtime of the oracle would use by default."""
    return int(_load().oracle_max_threads())


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def conv_multi(I, F, threads: int | None = None):
    """Eq. 1: ``I`` float32 ``[C, Wy, Wx]``, ``F`` float32 ``[M, C, K, K]``.

    Returns ``(O64, A64)``, both float64 ``[M, Wy-K+1, Wx-K+1]``.
    """
    I = np.ascontiguousarray(I, dtype=np.float32)
    F = np.ascontiguousarray(F, dtype=np.float32)
    if I.ndim != 3 or F.ndim != 4:
        raise ValueError("expected I[C,Wy,Wx] and F[M,C,K,K]")
    C, Wy, Wx = I.shape
    M, C2, K, K2 = F.shape
    if C2 != C or K2 != K:
        raise ValueError("filter shape %r does not match input %r" % (F.shape, I.shape))
    if not (1 <= K <= min(Wx, Wy)):
        raise ValueError("need 1 <= K <= min(Wx, Wy)")
    Hout, Wout = Wy - K + 1, Wx - K + 1
    O = np.empty((M, Hout, Wout), dtype=np.float64)
    A = np.empty((M, Hout, Wout), dtype=np.float64)
    if threads is None:
        threads = default_threads()
    rc = _load().oracle_conv_f64(I.ctypes.data, F.ctypes.data, C, M, Wx, Wy, K,
                                 O.ctypes.data, A.ctypes.data, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the sizes (rc=%d)" % rc)
    return O, A


def conv_single(I, F, threads: int | None = None):
    """Eq. 2: ``I`` float32 ``[Wy, Wx]``, ``F`` float32 ``[M, K, K]``.

    Returns ``(O64, A64)``, both float64 ``[M, Wy-K+1, Wx-K+1]``.
    """
    I = np.asarray(I, dtype=np.float32)
    F = np.asarray(F, dtype=np.float32)
    if I.ndim != 2 or F.ndim != 3:
        raise ValueError("expected I[Wy,Wx] and F[M,K,K]")
    return conv_multi(I[None], F[:, None], threads=threads)
