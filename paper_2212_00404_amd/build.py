"""Build ``libdconv.so`` (the HIP kernels and the C ABI) for gfx950.

Each ``csrc/*.hip`` file is compiled with hipcc in parallel into ``_build/``
and linked into ``paper_2212_00404_amd/libdconv.so``.  Only the ``dconv_*``
entry points are exported (``-fvisibility=hidden`` plus explicit default
visibility on the API).

Packed fp32 VALU instructions are disabled for the device code
(``-target-feature -packed-fp32-ops``); the host pass warns that it does not
know that feature, which is harmless.
"""
import concurrent.futures
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libdconv.so")
# Debug build with every kernel's LDS filled with NaN before first use
# (-DDCONV_POISON_LDS): a GPU test runs it to catch reads of LDS that a
# kernel did not write first.
POISON_LIB = os.path.join(PKG, "libdconv_poison.so")
# Debug build whose multi-channel matrix-core kernel records clock counters
# around the phases of its stage loop (-DDCONV_STAGE_TRACE; bench.py
# --stage-trace reads them).
TRACE_LIB = os.path.join(PKG, "libdconv_trace.so")
PEAKS_SRC = os.path.join(PKG, "peaks", "peaks.hip")
PEAKS_LIB = os.path.join(PKG, "libdconv_peaks.so")
ARCH = "gfx950"

CFLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # fully unroll the long compile-time loops of the matrix-core single-map
    # kernel (its register arrays are indexed by the loop counters)
    "-mllvm", "-pragma-unroll-threshold=1000000",
    "-I" + INCLUDE, "-I" + CSRC,
]


def _code_only(text: str) -> str:
    """C/C++ source without its comments, trailing blanks and empty lines."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return "\n".join(l.rstrip() for l in "".join(out).splitlines() if l.strip())


def source_digest(names=None) -> str:
    """SHA-256 over the code of the kernel sources, comments excluded
    (identifies what is compiled).  ``names``: file names under ``csrc/`` to
    cover (default: every source and the ABI header)."""
    import hashlib
    h = hashlib.sha256()
    if names is None:
        files = sorted(glob.glob(os.path.join(CSRC, "*"))) + [os.path.join(INCLUDE, "dconv.h")]
    else:
        files = [os.path.join(CSRC, n) for n in names]
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


def _compile(src, out_dir=BUILD, extra=()):
    obj = os.path.join(out_dir, os.path.basename(src).replace(".hip", ".o"))
    cmd = [_hipcc()] + CFLAGS + list(extra) + ["-c", src, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s" % (src, err))
    return obj, err


def _link(objs, lib):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("link failed:\n" + res.stderr)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compile every source and link the library, its LDS-poisoning and
    stage-trace debug twins (libdconv_poison.so, libdconv_trace.so) and the
    peak microbenchmarks (libdconv_peaks.so, from peaks/); returns the
    library's path."""
    poison_dir = os.path.join(BUILD, "poison")
    trace_dir = os.path.join(BUILD, "trace")
    os.makedirs(poison_dir, exist_ok=True)
    os.makedirs(trace_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    jobs = ([(s, BUILD, ()) for s in srcs] + [(PEAKS_SRC, BUILD, ())] +
            [(s, poison_dir, ("-DDCONV_POISON_LDS",)) for s in srcs] +
            [(s, trace_dir, ("-DDCONV_STAGE_TRACE",)) for s in srcs])
    workers = min(len(jobs), max(1, min(8, os.cpu_count() or 1)))
    # the matrix-core kernel units take longest: start them first
    order = sorted(range(len(jobs)), key=lambda i: "multi_mfma" not in jobs[i][0])
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        futs = {i: ex.submit(_compile, *jobs[i]) for i in order}
        results = [futs[i].result() for i in range(len(jobs))]
    if verbose:
        for obj, err in results:
            if err.strip():
                print(err, file=sys.stderr)
    objs = [o for o, _ in results]
    n = len(srcs)
    _link(objs[:n], LIB)
    _link(objs[n:n + 1], PEAKS_LIB)
    _link(objs[n + 1:2 * n + 1], POISON_LIB)
    _link(objs[2 * n + 1:], TRACE_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
