"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU, no
GPU): the fp64 oracle (gcc), and the library's host side -- argument
validation, the planners, the candidate lists and the partition model --
built with the sanitizers on the host pass only (device code as usual) and
driven from the plain C caller tests/c_abi_check.c, which never launches a
kernel.  The instrumented library is built once per source state under
_build/san/ (about a minute and a half when it is not there)."""
import concurrent.futures
import glob
import hashlib
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "_build", "san")
CSRC = os.path.join(ROOT, "paper_2212_00404_amd", "csrc")
INC = os.path.join(ROOT, "include")
CLANG = "/opt/rocm/llvm/bin/clang"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "oracle", "dconv_oracle.c"),
                    os.path.join(ROOT, "tests", "oracle_san_check.c"), "-lm", "-o", exe],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=ENV)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout[-2000:] + r.stderr[-4000:]


def _sources_digest():
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(CSRC, "*"))) + [os.path.join(INC, "dconv.h")]:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def _build_host_sanitized():
    lib = os.path.join(SAN, "libdconv.so")
    stamp = os.path.join(SAN, "digest")
    digest = _sources_digest()
    if os.path.exists(lib) and os.path.exists(stamp) and open(stamp).read() == digest:
        return lib
    os.makedirs(SAN, exist_ok=True)
    # the sanitizers on the host pass only: each -fsanitize= right after
    # -Xarch_host, and none on the device code
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-fvisibility=hidden",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-fno-gpu-sanitize", "-fno-omit-frame-pointer",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I" + INC, "-I" + CSRC]
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))

    def cc(src):
        obj = os.path.join(SAN, os.path.basename(src) + ".o")
        subprocess.run(["/opt/rocm/bin/hipcc"] + flags + ["-c", src, "-o", obj], check=True,
                       capture_output=True, text=True)
        return obj
    with concurrent.futures.ThreadPoolExecutor(min(len(srcs), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(cc, srcs))
    subprocess.run(["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-shared", "-fPIC",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-o", lib] + objs, check=True, capture_output=True, text=True)
    with open(stamp, "w") as fh:
        fh.write(digest)
    return lib


@pytest.mark.skipif(not (os.path.exists(CLANG) and os.path.exists("/opt/rocm/bin/hipcc")),
                    reason="needs the ROCm compilers")
def test_host_library_under_sanitizers(tmp_path):
    lib = _build_host_sanitized()
    exe = str(tmp_path / "c_abi_check_san")
    subprocess.run([CLANG, "-std=c99", "-O1", "-g", "-fsanitize=address,undefined",
                    "-fno-omit-frame-pointer", "-I" + INC,
                    os.path.join(ROOT, "tests", "c_abi_check.c"), "-L" + SAN, "-ldconv",
                    "-Wl,-rpath," + SAN, "-o", exe], check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=ENV)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout[-2000:] + r.stderr[-4000:]
