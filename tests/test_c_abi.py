"""libdconv from a plain C99 program (no GPU): the public header compiles as
C with warnings as errors, the library links and its host-side checks,
planners and latency model answer as documented (tests/c_abi_check.c)."""
import os
import shutil
import subprocess

import pytest

import paper_2212_00404_amd as dc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi_check.c")
INC = os.path.join(ROOT, "include")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs a C compiler")
def test_c_caller(tmp_path):
    lib = dc.load()._name
    libdir = os.path.dirname(os.path.abspath(lib))
    exe = str(tmp_path / "c_abi_check")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I" + INC,
                    SRC, "-L" + libdir, "-ldconv", "-Wl,-rpath," + libdir, "-o", exe],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "ok"
