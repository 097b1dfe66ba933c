"""Plant plausible mistakes in copies of the C oracle and check the pins catch
each one (CPU only; the planted mistakes never leave a temporary directory).

A pin set that a dropped term, a wrong sign, a transposed or flipped filter
index, a wrong filter ordering or reduced-precision accumulation could slip
past would not pin anything, so each mutant below must fail at least one pin.
"""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "dconv_oracle.c")

# (name, original text, replacement); every replacement keeps all reads in bounds
MUTANTS = [
    ("transposed_filter", "F[((m * C + ch) * K + j) * K + i]", "F[((m * C + ch) * K + i) * K + j]"),
    ("flipped_filter", "F[((m * C + ch) * K + j) * K + i]",
     "F[((m * C + ch) * K + (K - 1 - j)) * K + (K - 1 - i)]"),
    ("channel_major_filters", "F[((m * C + ch) * K + j) * K + i]", "F[((ch * M + m) * K + j) * K + i]"),
    ("dropped_last_channel", "for (int64_t ch = 0; ch < C; ++ch)", "for (int64_t ch = 0; ch + 1 < C || (C == 1 && ch < 1); ++ch)"),
    ("dropped_last_tap", "for (int64_t i = 0; i < K; ++i)", "for (int64_t i = 0; i < K - (K > 1); ++i)"),
    ("dropped_last_row", "for (int64_t j = 0; j < K; ++j)", "for (int64_t j = 0; j < K - (K > 1); ++j)"),
    ("sign_of_second_channel", "acc += p;", "acc += (ch == 1) ? -p : p;"),
    ("abs_sum_not_abs", "absacc += fabs(p);", "absacc += p;"),
    ("float_accumulator", "double acc = 0.0;", "float acc = 0.0f;"),
    ("input_row_offset_doubled", "I[(ch * Wy + (y + j)) * Wx + (x + i)]",
     "I[(ch * Wy + (y + j / 2)) * Wx + (x + i)]"),
    ("output_rows_swapped", "O[(m * Hout + y) * Wout + x] = acc;",
     "O[(m * Hout + (Hout - 1 - y)) * Wout + x] = acc;"),
]


def _build_mutant(tmp_path, name, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, "mutation site for %s not unique" % name
    src = tmp_path / ("%s.c" % name)
    src.write_text(text.replace(old, new))
    lib = tmp_path / ("lib%s.so" % name)
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-shared", "-fPIC",
                    "-o", str(lib), str(src), "-lm"], check=True)
    dll = ctypes.CDLL(str(lib))
    dll.oracle_conv_f64.restype = ctypes.c_int
    dll.oracle_conv_f64.argtypes = [ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int] * 5 + \
        [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]

    def conv(I, F):
        I = np.ascontiguousarray(I, dtype=np.float32)
        F = np.ascontiguousarray(F, dtype=np.float32)
        C, Wy, Wx = I.shape
        M, _, K, _ = F.shape
        O = np.empty((M, Wy - K + 1, Wx - K + 1))
        A = np.empty_like(O)
        rc = dll.oracle_conv_f64(I.ctypes.data, F.ctypes.data, C, M, Wx, Wy, K,
                                 O.ctypes.data, A.ctypes.data, 1)
        assert rc == 0
        return O, A
    return conv


def test_unmutated_copy_passes(tmp_path):
    conv = _build_mutant(tmp_path, "identity", "double acc = 0.0;", "double acc = 0.0;")
    assert pins.run_all(conv, brute_max_w=4) == []


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    conv = _build_mutant(tmp_path, name, old, new)
    failed = pins.run_all(conv, brute_max_w=4)
    assert failed, "mutant %s passed every pin" % name
