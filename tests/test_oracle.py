"""The CPU oracle against its pins (no GPU needed).

Every pin compares the oracle with something fixed independently of its code
(see ``oracle_pins.py``).  The paper prints no worked numeric example for the
convolution (its result figures carry no data), so there is no printed value
to pin against; library routines, closed forms and invariants of Eq. 1 take
that role.
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import oracle_pins as pins
from dconv_workloads import WORKLOADS, make, random_arrays


def conv(I, F):
    return oracle.conv_multi(I, F, threads=2)


@pytest.mark.parametrize("name", [
    "torch_conv2d", "scipy_correlate2d", "sliding_window", "delta", "box_sum", "k1_gemm",
    "full_window_dot", "separable", "linearity", "channel_additivity",
    "filter_independence", "translation", "abs_sum"])
def test_pin(name):
    fn = {
        "torch_conv2d": lambda: pins.pin_torch_conv2d(conv, pins.SHAPES),
        "scipy_correlate2d": lambda: pins.pin_scipy_correlate2d(conv, pins.SHAPES_2D),
        "sliding_window": lambda: pins.pin_sliding_window(conv, pins.SHAPES),
        "delta": lambda: pins.pin_delta(conv, pins.SHAPES),
        "box_sum": lambda: pins.pin_box_sum(conv, pins.SHAPES_BOX),
        "k1_gemm": lambda: pins.pin_k1_is_gemm(conv, pins.SHAPES_K1),
        "full_window_dot": lambda: pins.pin_full_window_is_dot(conv, pins.SHAPES_FULL),
        "separable": lambda: pins.pin_separable(conv, pins.SHAPES_2D),
        "linearity": lambda: pins.pin_linearity(conv, pins.SHAPES),
        "channel_additivity": lambda: pins.pin_channel_additivity(conv, pins.SHAPES),
        "filter_independence": lambda: pins.pin_filter_independence(conv, pins.SHAPES),
        "translation": lambda: pins.pin_translation(conv, pins.SHAPES_SHIFT),
        "abs_sum": lambda: pins.pin_abs_sum(conv, pins.SHAPES),
    }[name]
    fn()


def test_brute_force_exhaustive_tiny():
    pins.pin_brute_force(conv, max_w=5)


@settings(max_examples=40, deadline=None)
@given(C=st.integers(1, 4), M=st.integers(1, 4), Wx=st.integers(1, 14), Wy=st.integers(1, 14),
       K=st.integers(1, 7), seed=st.integers(0, 2**31 - 1))
def test_random_shapes_against_torch(C, M, Wx, Wy, K, seed):
    K = min(K, Wx, Wy)
    I, F = random_arrays(C, M, Wx, Wy, K, seed)
    O, A = conv(I, F)
    import torch
    ref = torch.nn.functional.conv2d(torch.from_numpy(I).double()[None],
                                     torch.from_numpy(F).double())[0].numpy()
    pins.close(O, ref, A, "random shape")


def test_integer_data_is_exact():
    """Integer inputs: every partial sum is an integer below 2^53, so the fp64
    oracle equals exact int64 arithmetic."""
    for C, M, W, K in [(3, 2, 9, 3), (8, 4, 12, 5)]:
        I, F = random_arrays(C, M, W, W, K, 77, variant="int")
        O, _ = conv(I, F)
        win = np.lib.stride_tricks.sliding_window_view(I.astype(np.int64), (K, K), axis=(1, 2))
        ref = np.einsum("cyxrs,mcrs->myx", win, F.astype(np.int64))
        assert np.array_equal(O, ref.astype(np.float64))


def test_single_is_multi_with_one_channel():
    """Eq. 2 is Eq. 1 with C = 1."""
    I, F = random_arrays(1, 3, 10, 8, 3, 5)
    O1, A1 = oracle.conv_single(I[0], F[:, 0], threads=1)
    O2, A2 = oracle.conv_multi(I, F, threads=1)
    assert np.array_equal(O1, O2) and np.array_equal(A1, A2)


def test_thread_count_does_not_change_result():
    I, F = random_arrays(4, 5, 17, 13, 3, 6)
    O1, A1 = oracle.conv_multi(I, F, threads=1)
    O2, A2 = oracle.conv_multi(I, F, threads=4)
    assert np.array_equal(O1, O2) and np.array_equal(A1, A2)


def test_rejects_bad_sizes():
    I, F = random_arrays(1, 1, 4, 4, 3, 0)
    with pytest.raises(ValueError):
        oracle.conv_multi(I[:, :2, :], F)           # K > Wy
    with pytest.raises(ValueError):
        oracle.conv_multi(I, F[:, :, :2, :])        # non-square filter


def test_workload_recipes():
    """The seeded generators give the documented shapes and distributions."""
    I, F = make("single_64x64_m1_k3")
    assert I.shape == (64, 64) and F.shape == (1, 3, 3) and I.dtype == np.float32
    assert I.min() >= -1 and I.max() < 1
    I, F = make("multi_c512_9x9_m512_k3")
    assert I.shape == (512, 9, 9) and F.shape == (512, 512, 3, 3)
    assert I.min() >= 0 and I.max() < 1
    assert abs(F.std() - np.sqrt(2.0 / (512 * 9))) < 1e-3 * 5
    Ii, Fi = make("multi_c512_9x9_m512_k3", "int")
    assert set(np.unique(Ii)) <= set(range(-3, 4)) and set(np.unique(Fi)) <= set(range(-3, 4))
    # deterministic
    assert np.array_equal(make("single_64x64_m1_k3")[0], make("single_64x64_m1_k3")[0])
    w = WORKLOADS["single_4096x4096_m1_k11"]
    assert w.flops == 2 * 121 * 4086 * 4086
