"""Independent checks ("pins") for the convolution oracle.

Each pin takes ``conv(I[C,Wy,Wx], F[M,C,K,K]) -> (O64, A64)`` and raises
``AssertionError`` if the result contradicts something fixed independently of
the oracle's own code: a library routine, a closed form, an invariant of
Eq. 1 (paper, Section 2.1) or exhaustive brute force on tiny inputs.  They are
written as plain functions so the same pins can be run against deliberately
broken copies of the oracle (see ``test_oracle_mutants.py``) to show that each
plausible mistake is caught.
"""
import numpy as np
import scipy.signal
import torch

from dconv_workloads import random_arrays

REL = 1e-12   # fp64 sums in a different order: |err| <= n * 2^-53 * sum|terms|


def close(a, b, A, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, "%s: shape %r vs %r" % (what, a.shape, b.shape)
    err = np.abs(a - b)
    bound = REL * np.asarray(A) + 1e-300
    bad = err > bound
    assert not bad.any(), "%s: %d mismatches, worst err %g" % (what, bad.sum(), err.max())


def exact(a, b, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, "%s: shape %r vs %r" % (what, a.shape, b.shape)
    assert np.array_equal(a, b), "%s: max |diff| %g" % (what, np.abs(a - b).max())


# --- library routines --------------------------------------------------------

def pin_torch_conv2d(conv, shapes, seed=1):
    """torch.nn.functional.conv2d in fp64 on the CPU: cross-correlation with
    weight[m][c][r][s] multiplying input[c][y+r][x+s]."""
    for n, (C, M, Wx, Wy, K) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, K, seed + n)
        O, A = conv(I, F)
        ref = torch.nn.functional.conv2d(torch.from_numpy(I).double()[None],
                                         torch.from_numpy(F).double())[0].numpy()
        close(O, ref, A, "torch conv2d %r" % ((C, M, Wx, Wy, K),))


def pin_scipy_correlate2d(conv, shapes, seed=2):
    """scipy.signal.correlate2d(mode='valid') for one map and one filter."""
    for n, (Wx, Wy, K) in enumerate(shapes):
        I, F = random_arrays(1, 1, Wx, Wy, K, seed + n)
        O, A = conv(I, F)
        ref = scipy.signal.correlate2d(I[0].astype(np.float64), F[0, 0].astype(np.float64),
                                       mode="valid")
        close(O[0], ref, A[0], "correlate2d %r" % ((Wx, Wy, K),))


def pin_sliding_window(conv, shapes, seed=3):
    """numpy sliding_window_view + einsum in fp64."""
    for n, (C, M, Wx, Wy, K) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, K, seed + n)
        O, A = conv(I, F)
        win = np.lib.stride_tricks.sliding_window_view(I.astype(np.float64), (K, K), axis=(1, 2))
        ref = np.einsum("cyxrs,mcrs->myx", win, F.astype(np.float64))
        close(O, ref, A, "sliding window %r" % ((C, M, Wx, Wy, K),))


# --- special cases with closed forms ------------------------------------------

def pin_delta(conv, shapes, seed=4):
    """A filter that is 1 at (c0, r0, s0) and 0 elsewhere copies the shifted
    input: O[m][y][x] = I[c0][y + r0][x + s0].  Off-centre (r0 != s0) catches a
    transposed or flipped filter index; exact for any data."""
    rng = np.random.default_rng(seed)
    for n, (C, M, Wx, Wy, K) in enumerate(shapes):
        I, _ = random_arrays(C, M, Wx, Wy, K, seed + n)
        F = np.zeros((M, C, K, K), dtype=np.float32)
        picks = []
        for m in range(M):
            c0 = int(rng.integers(C))
            r0 = int(rng.integers(K))
            s0 = int(rng.integers(K))
            if K > 1 and r0 == s0:
                s0 = (r0 + 1) % K
            F[m, c0, r0, s0] = 1.0
            picks.append((c0, r0, s0))
        O, _ = conv(I, F)
        Hout, Wout = Wy - K + 1, Wx - K + 1
        for m, (c0, r0, s0) in enumerate(picks):
            exact(O[m], I[c0, r0:r0 + Hout, s0:s0 + Wout], "delta %r" % ((C, M, Wx, Wy, K, m),))


def pin_box_sum(conv, shapes, seed=5):
    """An all-ones filter gives the K x K box sum over all channels, which a
    zero-padded summed-area table S yields in closed form:
    S(y+K, x+K) - S(y, x+K) - S(y+K, x) + S(y, x).  Integer data: exact."""
    for n, (C, Wx, Wy, K) in enumerate(shapes):
        I, _ = random_arrays(C, 1, Wx, Wy, K, seed + n, variant="int")
        F = np.ones((2, C, K, K), dtype=np.float32)
        F[1] *= -1.0
        O, A = conv(I, F)
        plane = I.astype(np.float64).sum(axis=0)
        S = np.zeros((Wy + 1, Wx + 1))
        S[1:, 1:] = plane.cumsum(0).cumsum(1)
        Hout, Wout = Wy - K + 1, Wx - K + 1
        box = S[K:K + Hout, K:K + Wout] - S[0:Hout, K:K + Wout] - S[K:K + Hout, 0:Wout] + S[0:Hout, 0:Wout]
        exact(O[0], box, "box sum %r" % ((C, Wx, Wy, K),))
        exact(O[1], -box, "negated box sum %r" % ((C, Wx, Wy, K),))
        Sa = np.zeros((Wy + 1, Wx + 1))
        Sa[1:, 1:] = np.abs(I).astype(np.float64).sum(axis=0).cumsum(0).cumsum(1)
        abox = (Sa[K:K + Hout, K:K + Wout] - Sa[0:Hout, K:K + Wout] - Sa[K:K + Hout, 0:Wout]
                + Sa[0:Hout, 0:Wout])
        exact(A[0], abox, "abs box sum %r" % ((C, Wx, Wy, K),))
        exact(A[1], abox, "abs box sum of the negated filter %r" % ((C, Wx, Wy, K),))


def pin_k1_is_gemm(conv, shapes, seed=6):
    """K = 1: O[m] = sum_c F[m][c] * I[c], a matrix product (M x C)(C x P)."""
    for n, (C, M, Wx, Wy) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, 1, seed + n)
        O, A = conv(I, F)
        ref = (F.reshape(M, C).astype(np.float64) @ I.reshape(C, -1).astype(np.float64)).reshape(M, Wy, Wx)
        close(O, ref, A, "K=1 GEMM %r" % ((C, M, Wx, Wy),))


def pin_full_window_is_dot(conv, shapes, seed=7):
    """K = Wx = Wy: the single output of filter m is the dot product <I, F[m]>."""
    for n, (C, M, W) in enumerate(shapes):
        I, F = random_arrays(C, M, W, W, W, seed + n)
        O, A = conv(I, F)
        ref = F.reshape(M, -1).astype(np.float64) @ I.reshape(-1).astype(np.float64)
        close(O[:, 0, 0], ref, A[:, 0, 0], "full-window dot %r" % ((C, M, W),))


def pin_separable(conv, shapes, seed=8):
    """F = u v^T on one channel: a pass of v along x, then of u along y
    (numpy.correlate in 'valid' mode)."""
    rng = np.random.default_rng(seed)
    for n, (Wx, Wy, K) in enumerate(shapes):
        I, _ = random_arrays(1, 1, Wx, Wy, K, seed + n)
        u = rng.uniform(-1, 1, K).astype(np.float32)
        v = rng.uniform(-1, 1, K).astype(np.float32)
        F = np.outer(u, v).astype(np.float32)
        # the product u_r * v_s rounded to fp32 is what the oracle sees; use it
        # exactly, and compare the separable form within the fp64 order bound
        O, A = conv(I, F[None, None])
        rows = np.array([np.correlate(I[0, y].astype(np.float64), v.astype(np.float64), "valid")
                         for y in range(Wy)])
        ref = np.array([np.correlate(rows[:, x], u.astype(np.float64), "valid")
                        for x in range(rows.shape[1])]).T
        err = np.abs(O[0] - ref)
        # u_r*v_s in fp32 differs from the exact product by <= 2^-24 relative
        assert (err <= 2.0 ** -23 * A[0] + 1e-300).all(), "separable %r" % ((Wx, Wy, K),)


# --- invariants of Eq. 1 ---------------------------------------------------------

def pin_linearity(conv, shapes, seed=9):
    """conv(2 I1 - 3 I2, F) = 2 conv(I1, F) - 3 conv(I2, F), and the same in F.
    Integer data keeps every value exact, so equality is exact."""
    for n, (C, M, Wx, Wy, K) in enumerate(shapes):
        I1, F1 = random_arrays(C, M, Wx, Wy, K, seed + n, variant="int")
        I2, F2 = random_arrays(C, M, Wx, Wy, K, seed + 1000 + n, variant="int")
        O1, _ = conv(I1, F1)
        O2, _ = conv(I2, F1)
        O3, _ = conv(I1, F2)
        Oi, _ = conv((2 * I1 - 3 * I2).astype(np.float32), F1)
        Of, _ = conv(I1, (2 * F1 - 3 * F2).astype(np.float32))
        exact(Oi, 2 * O1 - 3 * O2, "linear in I %r" % ((C, M, Wx, Wy, K),))
        exact(Of, 2 * O1 - 3 * O3, "linear in F %r" % ((C, M, Wx, Wy, K),))


def pin_channel_additivity(conv, shapes, seed=10):
    """Eq. 1 sums Eq. 2 over channels: multi(I, F) = sum_c single(I[c], F[:, c])."""
    for n, (C, M, Wx, Wy, K) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, K, seed + n, variant="int")
        O, _ = conv(I, F)
        acc = np.zeros_like(O)
        for c in range(C):
            Oc, _ = conv(I[c:c + 1], F[:, c:c + 1])
            acc += Oc
        exact(O, acc, "channel additivity %r" % ((C, M, Wx, Wy, K),))


def pin_filter_independence(conv, shapes, seed=11):
    """Output map m depends on filter m only."""
    for n, (C, M, Wx, Wy, K) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, K, seed + n)
        O, A = conv(I, F)
        for m in range(M):
            Om, Am = conv(I, F[m:m + 1])
            exact(O[m], Om[0], "filter %d of %r" % (m, (C, M, Wx, Wy, K)))
            exact(A[m], Am[0], "abs-sum of filter %d" % m)


def pin_translation(conv, shapes, seed=12):
    """Cropping the input by (dy, dx) crops the output by the same amount."""
    for n, (C, M, Wx, Wy, K, dy, dx) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, K, seed + n)
        O, _ = conv(I, F)
        Oc, _ = conv(np.ascontiguousarray(I[:, dy:, dx:]), F)
        exact(Oc, O[:, dy:, dx:], "translation %r" % ((C, M, Wx, Wy, K, dy, dx),))


def pin_abs_sum(conv, shapes, seed=13):
    """A = sum |I * F| equals the convolution of |I| with |F|; for
    non-negative data A equals O."""
    for n, (C, M, Wx, Wy, K) in enumerate(shapes):
        I, F = random_arrays(C, M, Wx, Wy, K, seed + n)
        O, A = conv(I, F)
        Oa, Aa = conv(np.abs(I), np.abs(F))
        exact(Oa, Aa, "non-negative data: O == A %r" % ((C, M, Wx, Wy, K),))
        close(A, Oa, Aa, "A == conv(|I|, |F|) %r" % ((C, M, Wx, Wy, K),))


def brute_force(I, F):
    """Exhaustive evaluation of Eq. 1 with Python integers (exact) for tiny
    integer-valued inputs; the loops walk every (m, y, x) and every term."""
    C, Wy, Wx = I.shape
    M, _, K, _ = F.shape
    Ii = I.astype(np.int64).tolist()
    Fi = F.astype(np.int64).tolist()
    out = np.zeros((M, Wy - K + 1, Wx - K + 1), dtype=np.int64)
    for m in range(M):
        for y in range(Wy - K + 1):
            for x in range(Wx - K + 1):
                total = 0
                for c in range(C):
                    for j in range(K):
                        for i in range(K):
                            total += Ii[c][y + j][x + i] * Fi[m][c][j][i]
                out[m, y, x] = total
    return out


def pin_brute_force(conv, max_w=5, seed=14):
    """Every shape with 1 <= Wx, Wy <= max_w, 1 <= K <= min(Wx, Wy), C, M in
    {1, 2} on integer data: exact equality with the exhaustive sum."""
    n = 0
    for Wy in range(1, max_w + 1):
        for Wx in range(1, max_w + 1):
            for K in range(1, min(Wx, Wy) + 1):
                for C in (1, 2):
                    for M in (1, 2):
                        I, F = random_arrays(C, M, Wx, Wy, K, seed + n, variant="int")
                        n += 1
                        O, _ = conv(I, F)
                        exact(O, brute_force(I, F), "brute force %r" % ((C, M, Wx, Wy, K),))


# Shapes small enough for the whole pin set to run in seconds, covering
# C != M, Wx != Wy, odd and even K, and K at both extremes.
SHAPES = [(1, 1, 7, 5, 3), (3, 2, 9, 6, 4), (2, 5, 11, 13, 5), (4, 3, 8, 8, 1),
          (2, 2, 6, 6, 6), (5, 4, 16, 10, 7), (1, 3, 12, 12, 11)]
SHAPES_2D = [(7, 5, 3), (12, 9, 4), (20, 20, 5), (9, 9, 9), (30, 17, 2)]
SHAPES_BOX = [(1, 9, 7, 3), (3, 10, 12, 5), (2, 6, 6, 6), (4, 13, 9, 1)]
SHAPES_K1 = [(3, 2, 5, 4), (8, 6, 7, 7), (16, 9, 3, 11)]
SHAPES_FULL = [(1, 1, 1), (2, 3, 3), (3, 2, 5), (4, 4, 7)]
SHAPES_SHIFT = [(2, 3, 12, 10, 3, 2, 3), (1, 1, 15, 15, 5, 4, 1), (3, 2, 9, 11, 2, 0, 5)]


def run_all(conv, brute_max_w=5):
    """Every pin, in a fixed order; returns the names that passed."""
    pins = [
        ("torch_conv2d", lambda: pin_torch_conv2d(conv, SHAPES)),
        ("scipy_correlate2d", lambda: pin_scipy_correlate2d(conv, SHAPES_2D)),
        ("sliding_window", lambda: pin_sliding_window(conv, SHAPES)),
        ("delta", lambda: pin_delta(conv, SHAPES)),
        ("box_sum", lambda: pin_box_sum(conv, SHAPES_BOX)),
        ("k1_gemm", lambda: pin_k1_is_gemm(conv, SHAPES_K1)),
        ("full_window_dot", lambda: pin_full_window_is_dot(conv, SHAPES_FULL)),
        ("separable", lambda: pin_separable(conv, SHAPES_2D)),
        ("linearity", lambda: pin_linearity(conv, SHAPES)),
        ("channel_additivity", lambda: pin_channel_additivity(conv, SHAPES)),
        ("filter_independence", lambda: pin_filter_independence(conv, SHAPES)),
        ("translation", lambda: pin_translation(conv, SHAPES_SHIFT)),
        ("abs_sum", lambda: pin_abs_sum(conv, SHAPES)),
        ("brute_force", lambda: pin_brute_force(conv, brute_max_w)),
    ]
    failed = []
    for name, fn in pins:
        try:
            fn()
        except AssertionError as e:
            failed.append((name, str(e)))
    return failed
