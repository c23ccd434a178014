"""Pins of the oracle's W8A8 GEMM: integer-exact, Fraction brute force, one-hot selection."""

from fractions import Fraction

import numpy as np

from oracle import e4m3, gemm as og

FINITE = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)


def _codes(rng, shape):
    return rng.choice(FINITE, size=shape).astype(np.uint8)


def test_decode_int_matches_value_times_512():
    v = e4m3.decode(FINITE) * 512.0
    np.testing.assert_array_equal(og.decode_int512(FINITE).astype(np.float64), v)


def test_fp64_accumulation_equals_integer_gemm():
    rng = np.random.default_rng(0)
    for (M, N, K) in [(8, 16, 128), (33, 40, 512), (4, 8, 14336)]:
        a = _codes(rng, (M, K))
        w = _codes(rng, (N, K))
        acc = og.gemm_acc(a, w)
        ref = og.gemm_acc_int(a, w)
        np.testing.assert_array_equal(acc * 2.0 ** 18, ref.astype(np.float64))
        assert np.all(np.abs(ref) < 2 ** 53)


def test_saturated_operands_k14336_exact():
    a = np.full((2, 14336), 0x7E, np.uint8)
    w = np.full((3, 14336), 0x7E, np.uint8)
    w[1] = 0xFE
    acc = og.gemm_acc(a, w)
    assert acc[0, 0] == 448.0 * 448.0 * 14336 and acc[0, 1] == -acc[0, 0]


def test_fraction_brute_force_tiny():
    rng = np.random.default_rng(1)
    a = _codes(rng, (3, 5))
    w = _codes(rng, (4, 5))
    sa = np.array([0.5, 1.25, 3.0], np.float32)
    sw = np.array([2.0, 0.125, 1.0, 7.5], np.float32)
    y = og.gemm(a, sa, w, sw)
    for m in range(3):
        for n in range(4):
            s = Fraction(0)
            for kk in range(5):
                s += Fraction(float(e4m3.decode(a[m:m + 1, kk])[0])) * Fraction(float(e4m3.decode(w[n:n + 1, kk])[0]))
            assert Fraction(y[m, n]) == s * Fraction(float(sa[m])) * Fraction(float(sw[n]))


def test_one_hot_rows_select_weight_columns():
    """A[m] = 1.0 at column c_m only => acc[m, n] = dec(W[n, c_m]) (catches a transposed W)."""
    rng = np.random.default_rng(2)
    M, N, K = 6, 10, 256
    cols = rng.choice(K, M, replace=False)
    a = np.zeros((M, K), np.uint8)
    a[np.arange(M), cols] = 0x38                   # 1.0
    w = _codes(rng, (N, K))
    acc = og.gemm_acc(a, w)
    np.testing.assert_array_equal(acc, e4m3.decode(w[:, cols]).T)


def test_order_independence_is_exact():
    rng = np.random.default_rng(3)
    a = _codes(rng, (5, 4096))
    w = _codes(rng, (7, 4096))
    perm = rng.permutation(4096)
    np.testing.assert_array_equal(og.gemm_acc(a, w), og.gemm_acc(a[:, perm], w[:, perm]))


def test_scales_per_row_per_tensor():
    rng = np.random.default_rng(4)
    a = _codes(rng, (4, 128))
    w = _codes(rng, (6, 128))
    acc = og.gemm_acc(a, w)
    y = og.gemm(a, np.float32(0.25), w, np.float32(8.0))
    np.testing.assert_array_equal(y, acc * 2.0)
    sa = np.array([1, 2, 4, 8], np.float32)
    y2 = og.gemm(a, sa, w, np.float32(1.0))
    np.testing.assert_array_equal(y2, acc * sa[:, None])
    np.testing.assert_array_equal(og.gemm_rows(a, sa, w, np.float32(1.0), [2]), y2[2:3])


def test_rel_error_metric():
    y_ref = np.array([[100.0, -50.0, 0.0], [0.0, 0.0, 0.0]])
    assert og.rel_error(y_ref, y_ref) == 0.0
    y = y_ref + np.array([[0.1, 0.0, 0.05], [0.0, 1e-3, 0.0]])
    # row 0: 0.1 / 100; row 1 has no magnitude, its error is taken absolutely
    assert abs(og.rel_error(y, y_ref) - 1e-3) < 1e-15


def test_elementwise_metric_floors_vanishing_outputs():
    y_ref = np.array([[1.0, -2.0, 0.0, 4.0], [3.0, 3.0, 3.0, 3.0]])
    rms0 = np.sqrt(np.mean(y_ref[0] ** 2))
    y = y_ref.copy()
    y[0, 1] *= 1 + 1e-3                                 # relative 1e-3 on its own magnitude
    assert abs(og.rel_error_elementwise(y, y_ref) - 1e-3) < 1e-12
    y = y_ref.copy()
    y[0, 2] = 1e-4                                      # a zero output: measured against 0.01 rms
    assert abs(og.rel_error_elementwise(y, y_ref) - 1e-4 / (0.01 * rms0)) < 1e-9
    y = y_ref.copy()
    y[1, 0] = 3.0 * (1 - 5e-4)
    assert abs(og.rel_error_elementwise(y, y_ref) - 5e-4) < 1e-12
    # never looser than the row-normwise metric on the same outputs
    rng = np.random.default_rng(3)
    y_ref = rng.standard_normal((20, 300))
    y = y_ref + 1e-4 * rng.standard_normal((20, 300))
    assert og.rel_error_elementwise(y, y_ref) >= og.rel_error(y, y_ref)
