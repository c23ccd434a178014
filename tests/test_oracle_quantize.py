"""Pins of the oracle's row quantization (closed-form bounds, invariants, torch)."""

import numpy as np
import torch

import workloads as wl
from oracle import e4m3, quantize as oq


def _rows(seed, M=16, K=512):
    return wl.linear_activations(M, K, seed, outlier_frac=0.01, outlier_scale=20.0)


def test_bf16_helpers_match_torch():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(100000) * 10.0 ** rng.uniform(-30, 30, 100000)).astype(np.float32)
    bits = wl.bf16_bits_from_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bits, ref)
    back = oq.bf16_to_f32(bits)
    np.testing.assert_array_equal(back, torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())
    # fp64 -> bf16 equals torch's fp32 -> bf16 on fp32-exact values
    np.testing.assert_array_equal(oq.f64_to_bf16(x.astype(np.float64)), ref)


def test_error_bound_closed_form():
    x_bits = _rows(0)
    q, s = oq.quantize_rows(x_bits)
    x = oq.bf16_to_f32(x_bits).astype(np.float64)
    xr = e4m3.decode(q) * s[:, None].astype(np.float64)
    err = np.abs(xr - x)
    y_abs = np.abs(x) / s[:, None]
    normal = y_abs >= 2.0 ** -6
    # E4M3 RNE: half an ulp (2^-4 relative) in the normal range, half of 2^-9 absolute
    # below it; the fp32 product x * fl32(1/s) adds at most a few 2^-24 relative.
    assert np.all(err[normal] <= (2.0 ** -4) * np.abs(x[normal]) * (1 + 2.0 ** -20))
    sub = ~normal
    assert np.all(err[sub] <= (2.0 ** -10) * s[:, None].repeat(x.shape[1], 1)[sub] * (1 + 2.0 ** -20))


def test_amax_maps_to_448():
    x_bits = _rows(3)
    q, s = oq.quantize_rows(x_bits)
    x = oq.bf16_to_f32(x_bits)
    idx = np.argmax(np.abs(x), axis=1)
    top = q[np.arange(q.shape[0]), idx]
    assert np.all((top & 0x7F) == 0x7E)
    assert np.all(s == (x.astype(np.float64)[np.arange(len(idx)), idx].__abs__() / 448.0).astype(np.float32))


def test_zero_row_and_signed_zero():
    x = np.zeros((2, 64), np.float32)
    x[1, ::2] = -0.0
    q, s = oq.quantize_rows(wl.bf16_bits_from_f32(x))
    assert np.all(s == np.float32(2.0 ** -100))
    assert np.all(q[0] == 0)
    assert np.all(q[1, ::2] == 0x80) and np.all(q[1, 1::2] == 0)


def test_power_of_two_scaling_invariance():
    """Scaling a row by 2^j scales s by 2^j and leaves every code unchanged."""
    x_bits = _rows(4)
    q0, s0 = oq.quantize_rows(x_bits)
    x = oq.bf16_to_f32(x_bits)
    for j in (-20, -3, 5, 40):
        xj = wl.bf16_bits_from_f32((x * np.float32(2.0 ** j)).astype(np.float32))
        qj, sj = oq.quantize_rows(xj)
        np.testing.assert_array_equal(qj, q0)
        np.testing.assert_array_equal(sj, (s0 * np.float32(2.0 ** j)).astype(np.float32))


def test_sign_symmetry():
    x_bits = _rows(6)
    q, s = oq.quantize_rows(x_bits)
    qn, sn = oq.quantize_rows(x_bits ^ np.uint16(0x8000))
    np.testing.assert_array_equal(sn, s)
    np.testing.assert_array_equal(qn, q ^ np.uint8(0x80))


def test_scale_is_correctly_rounded_quotient():
    rng = np.random.default_rng(9)
    amax = (rng.random(100000) * 10.0 ** rng.uniform(-20, 20, 100000)).astype(np.float32)
    s = oq.row_scale(amax)
    ref = (torch.from_numpy(amax) / 448.0).numpy()     # fp32 IEEE division
    np.testing.assert_array_equal(s, np.maximum(ref, np.float32(2.0 ** -100)))
    inv = oq.reciprocal(s)
    np.testing.assert_array_equal(inv, (1.0 / torch.from_numpy(s)).numpy())


def test_per_tensor_calibration_is_max_of_row_scales():
    batches = [wl.student_t_activations(32, 256, seed=100 + i) for i in range(4)]
    s_tensor = oq.calibrate_per_tensor(batches)
    row_max = max(oq.quantize_rows(b)[1].max() for b in batches)
    assert s_tensor == row_max


def test_per_tensor_equals_per_row_when_rows_share_amax():
    x = oq.bf16_to_f32(_rows(7)).copy()
    x[:, 0] = 100.0                                   # same amax on every row
    xb = wl.bf16_bits_from_f32(x)
    q_row, s_row = oq.quantize_rows(xb)
    assert np.all(s_row == s_row[0])
    np.testing.assert_array_equal(oq.quantize_per_tensor(xb, s_row[0]), q_row)


def test_silu_mul_against_torch_and_special_cases():
    xb = wl.gated_ffn_input(8, 256, seed=11, std=3.0)
    h = oq.silu_mul(xb)
    x = torch.from_numpy(oq.bf16_to_f32(xb).astype(np.float64))
    ref = torch.nn.functional.silu(x[:, :256]) * x[:, 256:]
    ref_b = oq.f64_to_bf16(ref.numpy())
    # torch's silu in fp64 differs from g/(1+exp(-g)) by an ulp of fp64 at most:
    # bf16 roundings agree except where the fp64 value sits on a bf16 tie.
    assert np.mean(h != ref_b) < 1e-3
    z = np.zeros((1, 4), np.float32)
    z[0, 2:] = [5.0, 7.0]                             # g = 0 -> h = 0
    assert np.all(oq.silu_mul(wl.bf16_bits_from_f32(z)) == 0)
    big = np.array([[30.0, 2.0]], np.float32)        # silu(30) = 30 to 1e-12 -> h = 60
    assert oq.bf16_to_f32(oq.silu_mul(wl.bf16_bits_from_f32(big)))[0, 0] == 60.0


def test_clip_rate_definition():
    cal = [wl.bf16_bits_from_f32(np.array([[-2.0, 0.5, 3.0]], np.float32))]
    lo, hi = oq.calibrate_minmax(cal)
    assert (lo, hi) == (-2.0, 3.0)
    test = wl.bf16_bits_from_f32(np.array([[-2.5, -2.0, 0.0, 3.0, 3.5, 1.0, 10.0, -1.0]], np.float32))
    assert oq.clip_rate(test, lo, hi) == 3 / 8


def test_clip_count_static_against_the_calibrated_range():
    """A value clips iff it lies beyond the calibrated amax (up to the rounding
    of s and 1/s); the calibration rows themselves never clip; every clipped
    value encodes to +-448."""
    cal = _rows(7, M=32)
    s = oq.calibrate_per_tensor([cal])
    assert oq.clip_count_static(cal, s) == 0
    amax = float(np.max(np.abs(oq.bf16_to_f32(cal))))
    vals = np.array([0.0, amax * 0.5, -amax * 0.99, amax * 1.02, -amax * 1.5, amax * 4.0, -amax * 1.02], np.float32)
    bits = wl.bf16_bits_from_f32(vals)[None, :]
    x = oq.bf16_to_f32(bits)[0]
    expect = int(np.count_nonzero(np.abs(x) > amax * (1 + 2.0 ** -8)))
    assert oq.clip_count_static(bits, s) == expect == 4
    q = oq.quantize_per_tensor(bits, s)
    clipped = np.abs(x) > amax * (1 + 2.0 ** -8)
    assert np.all((q[0][clipped] & 0x7F) == 0x7E)
    # halving the scale doubles the range needed: values above amax/2 now clip
    assert oq.clip_count_static(bits, np.float32(s / 2)) == int(np.count_nonzero(np.abs(x) > amax / 2 * (1 + 2.0 ** -8)))
