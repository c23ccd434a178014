"""GPU parity of spec_fp8_quantize / spec_silu_mul_bf16 against the CPU oracle.

FP8 codes and scales must match bit-exactly.  The SiLU-gated path is
bit-exact given the GPU's own bf16 intermediate h; against the oracle's h
(exp evaluated independently) codes may differ by one E4M3 step on a tiny
fraction of elements.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import e4m3, quantize as oq
from tests.gpu_util import dev_bf16, dev_f32, host, host_bf16_bits, need_gpu, say

pytestmark = pytest.mark.gpu


def _run(p, xb, per_tensor=None, silu=False):
    x = dev_bf16(xb)
    pt = None if per_tensor is None else dev_f32([per_tensor])
    q, s = p.quantize(x, per_tensor_scale=pt, silu_mul=silu)
    return host(q), host(s)


@pytest.mark.parametrize("rows,cols,seed", [
    (8, 512, 0),            # C1 activations
    (1, 8, 1), (3, 24, 2), (37, 520, 3),           # ragged, tiny
    (80, 4096, 4), (320, 4096, 5),                 # C2/C3 rows
    (5, 14336, 6),          # down-projection width, 7 chunks per thread
    (3, 16392, 7),          # wider than the register-resident path
    (2, 2056, 8),
])
def test_per_row_bit_exact(rows, cols, seed):
    p = need_gpu()
    say(f"quantize per-row rows={rows} cols={cols} seed={seed}")
    xb = wl.linear_activations(rows, cols, seed, outlier_frac=0.01, outlier_scale=20.0)
    q, s = _run(p, xb)
    q_ref, s_ref = oq.quantize_rows(xb)
    np.testing.assert_array_equal(s, s_ref)
    np.testing.assert_array_equal(q, q_ref)


def test_strided_rows_and_zero_rows():
    p = need_gpu()
    xb = wl.linear_activations(6, 256, 9)
    xb[2] = 0
    xb[4, ::3] = 0x8000                             # -0.0
    big = np.zeros((6, 264), np.uint16)
    big[:, :256] = xb
    x = dev_bf16(big)[:, :256]
    out = torch.zeros((6, 272), dtype=torch.uint8, device="cuda")
    q, s = p.quantize(x, out=out[:, :256])
    q_ref, s_ref = oq.quantize_rows(xb)
    np.testing.assert_array_equal(host(s), s_ref)
    np.testing.assert_array_equal(host(out)[:, :256], q_ref)
    assert np.all(host(out)[:, 256:] == 0)           # nothing written past cols


@pytest.mark.parametrize("scale", [1.0, 1.0 / 3.0, 0.7, 1.1e-5, 2.0 ** -20, 1e4])
def test_every_bf16_value_per_tensor(scale):
    """All 65536 bf16 patterns (finite) through encode(fl32(x * fl32(1/s)))."""
    p = need_gpu()
    say(f"quantize all bf16 values, per-tensor scale {scale}")
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    fin = np.isfinite(oq.bf16_to_f32(bits))
    bits = bits[fin]
    bits = bits.reshape(-1, 256)                    # 65280 finite patterns = 255 rows
    s = np.float32(scale)
    q, _ = _run(p, bits, per_tensor=s)
    np.testing.assert_array_equal(q, oq.quantize_per_tensor(bits, s))


def test_rounding_ties_and_neighbours():
    """Exact E4M3 midpoints (representable in bf16) and values nudged off them."""
    p = need_gpu()
    tab = e4m3.decode(np.arange(0, 0x7F, dtype=np.uint8))
    mids = ((tab[:-1] + tab[1:]) / 2).astype(np.float32)
    vals = np.concatenate([mids, -mids, tab.astype(np.float32), [448.0, 480.0, 1e6, -1e6]]).astype(np.float32)
    n = (len(vals) + 7) // 8 * 8
    vals = np.pad(vals, (0, n - len(vals)))
    xb = wl.bf16_bits_from_f32(vals).reshape(1, -1)
    for s in [1.0, float(np.float32(1.0) / np.float32(1 + 2 ** -22)), float(np.float32(1 + 2 ** -22))]:
        q, _ = _run(p, xb, per_tensor=np.float32(s))
        np.testing.assert_array_equal(q, oq.quantize_per_tensor(xb, np.float32(s)))


def test_silu_mul_intermediate_and_fused_codes():
    p = need_gpu()
    rows, inter = 37, 1032
    xb = wl.gated_ffn_input(rows, inter, seed=10, std=2.0)
    x = dev_bf16(xb)
    h_gpu = p.silu_mul(x)
    h_g = host_bf16_bits(h_gpu)
    q_o, s_o, h_o = oq.quantize_silu_mul_rows(xb)
    # h: independent exp implementations agree after bf16 rounding except at
    # rare near-ties, and then by one bf16 ulp
    diff = np.abs(h_g.astype(np.int32) - h_o.astype(np.int32))
    assert np.mean(diff != 0) < 1e-3 and np.max(diff) <= 1
    # the fused path is exactly the unfused composition on the GPU
    q, s = p.quantize(x, silu_mul=True)
    q2, s2 = p.quantize(h_gpu)
    np.testing.assert_array_equal(host(q), host(q2))
    np.testing.assert_array_equal(host(s), host(s2))
    # against the oracle: rows whose h agrees everywhere match bit-exactly;
    # elsewhere codes differ by at most one E4M3 step
    qg, sg = host(q), host(s)
    same = np.all(diff == 0, axis=1)
    assert same.sum() >= rows // 2
    np.testing.assert_array_equal(qg[same], q_o[same])
    np.testing.assert_array_equal(sg[same], s_o[same])
    step = np.abs(qg.astype(np.int32) - q_o.astype(np.int32))   # same sign: adjacent codes differ by 1
    assert np.max(step[~same], initial=0) <= 1
    assert np.mean(step != 0) <= 1e-4
    # given the GPU's own bf16 intermediate h, the fused codes and scales are the
    # oracle's quantization of h, bit for bit
    q_h, s_h = oq.quantize_rows(h_g)
    np.testing.assert_array_equal(qg, q_h)
    np.testing.assert_array_equal(sg, s_h)


def test_per_tensor_from_calibration_matches_row_scales():
    """C5 reading: the per-tensor scale from calibration is the max of the per-row scales."""
    p = need_gpu()
    batches = [wl.student_t_activations(64, 512, seed=200 + i) for i in range(4)]
    srow = [host(p.quantize(dev_bf16(b))[1]) for b in batches]
    assert np.float32(max(s.max() for s in srow)) == oq.calibrate_per_tensor(batches)


@pytest.mark.parametrize("cols", [512, 4096, 65536 + 512])     # registers, and the two-pass wide-row path
def test_calibrate_mode_bit_exact(cols):
    """SPEC_SCALE_CALIBRATE folds every batch into the running scale: equal
    to the oracle's min-max calibration bit for bit, also when the running
    value starts above the batches' own maximum (it must then stay put)."""
    p = need_gpu()
    batches = [wl.student_t_activations(rows, cols, seed=300 + i) for i, rows in enumerate((3, 17, 64, 1))]
    running = torch.zeros(1, dtype=torch.float32, device="cuda")
    for b in batches:
        p.calibrate(dev_bf16(b), running)
    ref = oq.calibrate_per_tensor(batches)
    assert host(running)[0].tobytes() == np.float32(ref).tobytes()
    big = torch.full((1,), float(ref) * 2.0, dtype=torch.float32, device="cuda")
    p.calibrate(dev_bf16(batches[0]), big)
    assert host(big)[0] == np.float32(float(ref) * 2.0)
    zero = torch.zeros(1, dtype=torch.float32, device="cuda")
    p.calibrate(dev_bf16(np.zeros((4, cols), np.uint16)), zero)      # all-zero rows: the scale floor 2^-100
    assert host(zero)[0] == np.float32(2.0 ** -100)


def test_calibrate_silu_mul_input():
    """Calibration of the SiLU-gated FFN input uses the same intermediate h
    as the fused quantize, so its scale equals the max of that path's row scales."""
    p = need_gpu()
    xb = wl.gated_ffn_input(40, 1024, seed=17)
    x = dev_bf16(xb)
    _, srow = p.quantize(x, silu_mul=True)
    running = torch.zeros(1, dtype=torch.float32, device="cuda")
    p.calibrate(x, running, silu_mul=True)
    assert host(running)[0] == host(srow).max()


def test_deterministic():
    p = need_gpu()
    xb = wl.linear_activations(64, 4096, 11, outlier_frac=0.005, outlier_scale=30.0)
    a = _run(p, xb)
    b = _run(p, xb)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_silu_mul_quantize_verify_step_width():
    """The SiLU-gated quantize at the width of the verify step's FFN
    (M = 320 rows of the gate|up output, 2 x 14336 bf16 -> 14336 codes), the
    shape and launch configuration the step runs.  The input is seeded
    synthetic gate|up output (N(0, 3^2), the spread of the C3 layer's gate|up
    values).  Given the GPU's own bf16 intermediate h the codes and scales
    are the oracle's quantization of h bit for bit; against the oracle's own
    h, codes differ by at most one E4M3 step on at most 1e-4 of elements."""
    p = need_gpu()
    cfg = wl.CONFIGS["C3"]
    M = cfg["M"]
    inter = dict((n, (N, K)) for n, N, K in cfg["linears"])["gate_up"][0] // 2
    say(f"SiLU-gated quantize {M} x 2*{inter}")
    xb = wl.gated_ffn_input(M, inter, seed=cfg["seed"] + 5, std=3.0)
    x = dev_bf16(xb)
    q, s = p.quantize(x, silu_mul=True)
    h_g = host_bf16_bits(p.silu_mul(x))
    qg, sg = host(q), host(s)
    q_h, s_h = oq.quantize_rows(h_g)
    np.testing.assert_array_equal(qg, q_h)
    np.testing.assert_array_equal(sg, s_h)
    q_o, s_o, h_o = oq.quantize_silu_mul_rows(xb)
    diff = np.abs(h_g.astype(np.int32) - h_o.astype(np.int32))
    assert np.max(diff) <= 1 and np.mean(diff != 0) < 1e-3
    same = np.all(diff == 0, axis=1)
    np.testing.assert_array_equal(qg[same], q_o[same])
    np.testing.assert_array_equal(sg[same], s_o[same])
    step = np.abs(qg.astype(np.int32) - q_o.astype(np.int32))
    say(f"h differs on {int((diff != 0).sum())} of {diff.size}; code steps {int((step != 0).sum())}")
    assert np.max(step, initial=0) <= 1
    assert np.mean(step != 0) <= 1e-4
