"""GPU parity of spec_fp8_gemm_silu_mul: the gate|up projection with the
SiLU gate in its epilogue, h = bf16(silu(gate) * up).

Against the oracle: its own codes (the device's must match bit for bit), the
exact GEMM rounded to bf16, then the oracle's SiLU gate in fp64.  Every
element must lie within the GEMM tolerance.  Exact equality is not the bar:
a gate or up value far below its row's largest output has a bf16 step
comparable to the fp32 accumulation error, so it often rounds to the
neighbouring value (a few percent of elements), and the device's fp32 SiLU
differs from an exact one at near-ties of h's rounding; the share of equal
elements is reported and must stay high (a wrong gate/up pairing would
leave almost none).  Against the unfused device path (bf16 GEMM output, then
spec_silu_mul_bf16, the same gate code) the only differences come from the
fp32 summation order.
"""

import numpy as np
import pytest

import workloads as wl
from oracle import gemm as og, quantize as oq
from tests.gpu_util import dev_bf16, host, host_bf16_bits, need_gpu, say

pytestmark = pytest.mark.gpu

TOL = 2e-3


def _operands(p, M, I, K, seed):
    xb = wl.linear_activations(M, K, seed, 0.005, 30.0)
    wb = wl.linear_weights(2 * I, K, seed + 1, 0.02)
    a, sa = p.quantize(dev_bf16(xb))
    w, sw = p.quantize(dev_bf16(wb))
    return xb, wb, a, sa, w, sw


def _close(h, y_ref, I):
    """Every device h within the error the oracle's inputs allow: each gate or
    up value g, u carries the GEMM tolerance (row-normwise over the 2I
    outputs) plus its bf16 rounding, dy = TOL max|y| + 2^-8 |y|, and
    |silu'| <= 1.1, so |dh| <= 1.1 dg |u| + |silu(g)| du + 1.1 dg du plus
    h's own rounding.  Returns (share of elements equal to the oracle's h,
    the oracle's h bits)."""
    y = oq.bf16_to_f32(oq.f64_to_bf16(y_ref)).astype(np.float64)
    h_ref = oq.silu_mul(oq.f64_to_bf16(y_ref))
    g, u = y[:, :I], y[:, I:]
    ymax = np.max(np.abs(y_ref), axis=1, keepdims=True)
    dg = TOL * ymax + 2.0 ** -8 * np.abs(g)
    du = TOL * ymax + 2.0 ** -8 * np.abs(u)
    sg = g / (1.0 + np.exp(-g))
    hf = oq.bf16_to_f32(h).astype(np.float64)
    rf = oq.bf16_to_f32(h_ref).astype(np.float64)
    bound = 1.1 * dg * np.abs(u) + np.abs(sg) * du + 1.1 * dg * du + 2.0 ** -8 * np.abs(rf) + 1e-30
    assert np.all(np.abs(hf - rf) <= bound)
    return float(np.mean(h == h_ref))


@pytest.mark.parametrize("M,I,K", [
    (8, 512, 512),          # 64-row tiles
    (80, 1000, 1024),       # 80-row tiles, ragged last tile
    (200, 2056, 512),       # ragged M and I
    (333, 1024, 256),       # M past 320
])
def test_silu_gemm_vs_oracle_and_unfused(M, I, K):
    p = need_gpu()
    say(f"silu gemm M={M} I={I} K={K}")
    xb, wb, a, sa, w, sw = _operands(p, M, I, K, seed=M + I + K)
    h = host_bf16_bits(p.gemm_silu_mul(a, sa, w, sw))
    qa, sa_ref = oq.quantize_rows(xb)
    qw, sw_ref = oq.quantize_rows(wb)
    np.testing.assert_array_equal(host(a), qa)
    np.testing.assert_array_equal(host(w), qw)
    same_oracle = _close(h, og.gemm(qa, sa_ref, qw, sw_ref), I)
    h_unfused = host_bf16_bits(p.silu_mul(p.gemm(a, sa, w, sw)))
    same_unfused = float(np.mean(h == h_unfused))
    say(f"  equal to the oracle on {same_oracle:.5f}, to the unfused path on {same_unfused:.5f} of elements")
    assert same_oracle >= 0.9
    assert same_unfused >= 0.995


def test_silu_gemm_full_size_sampled():
    """The benched FFN (M = 320, K = 4096, I = 14336), sampled h columns."""
    p = need_gpu()
    c = wl.CONFIGS["C3"]
    M = c["M"]
    I, K = 14336, 4096
    xb, wb, a, sa, w, sw = _operands(p, M, I, K, seed=c["seed"] + 3)
    h = host_bf16_bits(p.gemm_silu_mul(a, sa, w, sw))
    rng = np.random.default_rng(5)
    cols = np.unique(np.concatenate([[0, I - 1], rng.choice(I, 384, replace=False)]))
    rows = np.unique(np.concatenate([[0, M - 1], rng.choice(M, 6, replace=False)]))
    qa, sa_ref = oq.quantize_rows(xb[rows])
    wrows = np.concatenate([cols, I + cols])
    qw, sw_ref = oq.quantize_rows(wb[wrows])
    np.testing.assert_array_equal(host(a)[rows], qa)
    np.testing.assert_array_equal(host(w)[wrows], qw)
    same = _close(h[np.ix_(rows, cols)], og.gemm(qa, sa_ref, qw, sw_ref), len(cols))
    say(f"silu gemm full size: equal to the oracle on {same:.5f} of sampled elements")
    assert same >= 0.9
