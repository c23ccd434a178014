"""Row quantization to E4M3 with fp32 scales.

The paper applies W8A8 E4M3 quantization with min-max scales (paper §3.2 FP8
Post-Training Quantization).  E4M3 is symmetric and has no zero point, so a
min-max range [lo, hi] maps to the scale amax / 448 with
amax = max(|lo|, |hi|) = max |x|.  The verify path uses that rule per row:
per token for activations (dynamic, computed at run time) and per output
channel for weights (rows of W [N,K], computed once offline); the paper's own
static per-tensor scheme is the PER_TENSOR mode with one given scale.

For one row x (bf16 values, exact in fp32):
  amax = max_c |x_c|                       (exact)
  s    = max(fl32(amax / 448), S_MIN)      (the stored fp32 scale)
  inv  = fl32(1 / s)
  y_c  = fl32(x_c * inv)                   (one fp32 multiply, RNE)
  q_c  = E4M3_encode(y_c)                  (RNE, saturating)
so that x_c ~= decode(q_c) * s.  fl32(a / b) of two fp32 numbers is computed
as an fp64 quotient rounded once to fp32; that equals the correctly rounded
fp32 quotient (53 >= 2*24 + 2 bits).

S_MIN = 2^-100 keeps 1/s finite for an all-zero row (codes 0x00/0x80).

The SiLU-gated input of the down projection (the Llama FFN of the paper's
target model, §4 Experimental Setup) is h_c = silu(g_c) * u_c with
g = x[:, :I], u = x[:, I:], silu(g) = g / (1 + exp(-g)); h is rounded to bf16
(the model's activation dtype) before it is quantized.
"""

from __future__ import annotations

import numpy as np

from . import e4m3

S_MIN = np.float32(2.0 ** -100)


def bf16_to_f32(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> fp32 values, exact."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def f64_to_bf16(v) -> np.ndarray:
    """fp64 values -> bf16 bit patterns, one rounding to nearest-even.

    bf16 keeps 8 significand bits; rounding is done on the fp64 value
    directly (no intermediate fp32 rounding).  Finite inputs only.
    """
    v = np.asarray(v, dtype=np.float64)
    out = np.zeros(v.shape, dtype=np.uint16)
    sign = np.signbit(v)
    a = np.abs(v)
    nz = a > 0
    _, ex = np.frexp(np.where(nz, a, 1.0))
    e = ex.astype(np.int64) - 1                      # floor(log2 a)
    e = np.maximum(e, -126)                           # bf16 subnormal binade
    q = e - 7                                         # quantum exponent (8 significant bits)
    n = np.rint(np.ldexp(np.where(nz, a, 0.0), -q))   # exact scaling, RNE
    r = np.ldexp(n, q)
    r32 = r.astype(np.float32)                        # exact: r has <= 8 significant bits
    bits = (r32.view(np.uint32) >> 16).astype(np.uint16)
    bits = np.where(sign, bits | np.uint16(0x8000), bits)
    out[...] = bits
    return out


def row_scale(amax) -> np.ndarray:
    """s = max(fl32(amax/448), S_MIN) for fp32 amax values."""
    a = np.asarray(amax, dtype=np.float32).astype(np.float64)
    s = (a / 448.0).astype(np.float32)
    return np.maximum(s, S_MIN)


def reciprocal(s) -> np.ndarray:
    """fl32(1/s)."""
    return (1.0 / np.asarray(s, dtype=np.float32).astype(np.float64)).astype(np.float32)


def quantize_values(xf32: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Encode fp32 rows with given per-row scales [rows] -> codes uint8."""
    inv = reciprocal(scales)
    y = (xf32 * inv[:, None]).astype(np.float32)      # fp32 multiply, RNE
    return e4m3.encode(y)


def quantize_rows(x_bits: np.ndarray):
    """Dynamic per-row quantization of bf16 rows [R,C] -> (codes [R,C], s [R])."""
    x = bf16_to_f32(x_bits)
    amax = np.max(np.abs(x), axis=1) if x.shape[1] > 0 else np.zeros(x.shape[0], np.float32)
    s = row_scale(amax)
    return quantize_values(x, s), s


def quantize_per_tensor(x_bits: np.ndarray, scale: float):
    """Static per-tensor quantization with one given fp32 scale -> codes."""
    x = bf16_to_f32(x_bits)
    s = np.full(x.shape[0], np.float32(scale), dtype=np.float32)
    return quantize_values(x, s)


def silu_mul(x_bits: np.ndarray) -> np.ndarray:
    """h = bf16(silu(g) * u) for x = [g | u] bf16 [R, 2I] -> bf16 bits [R, I]."""
    x = bf16_to_f32(x_bits).astype(np.float64)
    inter = x.shape[1] // 2
    g, u = x[:, :inter], x[:, inter:]
    h = g / (1.0 + np.exp(-g)) * u
    return f64_to_bf16(h)


def quantize_silu_mul_rows(x_bits: np.ndarray):
    """Per-row quantization of h = silu(g)*u -> (codes [R,I], s [R], h bits)."""
    h = silu_mul(x_bits)
    q, s = quantize_rows(h)
    return q, s, h


def calibrate_per_tensor(batches) -> np.float32:
    """Static min-max calibration: one scale from all calibration batches.

    amax over every calibration activation, s = max(fl32(amax/448), S_MIN).
    """
    amax = np.float32(0.0)
    for xb in batches:
        x = bf16_to_f32(xb)
        if x.size:
            amax = max(amax, np.float32(np.max(np.abs(x))))
    return np.float32(row_scale(np.array([amax], np.float32))[0])


def calibrate_minmax(batches):
    """Per-tensor (min, max) of all calibration activations, fp32."""
    lo, hi = np.float32(np.inf), np.float32(-np.inf)
    for xb in batches:
        x = bf16_to_f32(xb)
        if x.size:
            lo = min(lo, np.float32(np.min(x)))
            hi = max(hi, np.float32(np.max(x)))
    return lo, hi


def clip_rate(x_bits: np.ndarray, lo: float, hi: float) -> float:
    """Fraction of the values in x below lo or above hi, where [lo, hi] is
    the per-tensor range calibration produced (the clip-rate metric of the
    section FP8 Calibration Performance)."""
    x = bf16_to_f32(x_bits)
    if x.size == 0:
        return 0.0
    return float(np.mean((x < np.float32(lo)) | (x > np.float32(hi))))


def clip_count_static(x_bits: np.ndarray, scale: float) -> int:
    """Number of values the static per-tensor quantizer saturates: those with
    |fl32(x * fl32(1/s))| > 448, the largest E4M3 magnitude.

    This is the clip-rate metric of the section FP8 Calibration Performance
    read through the quantizer itself: with s = fl32(amax/448) from min-max
    calibration, a value clips exactly when its scaled magnitude leaves the
    E4M3 range, i.e. when |x| exceeds the calibrated amax up to the rounding
    of s and 1/s.
    """
    x = bf16_to_f32(x_bits)
    inv = reciprocal(np.array([scale], np.float32))[0]
    y = (x * inv).astype(np.float32)
    return int(np.count_nonzero(np.abs(y) > np.float32(448.0)))
