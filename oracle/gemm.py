"""FP8 W8A8 linear: Y = (A_q W_q^T) scaled by per-row and per-channel scales.

In a W8A8 linear (paper §3.2 FP8 Post-Training Quantization) both operands
are E4M3 codes; the product is accumulated and then rescaled:

  acc[m,n] = sum_k dec(A[m,k]) * dec(W[n,k])      A [M,K], W [N,K] (nn.Linear)
  y[m,n]   = acc[m,n] * sa[m] * sw[n]

with sa the per-token (or one per-tensor) activation scale and sw the
per-output-channel (or one per-tensor) weight scale.

Exactness: every E4M3 value is an integer multiple of 2^-9, so each product is
a multiple of 2^-18 with magnitude <= 448^2.  For K <= 14336 every partial sum
is below 2^32 in magnitude, i.e. fewer than 2^50 units of 2^-18, so the fp64
accumulation below is exact in any summation order, and `gemm_acc_int` (an
int64 GEMM on value*2^9 integers) gives the same numbers times 2^18.
"""

from __future__ import annotations

import numpy as np

from . import e4m3

K_EXACT_MAX = 14336 * 4   # bound used by the exactness argument (with margin 4x under 2^53)


def decode_int512(codes) -> np.ndarray:
    """E4M3 codes -> int64 integers equal to value * 2^9 (finite codes only)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    s = (c >> 7) & 1
    e = (c >> 3) & 0xF
    m = c & 0x7
    mag = np.where(e == 0, m, (8 + m) << np.maximum(e - 1, 0))
    return np.where(s == 1, -mag, mag)


def gemm_acc(a_codes: np.ndarray, w_codes: np.ndarray) -> np.ndarray:
    """acc = dec(A) @ dec(W)^T in fp64 (exact for K <= K_EXACT_MAX)."""
    tab = e4m3.decode_table()
    a = tab[np.asarray(a_codes, dtype=np.uint8)]
    w = tab[np.asarray(w_codes, dtype=np.uint8)]
    if a.shape[1] > K_EXACT_MAX:
        raise ValueError("K beyond the exact-accumulation bound")
    return a @ w.T


def gemm_acc_int(a_codes: np.ndarray, w_codes: np.ndarray) -> np.ndarray:
    """Integer GEMM: (value*2^9 of A) @ (value*2^9 of W)^T in int64 (= acc * 2^18)."""
    a = decode_int512(a_codes)
    w = decode_int512(w_codes)
    return a @ w.T


def apply_scales(acc: np.ndarray, sa, sw) -> np.ndarray:
    """y = acc * sa[m] * sw[n] in fp64; sa/sw may be scalars (per-tensor)."""
    sa = np.asarray(sa, dtype=np.float32).astype(np.float64)
    sw = np.asarray(sw, dtype=np.float32).astype(np.float64)
    sa = sa.reshape(-1, 1) if sa.ndim else sa
    sw = sw.reshape(1, -1) if sw.ndim else sw
    return acc * sa * sw


def gemm(a_codes, sa, w_codes, sw) -> np.ndarray:
    """The W8A8 linear in fp64: [M,N]."""
    return apply_scales(gemm_acc(a_codes, w_codes), sa, sw)


def gemm_rows(a_codes, sa, w_codes, sw, rows) -> np.ndarray:
    """Selected output rows only (for sampled checks at full size)."""
    rows = np.asarray(rows)
    sa = np.asarray(sa, dtype=np.float32)
    sa_r = sa[rows] if sa.ndim else sa
    return gemm(np.asarray(a_codes)[rows], sa_r, w_codes, sw)


def rel_error(y: np.ndarray, y_ref: np.ndarray) -> float:
    """Largest error of any output relative to the largest magnitude of its row.

    max_m max_n |y[m,n] - y_ref[m,n]| / max_n |y_ref[m,n]|: the infinity-norm
    relative error of every output row (one token's activations), which stays
    meaningful for outputs that cancel to near zero.
    """
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    if y_ref.size == 0:
        return 0.0
    scale = np.max(np.abs(y_ref), axis=1, keepdims=True)
    scale = np.where(scale > 0, scale, 1.0)
    return float(np.max(np.abs(y - y_ref) / scale))


def rel_error_elementwise(y: np.ndarray, y_ref: np.ndarray, floor_frac: float = 0.01) -> float:
    """Largest error of any output relative to its own magnitude, floored.

    max_{m,n} |y - y_ref| / max(|y_ref[m,n]|, floor_frac * rms_n(y_ref[m, :])):
    the per-output relative error, where outputs that cancel to below
    floor_frac of their row's root-mean-square are measured against that
    fraction of the rms instead of their own (vanishing) magnitude.
    """
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    if y_ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(y_ref * y_ref, axis=1, keepdims=True))
    den = np.maximum(np.abs(y_ref), floor_frac * rms)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(y - y_ref) / den))
