"""E4M3 (OCP "E4M3FN") codec written out from the format definition.

The paper quantizes weights and activations to FP8 E4M3 (paper §3.2 FP8
Post-Training Quantization).  E4M3 as defined by the OCP 8-bit floating point
specification (OFP8, rev. 1.0):

  code = S EEEE MMM   (sign, 4 exponent bits with bias 7, 3 mantissa bits)
  E == 0             -> (-1)^S * M * 2^-9            (subnormals, and +-0)
  1 <= E, not NaN    -> (-1)^S * (8 + M) * 2^(E-10)  (normals)
  S 1111 111         -> NaN (0x7F, 0xFF); there is no infinity
  largest finite magnitude 0x7E = (8+6) * 2^5 = 448.

Encoding follows the saturating ("satfinite") conversion used by the verify
path: finite values are rounded to the nearest representable value with ties
to the even mantissa; any magnitude above 448, infinities included, becomes
+-448; NaN becomes 0x7F.  The sign is always kept, so -0 encodes to 0x80.
"""

from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
NAN_CODE = 0x7F


def decode(codes) -> np.ndarray:
    """Codes (uint8, any shape) -> values in fp64; NaN codes give NaN."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    s = (c >> 7) & 1
    e = (c >> 3) & 0xF
    m = c & 0x7
    sub = m.astype(np.float64) * 2.0 ** -9
    nrm = np.ldexp((8 + m).astype(np.float64), (e - 10).astype(np.int64))
    v = np.where(e == 0, sub, nrm)
    v = np.where(s == 1, -v, v)
    v = np.where((e == 15) & (m == 7), np.nan, v)
    return v


def decode_table() -> np.ndarray:
    """Value of each of the 256 codes, fp64 [256]."""
    return decode(np.arange(256, dtype=np.uint8))


def encode(y) -> np.ndarray:
    """fp32 values (any shape) -> E4M3 codes (uint8), RNE, saturating.

    Works exactly in fp64: for 0 < a <= 448 the exponent of the quantum is
    e = max(floor(log2 a), -6) and the quantum is 2^(e-3); n = a / quantum is
    exact (a power-of-two scaling) and is rounded to the nearest integer with
    ties to even; n * quantum is then re-encoded, a mantissa carry (n == 16)
    moving to the next binade and n == 8 at e == -6 becoming the smallest
    normal 0x08.
    """
    y = np.asarray(y, dtype=np.float32)
    y64 = y.astype(np.float64)
    sign = np.signbit(y).astype(np.int64)
    a = np.abs(y64)
    nan = np.isnan(y64)
    sat = (a > E4M3_MAX) & ~nan
    fin = ~nan & ~sat
    a_f = np.where(fin, a, 0.0)

    # floor(log2 a) exactly: a = f * 2^ex with f in [0.5, 1).
    _, ex = np.frexp(a_f)
    e = np.maximum(ex.astype(np.int64) - 1, -6)
    quantum_exp = e - 3
    n = np.rint(np.ldexp(a_f, -quantum_exp))          # exact scaling, RNE
    val = np.ldexp(n, quantum_exp)                    # the rounded magnitude

    # re-encode val into (E, M)
    _, ex2 = np.frexp(val)
    e2 = ex2.astype(np.int64) - 1                     # floor(log2 val) for val > 0
    is_sub = val < 2.0 ** -6
    m_sub = np.ldexp(val, 9).astype(np.int64)         # val / 2^-9, integer 0..7
    E_nrm = e2 + 7
    m_nrm = np.ldexp(val, -(e2 - 3)).astype(np.int64) - 8
    E = np.where(is_sub, 0, E_nrm)
    M = np.where(is_sub, m_sub, m_nrm)
    code = (sign << 7) | (E << 3) | M
    code = np.where(sat, (sign << 7) | 0x7E, code)
    code = np.where(nan, NAN_CODE, code)
    return code.astype(np.uint8)
