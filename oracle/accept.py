"""Verification of a drafted chain: greedy match and speculative sampling.

In the paper's serving stack a draft model proposes k tokens and the target
model checks them all in one parallel forward pass, accepting k_bar > 1
tokens per step (paper §3.1 EAGLE; optimization-stack figure, "Layer 2").
The paper states that this preserves the target's output distribution
exactly and defers the acceptance rule to Leviathan et al. (2023) and Chen et
al. (2023).  That rule, restated here from its mathematics:

Inputs for one sequence b: target distributions p_0..p_k over the vocabulary
(position i scores draft x_i; position k scores the bonus token), draft
distributions q_0..q_{k-1}, drafts x_0..x_{k-1}, and k+1 uniforms u in [0,1).

  for i = 0..k-1:
      accept x_i iff u_i * q_i(x_i) < p_i(x_i)        (prob. min(1, p/q))
      on the first rejection: emit one token drawn from the residual
          r = max(0, p_i - q_i), normalised, by inverse CDF with u_k; stop.
  if all k are accepted: emit a bonus token drawn from p_k with u_k.

Greedy verification (temperature 0, argmax drafting as in the paper's greedy
EAGLE rows, Table 1/Table 2 and App. E "Draft Model Quantization and Greedy
Decoding") keeps x_i while x_i equals the target argmax g_i, then emits g_a
at the first mismatch a (or g_k after k matches).

Readings fixed here (the paper is silent on them):
  * p_i = softmax(z_t[b,i] / T), q_i = softmax(z_d[b,i] / T): one temperature
    for target and draft; T = 0 means greedy on the raw logits.
  * With no draft logits, q_i is one-hot at x_i (an argmax drafter): accept
    with probability p_i(x_i); the residual is p_i without x_i.
  * argmax ties go to the lowest vocabulary index.
  * A draft id outside [0, V) is a rejection with p(x) = q(x) = 0.
  * The residual sample: the smallest v with sum_{w<=v} r_w > u_k * R,
    R = sum_w r_w.  If R is 0 (only possible through rounding) the token is
    drawn from p_i instead; if u_k * R is not below the last cumulative value
    (rounding again) the last v with r_v > 0 is taken.
  * Outputs per sequence: out_tokens[b, 0..a_b] (a_b accepted drafts, then the
    resampled or bonus token), padded with -1 to k+1; num_accepted[b] = a_b.

The decision logic in `accept_chain` is written once and runs on fp64 numpy
vectors and on numpy object vectors of Fractions alike (the latter for the
exact-enumeration proof in oracle.enumerate).
"""

from __future__ import annotations

import numpy as np

from .quantize import bf16_to_f32


# --------------------------------------------------------------------------
# greedy
# --------------------------------------------------------------------------

def target_argmax(zt_bits: np.ndarray) -> np.ndarray:
    """argmax over the vocabulary of bf16 logits [..., V], lowest index on ties."""
    return np.argmax(bf16_to_f32(zt_bits), axis=-1).astype(np.int64)


def accept_greedy(zt_bits: np.ndarray, draft_tokens: np.ndarray):
    """Greedy chain verification -> (out_tokens [B,k+1] int32, num_accepted [B] int32)."""
    zt_bits = np.asarray(zt_bits)
    B, k1, V = zt_bits.shape
    k = k1 - 1
    x = np.asarray(draft_tokens, dtype=np.int64).reshape(B, k)
    g = target_argmax(zt_bits)                       # [B, k+1]
    out = np.full((B, k1), -1, dtype=np.int32)
    num = np.zeros(B, dtype=np.int32)
    for b in range(B):
        a = 0
        while a < k and x[b, a] == g[b, a]:
            out[b, a] = x[b, a]
            a += 1
        out[b, a] = g[b, a]
        num[b] = a
    return out, num


# --------------------------------------------------------------------------
# stochastic (speculative sampling)
# --------------------------------------------------------------------------

def softmax64(z_bits_row: np.ndarray, temperature: float) -> np.ndarray:
    """softmax(z / T) in fp64 for bf16 logits (T taken as the fp32 value passed)."""
    z = bf16_to_f32(z_bits_row).astype(np.float64) / float(np.float32(temperature))
    e = np.exp(z - np.max(z))
    return e / np.sum(e)


def softmax_normalizer(z_bits: np.ndarray, temperature: float):
    """The two numbers the first pass of speculative sampling needs per logit
    row (the softmax of section 3.1's acceptance rule, p = softmax(z / T)):
    the largest logit zmax and Z = sum_v exp((z_v - zmax) / T), so that
    p_v = exp((z_v - zmax) / T) / Z.  fp64, rows along the last axis; T is
    taken as the fp32 value passed.  Returns (zmax [...], Z [...])."""
    z = bf16_to_f32(z_bits).astype(np.float64)
    zmax = np.max(z, axis=-1)
    Z = np.sum(np.exp((z - zmax[..., None]) / float(np.float32(temperature))), axis=-1)
    return zmax, Z


def _residual(p, q, x, V):
    """r = max(0, p - q); with q None (one-hot at x) that is p with r[x] = 0."""
    if q is None:
        r = np.array(p, copy=True)
        if 0 <= x < V:
            r[x] = 0
        return r
    return np.maximum(p - q, 0)


def _inverse_cdf(r, u, margins=None):
    """Smallest v with cumsum(r)[v] > u * R; None if R is not positive."""
    cum = np.cumsum(r)
    R = cum[-1]
    if not R > 0:
        return None
    t = u * R
    v = int(np.searchsorted(cum, t, side="right"))
    if v >= len(r):
        nz = np.nonzero(np.asarray([ri > 0 for ri in r]))[0]
        v = int(nz[-1])
        if margins is not None:
            margins.append(0.0)
        return v
    if margins is not None:
        lo = cum[v - 1] if v > 0 else 0
        margins.append(float(min(cum[v] - t, t - lo) / R))
    return v


def accept_chain(p, q, x, u, margins=None):
    """Decide one sequence.

    p: k+1 target probability vectors; q: k draft probability vectors or None
    (one-hot drafts); x: k draft ids; u: k+1 uniforms.
    Returns (emitted tokens list, number of accepted drafts).
    If `margins` is a list, the relative distance of every decision to its
    boundary is appended to it (|u q - p| / p for accept tests; distance of
    u R to the nearest cumulative boundary over R for samples).
    """
    k = len(x)
    V = len(p[0])
    out = []
    for i in range(k):
        xi = int(x[i])
        valid = 0 <= xi < V
        px = p[i][xi] if valid else 0
        qx = (q[i][xi] if q is not None else 1) if valid else 0
        if margins is not None:
            margins.append(float(abs(u[i] * qx - px) / px) if px > 0 else float("inf"))
        if u[i] * qx < px:
            out.append(xi)
            continue
        r = _residual(p[i], None if q is None else q[i], xi, V)
        v = _inverse_cdf(r, u[k], margins)
        if v is None:
            v = _inverse_cdf(p[i], u[k], margins)
        out.append(v)
        return out, i
    out.append(_inverse_cdf(p[k], u[k], margins))
    return out, k


def accept_stochastic(zt_bits, zd_bits, draft_tokens, uniforms, temperature,
                      return_margins: bool = False):
    """Speculative-sampling verification over bf16 logits.

    zt_bits [B,k+1,V], zd_bits [B,k,V] or None, draft_tokens [B,k],
    uniforms [B,k+1] fp32, temperature > 0.
    Returns (out_tokens [B,k+1] int32, num_accepted [B] int32[, min_margin [B]]).
    """
    zt_bits = np.asarray(zt_bits)
    B, k1, V = zt_bits.shape
    k = k1 - 1
    x = np.asarray(draft_tokens, dtype=np.int64).reshape(B, k)
    u = np.asarray(uniforms, dtype=np.float32).reshape(B, k1).astype(np.float64)
    out = np.full((B, k1), -1, dtype=np.int32)
    num = np.zeros(B, dtype=np.int32)
    min_margin = np.full(B, np.inf)
    for b in range(B):
        p = [softmax64(zt_bits[b, i], temperature) for i in range(k1)]
        q = None if zd_bits is None else [softmax64(zd_bits[b, i], temperature) for i in range(k)]
        mg = [] if return_margins else None
        toks, a = accept_chain(p, q, x[b], u[b], mg)
        out[b, :len(toks)] = toks
        num[b] = a
        if mg:
            min_margin[b] = min(mg)
    if return_margins:
        return out, num, min_margin
    return out, num


def accept_probabilities(zt_bits, zd_bits, draft_tokens, temperature):
    """p_i(x_i) and q_i(x_i) in fp64 for every drafted position -> ([B,k], [B,k])."""
    zt_bits = np.asarray(zt_bits)
    B, k1, V = zt_bits.shape
    k = k1 - 1
    x = np.asarray(draft_tokens, dtype=np.int64).reshape(B, k)
    px = np.zeros((B, k))
    qx = np.zeros((B, k))
    for b in range(B):
        for i in range(k):
            if 0 <= x[b, i] < V:
                px[b, i] = softmax64(zt_bits[b, i], temperature)[x[b, i]]
                qx[b, i] = 1.0 if zd_bits is None else softmax64(zd_bits[b, i], temperature)[x[b, i]]
    return px, qx


def expected_accepted(p, q):
    """Closed form E[a] = sum_{j=1..k} prod_{i<j} beta_i, beta_i = sum_v min(p_i, q_i).

    For drafts drawn independently from q_i at each position, draft i is
    accepted with probability beta_i = sum_x q_i(x) min(1, p_i(x)/q_i(x)).
    Works on floats or Fractions.
    """
    k = len(q)
    total = 0
    prod = 1
    for j in range(k):
        beta = sum(min(a, b) for a, b in zip(p[j], q[j]))
        prod = prod * beta
        total = total + prod
    return total
