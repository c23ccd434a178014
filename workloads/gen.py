"""Seeded generators for every synthetic input of the verify path.

All generators use numpy's counter-based Philox bit generator, so a given
(seed, shape) always yields the same array on any machine.  Floating-point
inputs are drawn in fp32 and stored as bf16 bit patterns (uint16), rounded to
nearest-even, which is the activation/logit dtype of the served model.
"""

from __future__ import annotations

import math

import numpy as np


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(int(seed)))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even; NaN -> 0x7FC0."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def _outlier_columns(K: int, frac: float, seed: int) -> np.ndarray:
    n_out = int(round(frac * K))
    perm = _rng(seed + 0x5EED).permutation(K)
    return np.sort(perm[:n_out])


def linear_activations(M: int, K: int, seed: int, outlier_frac: float = 0.0,
                       outlier_scale: float = 1.0) -> np.ndarray:
    """Activations X ~ N(0,1) [M,K] with a fixed set of outlier channels.

    The outlier channels are the first round(outlier_frac*K) indices of a
    seeded permutation of the K channels; those columns are multiplied by
    outlier_scale (the per-channel outliers typical of LLM activations).
    Returns bf16 bits [M,K].
    """
    x = _rng(seed).standard_normal((M, K), dtype=np.float32)
    if outlier_frac > 0.0:
        cols = _outlier_columns(K, outlier_frac, seed)
        x[:, cols] *= np.float32(outlier_scale)
    return bf16_bits_from_f32(x)


def linear_weights(N: int, K: int, seed: int, std: float = 0.02) -> np.ndarray:
    """Weights W ~ N(0, std^2) in nn.Linear layout [N,K] (row = output channel)."""
    w = _rng(seed).standard_normal((N, K), dtype=np.float32)
    w *= np.float32(std)
    return bf16_bits_from_f32(w)


def fp8_code_bytes(rows: int, cols: int, seed: int) -> np.ndarray:
    """Random E4M3 code bytes [rows, cols] (uint8): every byte pattern except
    the two NaN patterns 0x7F and 0xFF, equally likely.  Operands for GEMM
    tests that span the whole format without a quantizer in between."""
    c = _rng(seed).integers(0, 254, size=(rows, cols), dtype=np.uint16)
    return (c + (c >= 0x7F)).astype(np.uint8)          # 0..126 -> 0x00..0x7E, 127..253 -> 0x80..0xFE


def uniform_scales(n: int, seed: int, lo: float = 1e-3, hi: float = 2e-3) -> np.ndarray:
    """n fp32 scales drawn uniformly from [lo, hi)."""
    return _rng(seed).uniform(lo, hi, size=n).astype(np.float32)


def student_t_activations(M: int, K: int, seed: int, df: float = 3.0) -> np.ndarray:
    """Heavy-tailed activations ~ Student-t(df) [M,K] as bf16 bits."""
    x = _rng(seed).standard_t(df, size=(M, K)).astype(np.float32)
    return bf16_bits_from_f32(x)


def gated_ffn_input(M: int, inter: int, seed: int, std: float = 1.0) -> np.ndarray:
    """Fused gate|up projection output [M, 2*inter] as bf16 bits.

    Columns [0, inter) are the gate, [inter, 2*inter) the up projection.
    """
    g = _rng(seed).standard_normal((M, 2 * inter), dtype=np.float32)
    g *= np.float32(std)
    return bf16_bits_from_f32(g)


def accept_logits(B: int, k: int, V: int, seed: int, c: float,
                  scale: float = 3.0, rank: int = 8):
    """Target and draft logits with a shared low-rank component.

    S = (A @ Bm) / sqrt(rank), A ~ N(0,1) [B,k+1,rank], Bm ~ N(0,1) [rank,V].
    z_t = scale*(c*S + sqrt(1-c^2)*E_t)             [B,k+1,V]
    z_d = scale*(c*S[:, :k] + sqrt(1-c^2)*E_d)      [B,k,V]
    so each position has marginal N(0, scale^2) logits and the draft/target
    logits at a position are correlated with coefficient c^2.
    Returns (z_t bits, z_d bits) as bf16 uint16 arrays.
    """
    if not (0.0 <= c <= 1.0):
        raise ValueError("c must lie in [0, 1]")
    g = _rng(seed)
    a = g.standard_normal((B, k + 1, rank), dtype=np.float32)
    bm = g.standard_normal((rank, V), dtype=np.float32)
    s = (a.reshape(-1, rank) @ bm).reshape(B, k + 1, V)
    s *= np.float32(1.0 / math.sqrt(rank))
    cc = np.float32(c)
    nn = np.float32(math.sqrt(max(0.0, 1.0 - c * c)))
    sc = np.float32(scale)
    zt = g.standard_normal((B, k + 1, V), dtype=np.float32)
    zt *= nn
    zt += cc * s
    zt *= sc
    zt_bits = bf16_bits_from_f32(zt)
    del zt
    zd = g.standard_normal((B, k, V), dtype=np.float32)
    zd *= nn
    zd += cc * s[:, :k]
    zd *= sc
    zd_bits = bf16_bits_from_f32(zd)
    return zt_bits, zd_bits


def draft_tokens_greedy(zd_bits: np.ndarray) -> np.ndarray:
    """Argmax drafting (a greedy chain): x_i = argmax_v z_d[b,i,v], lowest index on ties."""
    zd = f32_from_bf16_bits(zd_bits)
    return np.argmax(zd, axis=-1).astype(np.int32)


def draft_tokens_sampled(zd_bits: np.ndarray, temperature: float, seed: int = 8) -> np.ndarray:
    """Drafts drawn from softmax(z_d / T) with the Gumbel-max construction.

    x_i = argmax_v (z_d[b,i,v]/T + G_v) with G_v iid standard Gumbel; this
    draws x_i from the draft's tempered distribution without normalising it.
    """
    if temperature <= 0:
        return draft_tokens_greedy(zd_bits)
    zd = f32_from_bf16_bits(zd_bits).astype(np.float64) / float(temperature)
    u = _rng(seed).random(zd.shape)
    # Gumbel(0,1) = -log(-log U); U=0 has probability ~2^-53 and is nudged.
    u = np.clip(u, np.finfo(np.float64).tiny, 1.0)
    zd += -np.log(-np.log(u))
    return np.argmax(zd, axis=-1).astype(np.int32)


def philox_uniforms(shape, seed: int = 7) -> np.ndarray:
    """Uniforms in [0,1) as fp32 from Philox(seed)."""
    return _rng(seed).random(shape, dtype=np.float32)


def tree_shape(N: int, branching) -> np.ndarray:
    """Parents [N] of a breadth-first token tree: a node at depth d gets
    branching[d] children (the last entry repeats) until N nodes exist; -1 is
    the root (the last accepted token)."""
    parent = []
    frontier = [(-1, 0)]
    while frontier and len(parent) < N:
        nxt = []
        for p, d in frontier:
            k = branching[min(d, len(branching) - 1)]
            for _ in range(k):
                if len(parent) == N:
                    break
                parent.append(p)
                nxt.append((len(parent) - 1, d + 1))
        frontier = nxt
    return np.asarray(parent, dtype=np.int32)


def tree_tokens_topk(zd_bits: np.ndarray, parent: np.ndarray) -> np.ndarray:
    """Candidate tokens of a top-k tree expansion: the children of node p (in
    index order) are k highest-scoring tokens of draft row p+1 (which of
    several equal scores at the k-th place is taken is unspecified), in
    decreasing order of score, equal scores by lowest index.  zd_bits
    [B, N, V]; returns int32 [B, N]."""
    zd = f32_from_bf16_bits(zd_bits)
    B, N = zd.shape[0], len(parent)
    x = np.zeros((B, N), dtype=np.int32)
    for p in range(-1, N):
        kids = [n for n in range(N) if parent[n] == p]
        if not kids:
            continue
        row = zd[:, p + 1]
        k = len(kids)
        top = np.argpartition(-row, k - 1, axis=-1)[:, :k] if k < row.shape[-1] else \
            np.broadcast_to(np.arange(row.shape[-1]), row.shape)[:, :k]
        # the k selected tokens by decreasing score, ties by lowest index
        val = np.take_along_axis(row, top, axis=-1)
        order = np.lexsort((top, -val), axis=-1)
        x[:, kids] = np.take_along_axis(top, order, axis=-1)
    return x


def paged_slot_mapping(B: int, new_tokens: int, ctx_lens, block_size: int, seed: int):
    """Cache slots of the verify step's new tokens in a paged KV cache.

    Sequence b already holds ctx_lens[b] tokens; its new_tokens tokens take
    positions ctx_lens[b] .. ctx_lens[b] + new_tokens - 1.  Every sequence
    owns ceil((ctx_lens[b] + new_tokens) / block_size) blocks, drawn as one
    seeded random permutation of all blocks, and position p of sequence b
    lives in slot page[b][p // block_size] * block_size + p % block_size.
    Returns (slot_mapping int64 [B * new_tokens] in sequence-major token
    order, num_slots)."""
    ctx = np.asarray(ctx_lens, dtype=np.int64)
    need = (ctx + new_tokens + block_size - 1) // block_size
    perm = _rng(seed).permutation(int(need.sum()))
    starts = np.concatenate([[0], np.cumsum(need)[:-1]])
    slots = np.empty(B * new_tokens, dtype=np.int64)
    for b in range(B):
        page = perm[starts[b]:starts[b] + need[b]]
        pos = ctx[b] + np.arange(new_tokens)
        slots[b * new_tokens:(b + 1) * new_tokens] = page[pos // block_size] * block_size + pos % block_size
    return slots, int(need.sum()) * block_size


def calibration_sets(L: int, K: int, seed: int, public_outlier_frac: float, public_outlier_scale: float,
                     indomain_df: float):
    """Calibration pools of L tokens for the calibration study: 'public'
    (Gaussian activations with a few large outlier channels), 'in_domain'
    (heavy-tailed Student-t activations, the test set's law) and 'mixed'
    (the first half of each).  Returns {name: bf16 bits [L, K]}."""
    pub = linear_activations(L, K, seed, public_outlier_frac, public_outlier_scale)
    ind = student_t_activations(L, K, seed + 1, indomain_df)
    h = L // 2
    mix = np.concatenate([pub[:h], ind[:L - h]], axis=0)
    return {"public": pub, "in_domain": ind, "mixed": mix}
