"""GPU parity of the LM-head verify GEMM with the acceptance statistics in its
epilogue (spec_fp8_gemm_logit_stats) and of the acceptance that consumes
those statistics (spec_verify_accept_stats).

The LM head maps the final hidden states of the M = B*(k+1) verify rows to
V logits (section 3.1: the target scores every drafted position in one
pass; V = 128256 and hidden size 4096 of the Llama-3.1-8B-shaped target).
Three legs, so that no oracle input comes from the device:
  A. seeded hidden states and LM-head weights -> the oracle quantizes them
     (the device's codes must match bit for bit), forms the exact GEMM and
     rounds it to bf16; the device's logits match to the GEMM tolerance, and
     its merged statistics match the oracle's softmax normalizer / argmax of
     the oracle's logits within what the measured logit difference allows (a
     logit sits one bf16 step away where the fp32 sum lands next to a
     rounding boundary).
     The statistics must also describe the device's own stored logits
     exactly (max) or to fp32 rounding (sums).
  B. seeded synthetic logits (the C4 generator) and statistics the test
     forms in the documented grouped layout -> spec_verify_accept_stats
     equals the oracle's acceptance on every clear sequence.
  C. the full-size LM head (M=320, K=4096, V=128256): sampled logits against
     the oracle GEMM, statistics against the device's logits, and the fused
     acceptance equal to spec_verify_accept on the same logits.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import accept as oa, gemm as og, quantize as oq
from tests.accept_checks import check_chain
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, host, host_bf16_bits, need_gpu, say

pytestmark = pytest.mark.gpu

TOL = 2e-3
MARGIN = 4e-6
INT_MAX = 0x7FFFFFFF


def c2_of(T):
    """The library's base-2 factor log2(e)/T, rounded once to fp32."""
    return np.float32(1.4426950408889634 / float(np.float32(T)))


def merge_softmax(st):
    """Per-row (max_c Mc, sum_c Zc 2^(Mc - max)) of [M, G, 2] statistics, fp64."""
    m = st[..., 0].astype(np.float64)
    z = st[..., 1].astype(np.float64)
    M = m.max(axis=1)
    w = np.where(np.isfinite(m), z * np.exp2(np.where(np.isfinite(m), m, 0.0) - M[:, None]), 0.0)
    return M, w.sum(axis=1)


def merge_argmax(st):
    v = st[..., 0]
    i = np.ascontiguousarray(st[..., 1]).view(np.int32)
    best = v.max(axis=1)
    idx = np.where(v == best[:, None], i, INT_MAX).min(axis=1)
    return best, idx


def _lm_operands(p, M, V, K, seed, w_std):
    xb = wl.linear_activations(M, K, seed, 0.005, 30.0)
    wb = wl.linear_weights(V, K, seed + 1, w_std)
    a, sa = p.quantize(dev_bf16(xb))
    w, sw = p.quantize(dev_bf16(wb))
    return xb, wb, a, sa, w, sw


@pytest.mark.parametrize("M,V,K,T", [
    (8, 256, 512, 0.7),             # C1-sized
    (80, 1000, 1024, 0.7),          # 80-row tile, ragged last column tile
    (320, 13000, 512, 0.7),         # wide V: 160x192 tiles with a ragged last tile
    (333, 4104, 256, 1.3),          # M past 320, ragged M and V
    (200, 1024, 4096, 0.7),         # long K: 160x128 tiles (never split here)
    (320, 6144, 1024, 0.0),         # greedy statistics
    (100, 4096, 512, 0.0),
    (300, 32008, 256, 0.7),         # 160x384 tiles (fewer operand rows per CU than 160x224): ragged M,
    (300, 32008, 256, 0.0),         #   a last tile of 136 columns (its second wave's column group empty)
])
def test_logit_stats_vs_oracle(M, V, K, T):
    p = need_gpu()
    say(f"logit stats M={M} V={V} K={K} T={T}")
    xb, wb, a, sa, w, sw = _lm_operands(p, M, V, K, seed=M + V + K, w_std=0.1)
    logits, stats = p.gemm_logit_stats(a, sa, w, sw, T)
    G = p.logit_stats_count(M, V, K)
    assert tuple(stats.shape) == (M, G, 2)
    z = host_bf16_bits(logits)                     # [M, V]
    st = host(stats)

    # oracle: its own codes (the device's must match), exact GEMM, bf16 rounding
    qa, sa_ref = oq.quantize_rows(xb)
    qw, sw_ref = oq.quantize_rows(wb)
    np.testing.assert_array_equal(host(a), qa)
    np.testing.assert_array_equal(host(w), qw)
    y_ref = og.gemm(qa, sa_ref, qw, sw_ref)
    z_ref = oq.f64_to_bf16(y_ref)
    zf, zf_ref = oq.bf16_to_f32(z).astype(np.float64), oq.bf16_to_f32(z_ref).astype(np.float64)
    scale = np.max(np.abs(y_ref), axis=1, keepdims=True)
    assert np.all(np.abs(zf - y_ref) <= TOL * scale + 2.0 ** -8 * np.abs(y_ref))
    # Where the device's fp32 sum lands next to a bf16 rounding boundary its
    # logit is one bf16 step from the oracle's; dz bounds the row's shift, and
    # every quantity below moves by at most what that shift allows.
    dz = np.max(np.abs(zf - zf_ref), axis=1)

    if T > 0:
        c2 = c2_of(T)
        Mg, Zg = merge_softmax(st)
        # against the device's own logits: the max exactly, the sum to fp32 rounding
        zmax_dev, Z_dev = oa.softmax_normalizer(z, T)
        np.testing.assert_array_equal(Mg.astype(np.float32), (zmax_dev * np.float64(c2)).astype(np.float32))
        np.testing.assert_allclose(Zg, Z_dev, rtol=2e-5)
        # against the oracle's logits: shifting every logit by at most dz moves
        # the max by dz and ln Z by at most 2 dz / T
        zmax_ref, Z_ref = oa.softmax_normalizer(z_ref, T)
        assert np.all(np.abs(Mg / np.float64(c2) - zmax_ref) <= dz + 1e-6 * np.abs(zmax_ref))
        assert np.all(np.abs(np.log(Zg) - np.log(Z_ref)) <= 2 * dz / float(np.float32(T)) + 2e-5)
    else:
        best, idx = merge_argmax(st)
        np.testing.assert_array_equal(idx, np.argmax(zf, axis=1))             # the device's logits, exactly
        np.testing.assert_array_equal(best, zf.max(axis=1).astype(np.float32))
        # the oracle's: the chosen logit is within 2 dz of the oracle's max
        rows = np.arange(M)
        assert np.all(zf_ref.max(axis=1) - zf_ref[rows, idx] <= 2 * dz)


def _grouped_stats(zbits, T, G):
    """Statistics of logit rows [R, V] in the layout spec_fp8_gemm_logit_stats
    documents, over G contiguous column groups (the last ones may be empty),
    formed here in fp64 and rounded to fp32 (test input; the oracle itself
    works on the logits)."""
    R, V = zbits.shape
    z = oq.bf16_to_f32(zbits).astype(np.float64)
    bounds = np.linspace(0, V, G + 1).astype(np.int64)
    if G >= 2:
        bounds[-2:] = V                                            # one empty trailing group
    st = np.zeros((R, G, 2), np.float32)
    for c in range(G):
        lo, hi = bounds[c], bounds[c + 1]
        if hi <= lo:
            st[:, c, 0] = -np.inf
            st[:, c, 1] = 0.0 if T > 0 else np.array([INT_MAX], np.int32).view(np.float32)[0]
            continue
        blk = z[:, lo:hi]
        if T > 0:
            c2 = np.float64(c2_of(T))
            Mc = (blk.max(axis=1) * c2).astype(np.float32).astype(np.float64)
            st[:, c, 0] = Mc
            st[:, c, 1] = np.exp2(blk * c2 - Mc[:, None]).sum(axis=1)
        else:
            st[:, c, 0] = blk.max(axis=1)
            st[:, c, 1] = (lo + np.argmax(blk, axis=1)).astype(np.int32).view(np.float32)
    return st


@pytest.mark.parametrize("B,k,V,seed,c,with_draft,T,G", [
    (16, 4, 5000, 1, 0.95, True, 0.7, 27),
    (9, 3, 1001, 2, 0.9, True, 0.7, 5),           # V not a multiple of 8
    (16, 4, 20000, 3, 0.99, False, 0.7, 200),     # one-hot drafts: no statistics kernel runs
    (8, 8, 3000, 4, 0.0, True, 0.7, 1),           # uncorrelated, one group per row
    (12, 4, 9000, 5, 0.9, True, 0.0, 40),         # greedy from statistics
    (12, 4, 9000, 6, 0.9, False, 0.0, 3),
])
def test_accept_from_stats_vs_oracle(B, k, V, seed, c, with_draft, T, G):
    p = need_gpu()
    say(f"accept from stats B={B} k={k} V={V} draft_logits={with_draft} T={T} G={G}")
    zt, zd = wl.accept_logits(B, k, V, seed, c, scale=2.0)
    if T > 0:
        x = wl.draft_tokens_sampled(zd, T, seed=seed + 1)
    else:
        x = wl.draft_tokens_greedy(zd)
    x[0, 0] = V + 3                                    # an out-of-range draft is a rejection
    u = wl.philox_uniforms((B, k + 1), seed=seed + 2)
    st = _grouped_stats(zt.reshape(B * (k + 1), V), T, G)
    zd_in = zd if with_draft else None
    out, num = p.verify_accept(dev_bf16(zt), None if zd_in is None else dev_bf16(zd_in), dev_i32(x),
                               dev_f32(u) if T > 0 else None, T, target_stats=dev_f32(st))
    out, num = host(out), host(num)
    if T == 0:
        out_ref, num_ref = oa.accept_greedy(zt, x)
        np.testing.assert_array_equal(num, num_ref)
        np.testing.assert_array_equal(out, out_ref)
        return
    out_ref, num_ref, mg = oa.accept_stochastic(zt, zd_in, x, u, T, return_margins=True)
    clear = mg > MARGIN
    assert clear.mean() >= 0.85
    np.testing.assert_array_equal(num[clear], num_ref[clear])
    np.testing.assert_array_equal(out[clear], out_ref[clear])
    check_chain(out, num, zt, zd_in, x, u, T)


def test_lm_head_full_size():
    """The verify step's LM head at full size: M = 64*(4+1) = 320 rows, K = 4096,
    V = 128256, in the launch configuration the bench times."""
    p = need_gpu()
    B, k = wl.CONFIGS["C4"]["B"], wl.CONFIGS["C4"]["k"]
    V, K, T = wl.CONFIGS["C4"]["V"], 4096, 0.7
    M = B * (k + 1)
    seed = 41
    say(f"LM head M={M} K={K} V={V}: weights")
    wb = wl.linear_weights(V, K, seed + 1, 0.05)
    w, sw = p.quantize(dev_bf16(wb))
    say("LM head: hidden states")
    xt = wl.linear_activations(M, K, seed, 0.005, 30.0)
    # draft rows: the drafter's hidden states track the target's (EAGLE reuses the target's LM head)
    xt_f = oq.bf16_to_f32(xt).reshape(B, k + 1, K)
    noise = np.random.default_rng(seed + 2).standard_normal((B, k, K)).astype(np.float32)
    xd = wl.bf16_bits_from_f32((xt_f[:, :k] + 0.5 * noise).reshape(B * k, K))
    a_t, sa_t = p.quantize(dev_bf16(xt))
    a_d, sa_d = p.quantize(dev_bf16(xd))

    logits, stats = p.gemm_logit_stats(a_t, sa_t, w, sw, T)
    plain = p.gemm(a_t, sa_t, w, sw)
    assert p.gemm_workspace_bytes(M, V, K) == 0        # no K split; both GEMMs walk K in order: identical bits
    assert torch.equal(logits.contiguous().view(torch.int16), plain.contiguous().view(torch.int16))
    zd = p.gemm(a_d, sa_d, w, sw)

    # sampled logits against the oracle GEMM on the oracle's own codes
    rng = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([[0, M - 1], rng.choice(M, 4, replace=False)]))
    cols = np.unique(np.concatenate([[0, V - 1], rng.choice(V, 2048, replace=False)]))
    qa, sa_ref = oq.quantize_rows(xt[rows])
    qw, sw_ref = oq.quantize_rows(wb[cols])
    np.testing.assert_array_equal(host(a_t)[rows], qa)
    np.testing.assert_array_equal(host(w)[cols], qw)
    y_ref = og.gemm(qa, sa_ref, qw, sw_ref)
    z = host_bf16_bits(logits)
    zs = oq.bf16_to_f32(z[np.ix_(rows, cols)]).astype(np.float64)
    assert np.all(np.abs(zs - y_ref) <= TOL * np.max(np.abs(y_ref), axis=1, keepdims=True) + 2.0 ** -8 * np.abs(y_ref))

    # the statistics describe the stored logits
    Mg, Zg = merge_softmax(host(stats))
    zmax, Zs = oa.softmax_normalizer(z, T)
    np.testing.assert_array_equal(Mg.astype(np.float32), (zmax * np.float64(c2_of(T))).astype(np.float32))
    np.testing.assert_allclose(Zg, Zs, rtol=2e-5)

    # fused acceptance = acceptance that reads the logits for its statistics
    zt3 = logits.contiguous().view(B, k + 1, V)
    zd3 = zd.contiguous().view(B, k, V)
    zd_bits = host_bf16_bits(zd3)
    x = wl.draft_tokens_sampled(zd_bits, T, seed=seed + 3)
    u = wl.philox_uniforms((B, k + 1), seed=seed + 4)
    out_f, num_f = p.verify_accept(zt3, zd3, dev_i32(x), dev_f32(u), T, target_stats=stats)
    out_p, num_p = p.verify_accept(zt3, zd3, dev_i32(x), dev_f32(u), T)
    out_f, num_f, out_p, num_p = host(out_f), host(num_f), host(out_p), host(num_p)
    same = np.all(out_f == out_p, axis=1) & (num_f == num_p)
    say(f"LM head: MGL {np.mean(num_f + 1):.3f}; fused == unfused on {int(same.sum())} of {B} sequences")
    assert same.mean() >= 0.95
    # both results, every sequence: fp64 decisions outside 1e-6 of their
    # boundary, samples at their inverse-CDF positions (the logits are the
    # stored bf16 values both acceptances read)
    zt_bits = host_bf16_bits(zt3)
    check_chain(out_f, num_f, zt_bits, zd_bits, x, u, T)
    check_chain(out_p, num_p, zt_bits, zd_bits, x, u, T)
    # greedy from the epilogue's argmax statistics
    lg, sg = p.gemm_logit_stats(a_t, sa_t, w, sw, 0.0)
    xg = np.argmax(oq.bf16_to_f32(zd_bits), axis=-1).astype(np.int32)
    og_, ng = p.verify_accept(lg.contiguous().view(B, k + 1, V), None, dev_i32(xg), None, 0.0, target_stats=sg)
    og2, ng2 = p.verify_accept(lg.contiguous().view(B, k + 1, V), None, dev_i32(xg), None, 0.0)
    np.testing.assert_array_equal(host(og_), host(og2))
    np.testing.assert_array_equal(host(ng), host(ng2))
