"""GPU parity of spec_verify_accept against the oracle.

Greedy: token ids and accepted counts bit-exact.  Speculative sampling: the
GPU evaluates probabilities in fp32 and the oracle in fp64.  The GPU's
probabilities carry a relative error of about 1e-6 (fp32 exponent argument and
sums; a common normalisation error cancels between u*R and the cumulative
sums), so every sequence whose decisions all lie farther than MARGIN (relative
to p for accept tests, to R for samples) from their boundary must match
exactly.  At V=128256 the sampled token typically carries ~1e-4 of the
mass, so a few sequences of a batch of 64 fall inside the margin; every
sequence, those included, is then replayed in fp64 along the device's own
decisions (tests/accept_checks.py): each accept test must be the fp64
decision unless it lies within 1e-6 of its boundary, and the emitted token
must sit at its inverse-CDF position within 1e-5 of the residual mass.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import accept as oa
from tests.accept_checks import check_chain
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, host, need_gpu, say

pytestmark = pytest.mark.gpu

MARGIN = 4e-6


def _check_valid(out, num, x, V):
    B, k1 = out.shape
    for b in range(B):
        a = num[b]
        assert 0 <= a < k1
        assert np.all(out[b, :a] == x[b, :a])
        assert 0 <= out[b, a] < V
        assert np.all(out[b, a + 1:] == -1)


def _stochastic_case(B, k, V, seed, c, T, with_draft=True, scale=2.0):
    zt, zd = wl.accept_logits(B, k, V, seed, c, scale=scale)
    x = wl.draft_tokens_sampled(zd, T, seed=seed + 1) if with_draft else wl.draft_tokens_greedy(zd)
    u = wl.philox_uniforms((B, k + 1), seed=seed + 2)
    return zt, (zd if with_draft else None), x, u


@pytest.mark.parametrize("B,k,V,seed,c", [
    (2, 3, 256, 0, 0.5),            # C1
    (7, 4, 1000, 1, 0.9),
    (5, 2, 1001, 2, 0.9),           # V not a multiple of 8: scalar path
    (33, 4, 20000, 3, 0.99),        # several vocabulary chunks, ragged last chunk
    (3, 16, 64, 4, 0.7),            # longest chain
    (4, 1, 1, 5, 0.5),              # one-token vocabulary
    (2, 1, 1 << 22, 6, 0.9),        # largest vocabulary (1024 slices, 256 sampling chunks)
])
def test_greedy_bit_exact(B, k, V, seed, c):
    p = need_gpu()
    say(f"greedy B={B} k={k} V={V}")
    zt, zd = wl.accept_logits(B, k, V, seed, c)
    x = wl.draft_tokens_greedy(zd)
    x[0, 0] = V + 5 if B > 1 else x[0, 0]          # an out-of-range draft is a rejection
    out, num = p.verify_accept(dev_bf16(zt), None, dev_i32(x), None, 0.0)
    out_ref, num_ref = oa.accept_greedy(zt, x)
    np.testing.assert_array_equal(host(num), num_ref)
    np.testing.assert_array_equal(host(out), out_ref)


def test_greedy_ties_lowest_index():
    p = need_gpu()
    B, k, V = 4, 2, 9000                            # ties across vocabulary chunks
    z = np.zeros((B, k + 1, V), np.float32)
    z[:, :, [8191, 8192, 100]] = 5.0
    zt = wl.bf16_bits_from_f32(z)
    x = np.full((B, k), 100, np.int32)
    out, num = p.verify_accept(dev_bf16(zt), None, dev_i32(x), None, 0.0)
    out_ref, num_ref = oa.accept_greedy(zt, x)
    np.testing.assert_array_equal(host(out), out_ref)
    assert np.all(host(out)[:, :k] == 100)


@pytest.mark.parametrize("B,k,V,seed,c,with_draft", [
    (2, 3, 256, 0, 0.5, True),     # C1
    (16, 4, 5000, 1, 0.95, True),
    (9, 3, 1001, 2, 0.9, True),    # scalar path
    (16, 4, 20000, 3, 0.99, False),  # one-hot drafts (no draft logits)
    (8, 8, 3000, 4, 0.0, True),    # uncorrelated: many rejections
])
def test_stochastic_parity(B, k, V, seed, c, with_draft):
    p = need_gpu()
    T = 0.7
    say(f"stochastic B={B} k={k} V={V} draft_logits={with_draft}")
    zt, zd, x, u = _stochastic_case(B, k, V, seed, c, T, with_draft)
    out, num = p.verify_accept(dev_bf16(zt), None if zd is None else dev_bf16(zd), dev_i32(x), dev_f32(u), T)
    out, num = host(out), host(num)
    out_ref, num_ref, mg = oa.accept_stochastic(zt, zd, x, u, T, return_margins=True)
    clear = mg > MARGIN
    assert clear.mean() >= 0.9
    np.testing.assert_array_equal(num[clear], num_ref[clear])
    np.testing.assert_array_equal(out[clear], out_ref[clear])
    _check_valid(out, num, x, V)
    check_chain(out, num, zt, zd, x, u, T)


def test_stochastic_many_pairs_and_invalid_drafts():
    """B*k = 333 (sequence, draft) pairs, past one workgroup of the statistics
    kernel's draft-logit gather and not a multiple of its 64 per wave, with
    draft ids out of range in both directions (each is a rejection)."""
    p = need_gpu()
    B, k, V, T = 37, 9, 4000, 0.7
    say(f"stochastic B={B} k={k} V={V} invalid drafts")
    zt, zd, x, u = _stochastic_case(B, k, V, 21, 0.97, T)
    x[3, 0], x[10, 4], x[36, 8] = -1, V + 3, V
    out, num = p.verify_accept(dev_bf16(zt), dev_bf16(zd), dev_i32(x), dev_f32(u), T)
    out, num = host(out), host(num)
    out_ref, num_ref, mg = oa.accept_stochastic(zt, zd, x, u, T, return_margins=True)
    assert num[3] == 0 and num[10] <= 4 and num[36] <= 8
    clear = mg > MARGIN
    assert clear.mean() >= 0.9
    np.testing.assert_array_equal(num[clear], num_ref[clear])
    np.testing.assert_array_equal(out[clear], out_ref[clear])
    _check_valid(out, num, x, V)
    check_chain(out, num, zt, zd, x, u, T)


def test_stochastic_full_vocab_c4():
    """C4 at full size (B=64, k=4, V=128256, T=0.7), greedy and stochastic."""
    p = need_gpu()
    cfg = wl.CONFIGS["C4"]
    B, k, V, T = cfg["B"], cfg["k"], cfg["V"], cfg["temperature"]
    say("C4 logits")
    zt, zd = wl.accept_logits(B, k, V, cfg["seed"], wl.C4_CORRELATION, scale=cfg["logit_std"], rank=cfg["rank"])
    dzt, dzd = dev_bf16(zt), dev_bf16(zd)
    xg = wl.draft_tokens_greedy(zd)
    out, num = p.verify_accept(dzt, None, dev_i32(xg), None, 0.0)
    out_ref, num_ref = oa.accept_greedy(zt, xg)
    np.testing.assert_array_equal(host(out), out_ref)
    np.testing.assert_array_equal(host(num), num_ref)
    say(f"C4 greedy MGL {np.mean(num_ref + 1):.3f}")
    xs = wl.draft_tokens_sampled(zd, T, seed=cfg["draft_seed"])
    u = wl.philox_uniforms((B, k + 1), seed=cfg["uniform_seed"])
    out, num = p.verify_accept(dzt, dzd, dev_i32(xs), dev_f32(u), T)
    out, num = host(out), host(num)
    out_ref, num_ref, mg = oa.accept_stochastic(zt, zd, xs, u, T, return_margins=True)
    clear = mg > MARGIN
    say(f"C4 stochastic MGL {np.mean(num_ref + 1):.3f}, margin events {int((~clear).sum())}")
    assert clear.sum() >= 0.8 * B
    np.testing.assert_array_equal(num[clear], num_ref[clear])
    np.testing.assert_array_equal(out[clear], out_ref[clear])
    _check_valid(out, num, xs, V)
    # every sequence, the margin ones included: the device's accept tests
    # are the fp64 decisions wherever those lie beyond 1e-6 of the boundary,
    # and its sample sits at the inverse-CDF position of u*R
    check_chain(out, num, zt, zd, xs, u, T)


def test_p_equals_q_accepts_all():
    p = need_gpu()
    B, k, V = 32, 4, 3000
    zt, _ = wl.accept_logits(B, k, V, 11, 0.5)
    zd = np.ascontiguousarray(zt[:, :k])
    x = wl.draft_tokens_sampled(zd, 0.7, seed=3)
    u = wl.philox_uniforms((B, k + 1), seed=4)
    out, num = p.verify_accept(dev_bf16(zt), dev_bf16(zd), dev_i32(x), dev_f32(u), 0.7)
    assert np.all(host(num) == k)
    np.testing.assert_array_equal(host(out)[:, :k], x)


def test_emitted_law_matches_target_chi_square():
    """Losslessness on the GPU: with one logit row replicated over many
    sequences, the first emitted token follows p_0 (chi-square, V=64)."""
    p = need_gpu()
    V, k, T = 64, 2, 1.0
    B = 13000
    rng = np.random.default_rng(21)
    zt1 = (rng.standard_normal((1, k + 1, V)) * 1.5).astype(np.float32)
    zd1 = (zt1[:, :k] + rng.standard_normal((1, k, V)).astype(np.float32)).astype(np.float32)
    zt = wl.bf16_bits_from_f32(np.repeat(zt1, B, 0))
    zd = wl.bf16_bits_from_f32(np.repeat(zd1, B, 0))
    p0 = oa.softmax64(zt[0, 0], T)
    counts = np.zeros(V)
    dzt, dzd = dev_bf16(zt), dev_bf16(zd)
    for rep in range(5):
        x = wl.draft_tokens_sampled(zd, T, seed=100 + rep)
        u = wl.philox_uniforms((B, k + 1), seed=200 + rep)
        out, _ = p.verify_accept(dzt, dzd, dev_i32(x), dev_f32(u), T)
        counts += np.bincount(host(out)[:, 0], minlength=V)
    n = counts.sum()
    exp = p0 * n
    keep = exp >= 5
    chi2 = np.sum((counts[keep] - exp[keep]) ** 2 / exp[keep]) + (counts[~keep].sum() - exp[~keep].sum()) ** 2 / max(exp[~keep].sum(), 1e-9)
    dof = keep.sum()
    assert chi2 < dof + 6 * np.sqrt(2 * dof), (chi2, dof)


def test_deterministic():
    p = need_gpu()
    zt, zd, x, u = _stochastic_case(16, 4, 20000, 7, 0.95, 0.7)
    args = (dev_bf16(zt), dev_bf16(zd), dev_i32(x), dev_f32(u), 0.7)
    a = [host(t) for t in p.verify_accept(*args)]
    b = [host(t) for t in p.verify_accept(*args)]
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_vanished_residual_samples_target():
    """p_j == q_j and an out-of-range draft: the rejection's residual is
    identically zero, so the token is drawn from p_j itself (several chunks)."""
    p = need_gpu()
    B, k, V, T = 16, 4, 40000, 0.7
    zt, _ = wl.accept_logits(B, k, V, 12, 0.5)
    zd = np.ascontiguousarray(zt[:, :k])
    x = wl.draft_tokens_sampled(zd, T, seed=5)
    x[0::2, 1] = V + 3                       # rejected at position <= 1, residual 0
    x[1::4, 0] = -2
    u = wl.philox_uniforms((B, k + 1), seed=6)
    out, num = p.verify_accept(dev_bf16(zt), dev_bf16(zd), dev_i32(x), dev_f32(u), T)
    out, num = host(out), host(num)
    out_ref, num_ref, mg = oa.accept_stochastic(zt, zd, x, u, T, return_margins=True)
    np.testing.assert_array_equal(num, num_ref)
    assert np.all(num[0::2] <= 1) and np.all(num[1::4] == 0)
    clear = mg > MARGIN
    assert clear.mean() >= 0.5
    np.testing.assert_array_equal(out[clear], out_ref[clear])
    _check_valid(out, num, x, V)
    check_chain(out, num, zt, zd, x, u, T)


def test_extreme_uniforms():
    """u = 0 draws the first token of positive residual mass (exactly); u just
    below 1 draws at the top of the CDF (ragged last chunk, scalar path too)."""
    p = need_gpu()
    T = 0.7
    for V in (20000, 20001):
        B, k = 8, 3
        zt, zd = wl.accept_logits(B, k, V, 13, 0.3)
        x = wl.draft_tokens_sampled(zd, T, seed=7)
        u = wl.philox_uniforms((B, k + 1), seed=8)
        u[:, 0] = 1.0 - 2.0 ** -24            # reject position 0 whenever p < q there
        u[0::2, k] = 0.0
        u[1::2, k] = np.float32(1.0 - 2.0 ** -24)
        out, num = p.verify_accept(dev_bf16(zt), dev_bf16(zd), dev_i32(x), dev_f32(u), T)
        out, num = host(out), host(num)
        out_ref, num_ref = oa.accept_stochastic(zt, zd, x, u, T)
        np.testing.assert_array_equal(num, num_ref)
        np.testing.assert_array_equal(out[0::2], out_ref[0::2])
        _check_valid(out, num, x, V)
        check_chain(out, num, zt, zd, x, u, T)


def test_stochastic_largest_vocabulary():
    """V = 2^22 (256 sampling chunks): accept decisions match, and every sample
    sits at its inverse-CDF position within the fp32 error."""
    p = need_gpu()
    B, k, V, T = 2, 2, 1 << 22, 0.7
    say("stochastic V=2^22")
    zt, zd = wl.accept_logits(B, k, V, 14, 0.9)
    x = wl.draft_tokens_sampled(zd, T, seed=9)
    u = wl.philox_uniforms((B, k + 1), seed=10)
    out, num = p.verify_accept(dev_bf16(zt), dev_bf16(zd), dev_i32(x), dev_f32(u), T)
    out, num = host(out), host(num)
    px, qx = oa.accept_probabilities(zt, zd, x, T)
    for b in range(B):                       # decisions are far from their boundaries here
        acc = [float(u[b, i]) * qx[b, i] < px[b, i] for i in range(k)]
        assert num[b] == (acc.index(False) if False in acc else k)
    _check_valid(out, num, x, V)
    check_chain(out, num, zt, zd, x, u, T)


def test_million_trials_law_and_mean_acceptance():
    """One target/draft logit set replicated over 9000 sequences (B (2k+1) <=
    65535), 112 rounds of fresh drafts (sampled from q) and uniforms: about
    10^6 verify trials at V = 256.  The first emitted token follows p_0 (chi-square), and the mean
    number of accepted drafts matches the closed form
    E[a] = sum_j prod_{i<j} beta_i, beta_i = sum_v min(p_i, q_i)
    (within 6 standard errors)."""
    p = need_gpu()
    V, k, T, B, R = 256, 3, 1.0, 9000, 112
    rng = np.random.default_rng(33)
    zt1 = (rng.standard_normal((1, k + 1, V)) * 1.5).astype(np.float32)
    zd1 = (zt1[:, :k] + 0.7 * rng.standard_normal((1, k, V))).astype(np.float32)
    zt = wl.bf16_bits_from_f32(np.repeat(zt1, B, 0))
    zd = wl.bf16_bits_from_f32(np.repeat(zd1, B, 0))
    pp = [oa.softmax64(zt[0, i], T) for i in range(k + 1)]
    qq = [oa.softmax64(zd[0, i], T) for i in range(k)]
    e_a = oa.expected_accepted(pp[:k], qq)
    dzt, dzd = dev_bf16(zt), dev_bf16(zd)
    counts = np.zeros(V)
    acc = []
    for rep in range(R):
        if rep % 16 == 0:
            say(f"round {rep}")
        x = wl.draft_tokens_sampled(zd, T, seed=1000 + rep)
        u = wl.philox_uniforms((B, k + 1), seed=2000 + rep)
        out, num = p.verify_accept(dzt, dzd, dev_i32(x), dev_f32(u), T)
        counts += np.bincount(host(out)[:, 0], minlength=V)
        acc.append(host(num).astype(np.float64))
    n = counts.sum()
    assert n == B * R
    exp = pp[0] * n
    keep = exp >= 5
    chi2 = np.sum((counts[keep] - exp[keep]) ** 2 / exp[keep]) + \
        (counts[~keep].sum() - exp[~keep].sum()) ** 2 / max(exp[~keep].sum(), 1e-9)
    dof = keep.sum()
    assert chi2 < dof + 6 * np.sqrt(2 * dof), (chi2, dof)
    a = np.concatenate(acc)
    se = a.std() / np.sqrt(a.size)
    say(f"mean accepted {a.mean():.5f}, closed form {e_a:.5f}, standard error {se:.2e}; chi2 {chi2:.1f} (dof {dof})")
    assert abs(a.mean() - e_a) < 6 * se + 1e-6
