"""Pins of the oracle's acceptance rule: planted greedy chains, exact enumeration of
the speculative-sampling law, reductions to greedy, closed-form acceptance length."""

import itertools
from fractions import Fraction

import numpy as np
import pytest

import workloads as wl
from oracle import accept as oa
from oracle import enumerate as oe


def _bits(x):
    return wl.bf16_bits_from_f32(np.asarray(x, np.float32))


# ---------------------------------------------------------------- greedy

def test_greedy_planted_chain():
    rng = np.random.default_rng(0)
    B, k, V = 6, 4, 50
    z = rng.standard_normal((B, k + 1, V)).astype(np.float32)
    g = rng.integers(0, V, (B, k + 1))
    z[np.arange(B)[:, None], np.arange(k + 1)[None, :], g] = 10.0
    acc_len = [0, 1, 2, 3, 4, 2]
    x = g[:, :k].copy()
    for b, a in enumerate(acc_len):
        if a < k:
            x[b, a] = (g[b, a] + 1) % V
    out, num = oa.accept_greedy(_bits(z), x)
    for b, a in enumerate(acc_len):
        assert num[b] == a
        assert list(out[b, :a + 1]) == list(g[b, :a]) + [g[b, a]]
        assert np.all(out[b, a + 1:] == -1)


def test_greedy_ties_take_lowest_index():
    z = np.zeros((1, 2, 8), np.float32)
    z[0, 0, [5, 2, 7]] = 3.0
    z[0, 1, [6, 1]] = 4.0
    out, num = oa.accept_greedy(_bits(z), np.array([[2]]))
    assert num[0] == 1 and list(out[0]) == [2, 1]
    out, num = oa.accept_greedy(_bits(z), np.array([[5]]))
    assert num[0] == 0 and list(out[0]) == [2, -1]


def test_greedy_invalid_draft_rejected():
    z = np.zeros((1, 2, 4), np.float32)
    z[0, 0, 3] = 1.0
    out, num = oa.accept_greedy(_bits(z), np.array([[99]]))
    assert num[0] == 0 and out[0, 0] == 3


# ---------------------------------------------------------------- stochastic

def _rand_dist(rng, V, lo=0):
    w = rng.integers(lo, 6, V)
    if w.sum() == 0:
        w[rng.integers(V)] = 1
    return [Fraction(int(t), int(w.sum())) for t in w]


@pytest.mark.parametrize("V,k,seed,lo", [(3, 1, 0, 0), (4, 2, 1, 0), (3, 3, 2, 1), (5, 2, 3, 0),
                                         (4, 3, 4, 1), (5, 3, 5, 0)])
def test_enumerated_law_equals_target(V, k, seed, lo):
    """Speculative sampling is lossless: given any emitted prefix, the next token ~ p."""
    rng = np.random.default_rng(seed)
    p = [_rand_dist(rng, V, lo) for _ in range(k + 1)]
    q = [_rand_dist(rng, V, lo) for _ in range(k)]
    law = oe.emitted_law(p, q)
    assert sum(law.values()) == 1
    beta = [sum(min(a, b) for a, b in zip(p[i], q[i])) for i in range(k)]
    for n in range(k + 1):
        prefixes = {seq[:n] for seq in law if len(seq) > n}
        reach = sum(pr for seq, pr in law.items() if len(seq) > n)
        expect = Fraction(1)
        for i in range(n):
            expect *= beta[i]
        assert reach == expect                      # P(position n reached) = prod beta_i
        assert bool(prefixes) == (reach > 0)
        for pre in prefixes:
            cond = oe.conditional_token_law(law, pre)
            for v in range(V):
                assert cond.get(v, Fraction(0)) == p[n][v], (n, pre, v)
    assert oe.expected_accepted_exact(law) == oa.expected_accepted(p, q)


def test_enumerated_law_with_disjoint_supports():
    # q puts mass where p has none: every draft is rejected, emitted token ~ p_0.
    p = [[Fraction(1, 2), Fraction(1, 2), Fraction(0)], [Fraction(1, 3)] * 3]
    q = [[Fraction(0), Fraction(0), Fraction(1)]]
    law = oe.emitted_law(p, q)
    assert law == {(0,): Fraction(1, 2), (1,): Fraction(1, 2)}


def test_p_equals_q_accepts_everything():
    rng = np.random.default_rng(5)
    B, k, V = 20, 4, 64
    z = rng.standard_normal((B, k + 1, V)).astype(np.float32) * 2
    zb = _bits(z)
    x = wl.draft_tokens_sampled(zb[:, :k], 0.7, seed=1)
    u = wl.philox_uniforms((B, k + 1), seed=3)
    out, num = oa.accept_stochastic(zb, zb[:, :k], x, u, 0.7)
    assert np.all(num == k)
    np.testing.assert_array_equal(out[:, :k], x)


def test_one_hot_distributions_reduce_to_greedy():
    rng = np.random.default_rng(6)
    B, k, V = 16, 3, 32
    zt = np.full((B, k + 1, V), -3e38, np.float32)
    zd = np.full((B, k, V), -3e38, np.float32)
    g = rng.integers(0, V, (B, k + 1))
    x = g[:, :k].copy()
    flip = rng.random((B, k)) < 0.3
    x[flip] = (x[flip] + 1 + rng.integers(0, V - 1, flip.sum())) % V
    zt[np.arange(B)[:, None], np.arange(k + 1)[None, :], g] = 1.0
    zd[np.arange(B)[:, None], np.arange(k)[None, :], x] = 1.0
    u = wl.philox_uniforms((B, k + 1), seed=2)
    out_s, num_s = oa.accept_stochastic(_bits(zt), _bits(zd), x, u, 0.7)
    out_g, num_g = oa.accept_greedy(_bits(zt), x)
    np.testing.assert_array_equal(out_s, out_g)
    np.testing.assert_array_equal(num_s, num_g)


def test_null_draft_logits_equal_one_hot_q():
    rng = np.random.default_rng(7)
    k, V = 3, 20
    for trial in range(50):
        p = [rng.dirichlet(np.ones(V)) for _ in range(k + 1)]
        x = rng.integers(0, V, k)
        u = rng.random(k + 1)
        qh = [np.eye(V)[x[i]] for i in range(k)]
        assert oa.accept_chain(p, None, x, u) == oa.accept_chain(p, qh, x, u)


def test_invalid_draft_is_rejected_and_residual_is_p():
    p = [np.array([0.25, 0.75]), np.array([0.5, 0.5])]
    toks, a = oa.accept_chain(p, None, [7], [0.0, 0.5])
    assert a == 0 and toks == [1]                   # u*R = 0.5 -> cumulative 0.25, 1.0


def test_inverse_cdf_boundaries():
    r = np.array([0.0, 0.5, 0.0, 0.5, 0.0])
    assert oa._inverse_cdf(r, 0.0) == 1
    assert oa._inverse_cdf(r, 0.4999) == 1
    assert oa._inverse_cdf(r, 0.5) == 3              # cumulative must exceed u*R
    assert oa._inverse_cdf(r, 1.0) == 3              # beyond the end: last nonzero
    assert oa._inverse_cdf(np.zeros(3), 0.3) is None


def test_monte_carlo_acceptance_length_matches_closed_form():
    rng = np.random.default_rng(8)
    k, V, T = 4, 12, 1.0
    zt = (rng.standard_normal((1, k + 1, V)) * 1.5).astype(np.float32)
    zd = (zt[:, :k] + rng.standard_normal((1, k, V)).astype(np.float32) * 0.8).astype(np.float32)
    ztb, zdb = _bits(zt), _bits(zd)
    p = [oa.softmax64(ztb[0, i], T) for i in range(k + 1)]
    q = [oa.softmax64(zdb[0, i], T) for i in range(k)]
    n = 40000
    xs = np.stack([rng.choice(V, n, p=q[i]) for i in range(k)], 1)
    us = rng.random((n, k + 1))
    a = np.array([oa.accept_chain(p, q, xs[t], us[t])[1] for t in range(n)])
    ea = oa.expected_accepted(p, q)
    assert abs(a.mean() - ea) < 4 * a.std() / np.sqrt(n)
    # and the emitted first token follows p_0 (chi-square, 11 dof, p > 1e-4)
    first = np.array([oa.accept_chain(p, q, xs[t], us[t])[0][0] for t in range(n // 4)])
    cnt = np.bincount(first, minlength=V)
    exp = p[0] * len(first)
    chi2 = np.sum((cnt - exp) ** 2 / exp)
    assert chi2 < 40.0


def test_margins_reported():
    rng = np.random.default_rng(9)
    zt = _bits(rng.standard_normal((3, 4, 30)) * 2)
    zd = _bits(rng.standard_normal((3, 3, 30)) * 2)
    x = wl.draft_tokens_sampled(zd, 0.7, seed=4)
    u = wl.philox_uniforms((3, 4), seed=5)
    out, num, mg = oa.accept_stochastic(zt, zd, x, u, 0.7, return_margins=True)
    assert mg.shape == (3,) and np.all(mg >= 0)
    out2, num2 = oa.accept_stochastic(zt, zd, x, u, 0.7)
    np.testing.assert_array_equal(out, out2)


# ---- softmax normalizer (the statistics an LM-head epilogue hands to the acceptance)

def test_softmax_normalizer_constant_row_is_vocabulary_size():
    for V in (1, 7, 4096, 128256):
        zmax, Z = oa.softmax_normalizer(_bits(np.full(V, -3.25)), 0.7)
        assert zmax == -3.25 and Z == V


def test_softmax_normalizer_two_level_closed_form():
    # one logit a, V-1 logits b: Z = 1 + (V-1) e^((b-a)/T)
    V, a, b, T = 1000, 2.0, 0.5, 0.5
    z = np.full(V, b)
    z[417] = a
    zmax, Z = oa.softmax_normalizer(_bits(z), T)
    assert zmax == a
    assert abs(Z - (1 + (V - 1) * np.exp((b - a) / T))) <= 1e-12 * Z


def test_softmax_normalizer_shift_and_batch():
    rng = np.random.default_rng(3)
    z = np.round(rng.normal(0, 4, size=(3, 5, 300)))            # integers: shifts by 8 stay exact in bf16
    zmax, Z = oa.softmax_normalizer(_bits(z), 1.3)
    zmax2, Z2 = oa.softmax_normalizer(_bits(z + 8), 1.3)
    assert zmax.shape == Z.shape == (3, 5)
    np.testing.assert_array_equal(zmax2, zmax + 8)
    np.testing.assert_allclose(Z2, Z, rtol=1e-14)
    # a very high temperature flattens the distribution towards uniform
    _, Zhot = oa.softmax_normalizer(_bits(z), 1e7)
    np.testing.assert_allclose(Zhot, 300, rtol=1e-5)


# ---- softmax64: the p = softmax(z / T) and q = softmax(z_d / T) of the acceptance rule

@pytest.mark.parametrize("T", [0.3, 0.7, 2.0])
def test_softmax64_two_level_closed_form(T):
    # one logit a and V-1 logits b: p_a = 1 / (1 + (V-1) e^((b-a)/T)), p_b = e^((b-a)/T) p_a
    V, a, b = 1000, 2.0, 0.5
    z = np.full(V, b)
    z[417] = a
    p = oa.softmax64(_bits(z), T)
    t = float(np.float32(T))
    pa = 1.0 / (1.0 + (V - 1) * np.exp((b - a) / t))
    assert abs(p[417] - pa) <= 1e-12 * pa
    others = np.delete(p, 417)
    np.testing.assert_allclose(others, np.exp((b - a) / t) * pa, rtol=1e-12)
    assert abs(p.sum() - 1.0) <= 1e-12


@pytest.mark.parametrize("T", [0.3, 0.7, 2.0])
def test_softmax64_log_ratios_are_logit_gaps_over_T(T):
    # log(p_i / p_j) = (z_i - z_j) / T for every pair: the temperature divides
    rng = np.random.default_rng(11)
    z = np.round(rng.normal(0, 3, 64) * 4) / 4               # quarter-integers: exact in bf16
    p = oa.softmax64(_bits(z), T)
    t = float(np.float32(T))
    i, j = np.meshgrid(np.arange(64), np.arange(64), indexing="ij")
    np.testing.assert_allclose(np.log(p[i] / p[j]), (z[i] - z[j]) / t, atol=1e-11)


@pytest.mark.parametrize("T", [0.3, 0.7, 2.0])
def test_softmax64_agrees_with_normalizer(T):
    # p_v = exp((z_v - zmax) / T) / Z with (zmax, Z) from the statistics form
    rng = np.random.default_rng(12)
    zb = _bits(rng.normal(0, 3, (3, 500)))
    zmax, Z = oa.softmax_normalizer(zb, T)
    z = (zb.astype(np.uint32) << 16).view(np.float32).astype(np.float64)   # bf16 -> f32 is a shift
    t = float(np.float32(T))
    for r in range(3):
        np.testing.assert_allclose(oa.softmax64(zb[r], T), np.exp((z[r] - zmax[r]) / t) / Z[r], rtol=1e-13)


def test_softmax64_temperature_limits():
    # T -> 0 concentrates on the argmax; a large T flattens to uniform
    z = np.array([0.0, 1.0, 3.0, 2.5, -1.0])
    p_cold = oa.softmax64(_bits(z), 0.01)
    assert np.argmax(p_cold) == 2
    assert abs(p_cold[3] / p_cold[2] - np.exp(-0.5 / float(np.float32(0.01)))) <= 1e-12 * p_cold[3] / p_cold[2]
    p_hot = oa.softmax64(_bits(z), 1e7)
    np.testing.assert_allclose(p_hot, 0.2, rtol=1e-6)
