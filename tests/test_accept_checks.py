"""The checkers that GPU acceptance tests apply to every sequence
(tests/accept_checks.py) accept the oracle's own results and reject planted
mistakes: a wrong emitted token, a wrong accepted count, a wrong tree path."""

import numpy as np
import pytest

import workloads as wl
from oracle import accept as oa
from oracle import tree as ot
from tests import accept_checks as ac


def _chain_case(B, k, V, seed, c, with_draft=True):
    zt, zd = wl.accept_logits(B, k, V, seed, c, scale=2.0)
    x = wl.draft_tokens_sampled(zd, 0.7, seed=seed + 1)
    u = wl.philox_uniforms((B, k + 1), seed=seed + 2)
    return zt, (zd if with_draft else None), x, u


@pytest.mark.parametrize("with_draft", [True, False])
def test_chain_checker_accepts_oracle(with_draft):
    zt, zd, x, u = _chain_case(12, 4, 700, 3, 0.9, with_draft)
    out, num = oa.accept_stochastic(zt, zd, x, u, 0.7)
    ac.check_chain(out, num, zt, zd, x, u, 0.7)


def test_chain_checker_rejects_planted_mistakes():
    zt, zd, x, u = _chain_case(12, 4, 700, 4, 0.9)
    out, num = oa.accept_stochastic(zt, zd, x, u, 0.7)
    b = int(np.argmax(num < 4))                    # a sequence with a rejection
    bad = out.copy()
    bad[b, num[b]] = (bad[b, num[b]] + 1) % 700    # neighbouring token: off the CDF position
    with pytest.raises(AssertionError):
        ac.check_chain(bad, num, zt, zd, x, u, 0.7)
    bad_num = num.copy()
    bad_num[b] += 1                                # claims an accept the fp64 test rejects
    bad2 = out.copy()
    bad2[b, num[b]] = x[b, num[b]]
    with pytest.raises(AssertionError):
        ac.check_chain(bad2, bad_num, zt, zd, x, u, 0.7)


def _tree_case(B, N, V, seed, c, branching):
    zt, zd = wl.accept_logits(B, N, V, seed, c, scale=2.0)
    par = np.asarray(wl.tree_shape(N, branching), np.int32)
    x = wl.tree_tokens_topk(zd, par)
    parents = np.tile(par, (B, 1))
    u = wl.philox_uniforms((B, N + 1), seed=seed + 2)
    return zt, parents, x, u


def test_tree_checker_accepts_oracle_and_rejects_mistakes():
    zt, parents, x, u = _tree_case(10, 13, 500, 5, 0.95, [3, 1])
    out, nodes, num = ot.accept_tree_stochastic(zt, parents, x, u, 0.7)
    ac.check_tree(out, nodes, num, zt, parents, x, u, 0.7)
    b = int(np.argmax(num > 0))
    assert num[b] > 0
    bad_out = out.copy()
    bad_out[b, num[b]] = (bad_out[b, num[b]] + 1) % 500
    with pytest.raises(AssertionError):
        ac.check_tree(bad_out, nodes, num, zt, parents, x, u, 0.7)
    # a path cut short: the device would then have rejected a child the fp64 walk accepts
    bad_nodes, bad_num = nodes.copy(), num.copy()
    bad_nodes[b, num[b] - 1] = -1
    bad_num[b] -= 1
    with pytest.raises(AssertionError):
        ac.check_tree(out, bad_nodes, bad_num, zt, parents, x, u, 0.7)
