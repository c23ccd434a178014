"""Pins of the oracle's tree verification: it reduces to the chain rule on a
chain-shaped tree, its exact emitted law (by enumeration over the uniforms)
follows the target at every step, and planted greedy trees walk the planted
path."""

from fractions import Fraction

import numpy as np
import pytest

import workloads as wl
from oracle import accept as oa
from oracle import tree as ot


def _bits(x):
    return wl.bf16_bits_from_f32(np.asarray(x, np.float32))


def _chain_parent(k):
    return np.arange(-1, k - 1, dtype=np.int32)


@pytest.mark.parametrize("seed", range(4))
def test_chain_shaped_tree_is_the_chain_rule(seed):
    B, k, V, T = 12, 4, 50, 0.8
    zt, zd = wl.accept_logits(B, k, V, seed, 0.9, scale=2.0)
    x = wl.draft_tokens_sampled(zd, T, seed=seed + 10)
    x[0, 1] = V + 2                                   # an invalid draft is a rejection in both
    u = wl.philox_uniforms((B, k + 1), seed=seed + 20)
    parent = np.tile(_chain_parent(k), (B, 1))
    out_c, num_c = oa.accept_stochastic(zt, None, x, u, T)
    out_t, nodes_t, num_t = ot.accept_tree_stochastic(zt, parent, x, u, T)
    np.testing.assert_array_equal(out_t, out_c)
    np.testing.assert_array_equal(num_t, num_c)
    for b in range(B):
        np.testing.assert_array_equal(nodes_t[b, :num_t[b]], np.arange(num_t[b]))
    xg = wl.draft_tokens_greedy(zd)
    out_g, num_g = oa.accept_greedy(zt, xg)
    out_tg, _, num_tg = ot.accept_tree_greedy(zt, parent, xg)
    np.testing.assert_array_equal(out_tg, out_g)
    np.testing.assert_array_equal(num_tg, num_g)


def _rand_dist(rng, V):
    w = rng.integers(0, 6, size=V)
    w[rng.integers(V)] += 1
    return [Fraction(int(a), int(w.sum())) for a in w]


TREES = [
    ([-1, -1, 0, 0, 1], [0, 2, 1, 3, 0]),      # two root candidates, both with children
    ([-1, -1, -1, 2], [1, 1, 3, 2]),          # duplicate root candidates
    ([-1, 0, 1, 2], [2, 0, 9, 1]),            # chain with an out-of-range candidate
    ([-1, -1, -1, -1], [0, 1, 2, 3]),         # every token a candidate: the residual is empty
]


@pytest.mark.parametrize("tree", TREES)
@pytest.mark.parametrize("seed", range(3))
def test_emitted_law_follows_the_target_at_every_step(tree, seed):
    parent, x = tree
    V = 4
    rng = np.random.default_rng(seed)
    P = [_rand_dist(rng, V) for _ in range(len(parent) + 1)]
    law = ot.tree_emitted_law(P, parent, x)
    assert sum(law.values()) == 1
    first = ot.marginal_first(law)
    for v in range(V):
        assert first.get(v, 0) == P[0][v]
    # after an accepted candidate the next token follows that node's row
    for v in range(V):
        kids = [n for n in ot.children(parent, -1) if x[n] == v]
        if not kids or first.get(v, 0) == 0:
            continue
        cond = ot.conditional_next(law, v)
        n = kids[0]                                 # only the first of duplicate candidates can be accepted
        for w in range(V):
            assert cond.get(w, 0) == P[n + 1][w], (v, w)


def test_greedy_walks_the_planted_path():
    V, N = 40, 7
    parent = np.array([-1, -1, 0, 0, 1, 3, 3], np.int32)
    x = np.array([5, 9, 7, 11, 2, 30, 31], np.int32)
    z = np.zeros((1, N + 1, V), np.float32)
    z[0, 0, 5] = 3.0                        # root -> node 0 (token 5)
    z[0, 1, 11] = 2.0                       # node 0 -> node 3 (token 11)
    z[0, 4, 31] = 4.0                       # node 3 -> node 6 (token 31)
    z[0, 7, 17] = 1.0                       # node 6 (leaf): bonus argmax 17
    out, nodes, num = ot.accept_tree_greedy(_bits(z), parent[None], x[None])
    assert num[0] == 3
    np.testing.assert_array_equal(nodes[0, :3], [0, 3, 6])
    np.testing.assert_array_equal(out[0, :4], [5, 11, 31, 17])
    assert np.all(out[0, 4:] == -1) and np.all(nodes[0, 3:] == -1)
    # a mismatch at the root emits the root's argmax
    z[0, 0, 5] = 0.0
    z[0, 0, 8] = 3.0
    out, nodes, num = ot.accept_tree_greedy(_bits(z), parent[None], x[None])
    assert num[0] == 0 and out[0, 0] == 8 and np.all(out[0, 1:] == -1)


def test_sampling_walk_with_certain_tokens():
    """One-hot rows: the walk accepts exactly the candidates that carry the mass."""
    V, N = 10, 4
    parent = [-1, -1, 1, 1]
    x = [3, 6, 2, 5]
    P = [np.eye(V)[6], np.eye(V)[0], np.eye(V)[5], np.eye(V)[1], np.eye(V)[8]]
    u = [0.999, 0.999, 0.999, 0.999, 0.5]
    toks, path = ot.walk(P, parent, x, u)
    # node 0 (token 3) has p = 0 -> rejected; node 1 (token 6) has p = 1 -> accepted even at u near 1;
    # at node 1 (row 2): node 2 (token 2) rejected, node 3 (token 5) accepted; node 3 is a leaf and its
    # row (row 4) puts all mass on 8, the bonus token
    assert path == [1, 3] and toks == [6, 5, 8]


def _visible_top_down(parent):
    """Independent construction of the ancestor sets: node j is visible to
    every node of its subtree (found by descending through children)."""
    N = len(parent)
    vis = [0] * N
    for j in range(N):
        stack = [j]
        while stack:
            n = stack.pop()
            vis[n] |= 1 << j
            stack.extend(ot.children(parent, n))
    return vis


def test_tree_mask_chain_star_and_subtrees():
    m, d = ot.tree_attention_mask(list(range(-1, 9)))           # a chain of 10
    assert m == [(1 << (n + 1)) - 1 for n in range(10)] and d == list(range(1, 11))
    m, d = ot.tree_attention_mask([-1] * 7)                    # a star
    assert m == [1 << n for n in range(7)] and d == [1] * 7
    for N, br in ((25, [4, 3, 2, 1]), (64, [2]), (13, [3, 1])):
        par = wl.tree_shape(N, br)
        m, d = ot.tree_attention_mask(par)
        assert m == _visible_top_down(par)
        assert d == [bin(x).count("1") for x in m]
    m, d = ot.tree_attention_mask(wl.TREE25)
    assert max(d) >= 3 and m == _visible_top_down(wl.TREE25)


def test_tree_mask_invalid_parents():
    par = [-1, 0, 5, 1, -3, 4, 2]      # node 2's parent lies after it; node 4's is below -1
    m, d = ot.tree_attention_mask(par)
    assert m[:2] == [1, 3] and m[3] == 0b1011 and d[3] == 3
    assert m[2] == 0 and m[4] == 0 and d[2] == d[4] == 0
    assert m[5] == 0 and m[6] == 0     # their descendants are unreachable too


def test_accepted_path_is_the_mask_of_its_last_node():
    B, N, V = 16, 25, 300
    zt, zd = wl.accept_logits(B, N, V, 3, 0.97, scale=2.0)
    par = np.asarray(wl.TREE25, np.int32)
    x = wl.tree_tokens_topk(zd, par)
    parents = np.tile(par, (B, 1))
    _, nodes, num = ot.accept_tree_greedy(zt, parents, x)
    masks, depths = ot.tree_attention_masks(parents)
    assert num.max() >= 2
    for b in range(B):
        a = int(num[b])
        if a == 0:
            continue
        last = int(nodes[b, a - 1])
        bits = [j for j in range(N) if (int(masks[b, last]) >> j) & 1]
        assert bits == sorted(nodes[b, :a].tolist()) and depths[b, last] == a
