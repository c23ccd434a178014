"""GPU parity of spec_verify_accept_tree (token-tree verification) against
the oracle's tree walk (oracle/tree.py).

Greedy walks are bit-exact.  Sampling walks evaluate probabilities in fp32
statistics (the tests in double), so every sequence whose decisions all lie
farther than MARGIN from their boundary must match exactly, and every
sequence is replayed in fp64 along the device's own walk
(tests/accept_checks.py): each child test must be the fp64 decision unless
it lies within 1e-6 of its boundary, and the emitted token must sit at its
inverse-CDF position.  A chain-shaped tree must give exactly what the chain
kernel gives without draft logits (the same rule), and on the device the
first emitted token of a replicated tree follows the target distribution.
"""

import numpy as np
import pytest
import torch

import workloads as wl
from oracle import tree as ot
from tests.accept_checks import check_tree
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, host, need_gpu, say

pytestmark = pytest.mark.gpu

MARGIN = 4e-6


def _check_valid_walk(out, nodes, num, parent, x, V):
    B, N1 = out.shape
    N = N1 - 1
    for b in range(B):
        a = int(num[b])
        assert 0 <= a <= N
        path = nodes[b, :a]
        prev = -1
        for n in path:
            assert parent[b, n] == prev                # every step moves to a child
            prev = n
        assert np.all(nodes[b, a:] == -1)
        np.testing.assert_array_equal(out[b, :a], x[b, path])
        assert 0 <= out[b, a] < V and np.all(out[b, a + 1:] == -1)


def _case(B, N, V, seed, c, branching=None, parent=None):
    zt, zd = wl.accept_logits(B, N, V, seed, c, scale=2.0)
    par = np.asarray(parent if parent is not None else wl.tree_shape(N, branching), np.int32)
    x = wl.tree_tokens_topk(zd, par)
    parents = np.tile(par, (B, 1))
    u = wl.philox_uniforms((B, N + 1), seed=seed + 2)
    return zt, parents, x, u


@pytest.mark.parametrize("B,N,V,seed,c,branching", [
    (4, 7, 256, 0, 0.9, [2, 2, 1]),
    (9, 25, 5000, 1, 0.95, [4, 3, 2, 1]),
    (5, 13, 1001, 2, 0.9, [3, 1]),           # V not a multiple of 8: scalar path
    (3, 64, 20000, 3, 0.99, [2]),            # the largest tree
    (6, 1, 300, 4, 0.5, [1]),                # one node
])
def test_tree_greedy_bit_exact(B, N, V, seed, c, branching):
    p = need_gpu()
    say(f"tree greedy B={B} N={N} V={V}")
    zt, parents, x, _ = _case(B, N, V, seed, c, branching)
    x[0, 0] = V + 4                                    # an out-of-range candidate never matches
    parents[-1, N - 1] = N + 3                         # a node with an invalid parent is never reached
    out, nodes, num = p.verify_accept_tree(dev_bf16(zt), dev_i32(parents), dev_i32(x), None, 0.0)
    out_ref, nodes_ref, num_ref = ot.accept_tree_greedy(zt, parents, x)
    np.testing.assert_array_equal(host(num), num_ref)
    np.testing.assert_array_equal(host(out), out_ref)
    np.testing.assert_array_equal(host(nodes), nodes_ref)


@pytest.mark.parametrize("B,N,V,seed,c,branching,T", [
    (16, 7, 256, 0, 0.9, [2, 2, 1], 0.7),
    (12, 25, 5000, 1, 0.95, [4, 3, 2, 1], 0.7),
    (9, 13, 1001, 2, 0.9, [3, 1], 1.0),      # scalar path
    (6, 64, 20000, 3, 0.99, [2], 0.7),
    (16, 10, 3000, 4, 0.0, [5, 1], 0.7),     # uncorrelated: most candidates rejected
])
def test_tree_sampling_parity(B, N, V, seed, c, branching, T):
    p = need_gpu()
    say(f"tree sampling B={B} N={N} V={V} T={T}")
    zt, parents, x, u = _case(B, N, V, seed, c, branching)
    x[0, 1] = x[0, 0]                                  # a repeated candidate has probability 0
    out, nodes, num = p.verify_accept_tree(dev_bf16(zt), dev_i32(parents), dev_i32(x), dev_f32(u), T)
    out, nodes, num = host(out), host(nodes), host(num)
    out_ref, nodes_ref, num_ref, mg = ot.accept_tree_stochastic(zt, parents, x, u, T, return_margins=True)
    clear = mg > MARGIN
    assert clear.mean() >= 0.85
    np.testing.assert_array_equal(num[clear], num_ref[clear])
    np.testing.assert_array_equal(out[clear], out_ref[clear])
    np.testing.assert_array_equal(nodes[clear], nodes_ref[clear])
    _check_valid_walk(out, nodes, num, parents, x, V)
    check_tree(out, nodes, num, zt, parents, x, u, T)


@pytest.mark.parametrize("T", [0.0, 0.7])
def test_chain_shaped_tree_equals_chain_kernel(T):
    p = need_gpu()
    B, k, V = 32, 4, 20000
    zt, zd = wl.accept_logits(B, k, V, 9, 0.98, scale=2.0)
    x = wl.draft_tokens_sampled(zd, 0.7, seed=10)
    u = wl.philox_uniforms((B, k + 1), seed=11)
    parents = np.tile(np.arange(-1, k - 1, dtype=np.int32), (B, 1))
    dzt, dx = dev_bf16(zt), dev_i32(x)
    du = dev_f32(u) if T > 0 else None
    out_c, num_c = p.verify_accept(dzt, None, dx, du, T)
    out_t, nodes_t, num_t = p.verify_accept_tree(dzt, dev_i32(parents), dx, du, T)
    np.testing.assert_array_equal(host(out_t), host(out_c))
    np.testing.assert_array_equal(host(num_t), host(num_c))


def test_tree_first_token_follows_target_chi_square():
    """Losslessness on the device: one tree replicated over many sequences
    with fresh uniforms; the first emitted token follows p_root."""
    p = need_gpu()
    V, T, B = 64, 1.0, 13000
    par = np.array([-1, -1, -1, 0, 0, 1, 2], np.int32)
    N = len(par)
    rng = np.random.default_rng(31)
    z1 = (rng.standard_normal((1, N + 1, V)) * 1.5).astype(np.float32)
    zt = wl.bf16_bits_from_f32(np.repeat(z1, B, 0))
    # candidates: three distinct tokens at the root, then children
    x1 = np.array([int(np.argmax(z1[0, 0])), 5, 7, 1, 2, 3, 4], np.int32)
    if x1[0] in (5, 7):
        x1[0] = 9
    x = np.repeat(x1[None], B, 0)
    parents = np.repeat(par[None], B, 0)
    from oracle.accept import softmax64
    p0 = softmax64(zt[0, 0], T)
    counts = np.zeros(V)
    dzt, dpar, dx = dev_bf16(zt), dev_i32(parents), dev_i32(x)
    for rep in range(5):
        u = wl.philox_uniforms((B, N + 1), seed=300 + rep)
        out, _, _ = p.verify_accept_tree(dzt, dpar, dx, dev_f32(u), T)
        counts += np.bincount(host(out)[:, 0], minlength=V)
    n = counts.sum()
    exp = p0 * n
    keep = exp >= 5
    chi2 = np.sum((counts[keep] - exp[keep]) ** 2 / exp[keep]) + \
        (counts[~keep].sum() - exp[~keep].sum()) ** 2 / max(exp[~keep].sum(), 1e-9)
    dof = keep.sum()
    assert chi2 < dof + 6 * np.sqrt(2 * dof), (chi2, dof)


def test_tree25_full_vocabulary():
    """B = 64 sequences, the 25-node EAGLE-style tree, V = 128256: greedy
    bit-exact, sampling exact on clear sequences."""
    p = need_gpu()
    cfg = wl.CONFIGS["C4"]
    B, V, T = cfg["B"], cfg["V"], cfg["temperature"]
    par = np.asarray(wl.TREE25, np.int32)
    N = len(par)
    say(f"tree25 logits B={B} N={N} V={V}")
    zt, zd = wl.accept_logits(B, N, V, cfg["seed"] + 100, wl.C4_CORRELATION, scale=cfg["logit_std"],
                              rank=cfg["rank"])
    x = wl.tree_tokens_topk(zd, par)
    parents = np.tile(par, (B, 1))
    u = wl.philox_uniforms((B, N + 1), seed=cfg["uniform_seed"] + 100)
    dzt, dpar, dx = dev_bf16(zt), dev_i32(parents), dev_i32(x)
    out, nodes, num = p.verify_accept_tree(dzt, dpar, dx, None, 0.0)
    out_ref, nodes_ref, num_ref = ot.accept_tree_greedy(zt, parents, x)
    np.testing.assert_array_equal(host(out), out_ref)
    np.testing.assert_array_equal(host(nodes), nodes_ref)
    say(f"tree25 greedy MGL {np.mean(num_ref + 1):.3f}")
    out, nodes, num = p.verify_accept_tree(dzt, dpar, dx, dev_f32(u), T)
    out, nodes, num = host(out), host(nodes), host(num)
    out_ref, nodes_ref, num_ref, mg = ot.accept_tree_stochastic(zt, parents, x, u, T, return_margins=True)
    clear = mg > MARGIN
    say(f"tree25 sampling MGL {np.mean(num_ref + 1):.3f}, margin events {int((~clear).sum())}")
    assert clear.sum() >= 0.8 * B
    np.testing.assert_array_equal(out[clear], out_ref[clear])
    np.testing.assert_array_equal(nodes[clear], nodes_ref[clear])
    _check_valid_walk(out, nodes, num, parents, x, V)
    # every sequence, the margin ones included, replayed along the device's walk
    check_tree(out, nodes, num, zt, parents, x, u, T)


@pytest.mark.parametrize("B,N,seed", [(1, 1, 0), (7, 7, 1), (301, 25, 2), (33, 64, 3), (5, 40, 4)])
def test_tree_attention_mask_bit_exact(B, N, seed):
    """Masks and depths of random trees (some with invalid parents, whose
    subtrees are unreachable) equal the oracle's, bit for bit."""
    p = need_gpu()
    say(f"tree mask B={B} N={N}")
    rng = np.random.default_rng(seed)
    parents = np.array([[int(rng.integers(-1, n)) if n else -1 for n in range(N)] for _ in range(B)], np.int32)
    for b in range(0, B, 3):
        i = int(rng.integers(0, N))
        parents[b, i] = int(rng.choice([i, i + 2, -2, 99]))
    mask, depth = p.tree_attention_mask(dev_i32(parents))
    ref_m, ref_d = ot.tree_attention_masks(parents)
    np.testing.assert_array_equal(host(mask).view(np.uint64), ref_m)
    np.testing.assert_array_equal(host(depth), ref_d)


def test_tree_attention_mask_holds_the_accepted_path():
    """On the device: the mask of the last accepted node of
    spec_verify_accept_tree is exactly the accepted path, and its depth the
    path length."""
    p = need_gpu()
    B, V = 24, 5000
    par = np.asarray(wl.TREE25, np.int32)
    N = len(par)
    zt, parents, x, u = _case(B, N, V, 21, 0.97, parent=par)
    out, nodes, num = p.verify_accept_tree(dev_bf16(zt), dev_i32(parents), dev_i32(x), dev_f32(u), 0.7)
    mask, depth = p.tree_attention_mask(dev_i32(parents))
    nodes, num, mask, depth = host(nodes), host(num), host(mask).view(np.uint64), host(depth)
    assert num.max() >= 2
    for b in range(B):
        a = int(num[b])
        if a:
            last = int(nodes[b, a - 1])
            bits = [j for j in range(N) if (int(mask[b, last]) >> j) & 1]
            assert bits == sorted(nodes[b, :a].tolist()) and depth[b, last] == a
