"""Verification of a drafted token tree.

Test infrastructure: a plain, slow restatement of the rule for the tests;
the product never imports it.

Standard EAGLE drafts a tree of candidate continuations and the target model
scores every node in one pass through a tree attention mask (paper, appendix
Detailed Discussions and Practical Takeaways: tree versus greedy drafting;
Table 2, tree rows, MGL 4.29 against 3.80 for the greedy chain).  The paper
states no acceptance rule of its own for the tree; the one restated here is
the tree form of the rule the EAGLE subsection cites for chains.

Encoding of one sequence's tree: N nodes, node n has parent[n] in
{-1, 0, .., n-1} (-1: a candidate for the first new token) and the drafted
token x[n]; the children of a node are its candidates, taken in index
order.  Target logits have N+1 rows: row 0 scores the first new position
(after the last accepted token), row n+1 the position after node n.
Uniforms: u[n] is the test of node n, u[N] the final draw (so a chain,
parent = [-1, 0, 1, ..], is exactly the chain verification of accept.py with
one-hot draft distributions).

Greedy (T == 0): from the root, descend into the first child whose token is
the argmax of the current row (lowest index on ties); where no child
matches, emit the argmax and stop.

Sampling (T > 0): the candidates are deterministic proposals (the top-k
expansion of an EAGLE tree), i.e. each is a one-hot draft distribution.  At
the current node with target distribution P, children are tested in order:
child n (token x) is accepted iff u[n] * (1 - S) < P(x), where S is the
mass of the tokens already rejected at this node (a token already rejected
has probability 0).  On acceptance the walk moves to that child; otherwise
x joins the rejected set.  When every child is rejected (or the node has
none), one token is drawn from P with the rejected tokens removed,
renormalised, by inverse CDF with u[N]: the smallest v whose cumulative
residual exceeds u[N] times the residual total (the last token of positive
mass if rounding leaves none; P itself if the residual vanished).
Accepting x with probability P(x)/(1 - S) and otherwise removing it is
sequential sampling from P, so the emitted tokens follow the target's law
exactly (pinned by tree_emitted_law).

Outputs per sequence: the accepted path's tokens then the emitted token,
and the accepted node indices.
"""

from __future__ import annotations

import itertools
from fractions import Fraction

import numpy as np

from .accept import _inverse_cdf, softmax64, target_argmax


def children(parent, p):
    """Children of node p (-1 = the root) in index order."""
    return [n for n in range(len(parent)) if int(parent[n]) == p]


def walk(P_rows, parent, x, u, margins=None):
    """One sequence's sampling walk over probability rows P_rows (N+1 rows,
    fp64 arrays or Fraction object arrays).  Returns (tokens, path nodes)."""
    N = len(parent)
    V = len(P_rows[0])
    cur = -1
    toks, path = [], []
    while True:
        P = P_rows[cur + 1]
        rejected = set()
        S = 0
        moved = False
        for n in children(parent, cur):
            xv = int(x[n])
            valid = 0 <= xv < V and xv not in rejected
            px = P[xv] if valid else 0
            rem = 1 - S
            if margins is not None:
                margins.append(float(abs(u[n] * rem - px) / px) if px > 0 else float("inf"))
            if u[n] * rem < px:
                toks.append(xv)
                path.append(n)
                cur = n
                moved = True
                break
            if valid:
                rejected.add(xv)
                S = S + px
        if moved:
            continue
        r = np.array(P, copy=True)
        for v in rejected:
            r[v] = 0
        v = _inverse_cdf(r, u[N], margins)
        if v is None:
            v = _inverse_cdf(P, u[N], margins)
        toks.append(int(v))
        return toks, path


def walk_greedy(zt_rows_f, parent, x):
    """One sequence's greedy walk over fp32 logit rows (N+1 rows)."""
    cur = -1
    toks, path = [], []
    while True:
        g = int(np.argmax(zt_rows_f[cur + 1]))
        nxt = next((n for n in children(parent, cur) if int(x[n]) == g), None)
        toks.append(g)
        if nxt is None:
            return toks, path
        path.append(nxt)
        cur = nxt


def _pack(B, N, results):
    out = np.full((B, N + 1), -1, dtype=np.int32)
    nodes = np.full((B, N), -1, dtype=np.int32)
    num = np.zeros(B, dtype=np.int32)
    for b, (toks, path) in enumerate(results):
        out[b, :len(toks)] = toks
        nodes[b, :len(path)] = path
        num[b] = len(path)
    return out, nodes, num


def accept_tree_greedy(zt_bits, parent, x):
    """zt_bits [B,N+1,V] bf16 bits, parent [B,N], x [B,N] ->
    (out_tokens [B,N+1], accepted_nodes [B,N], num_accepted [B])."""
    from .quantize import bf16_to_f32
    zt = bf16_to_f32(np.asarray(zt_bits))
    B, N1, V = zt.shape
    res = [walk_greedy(zt[b], parent[b], x[b]) for b in range(B)]
    return _pack(B, N1 - 1, res)


def accept_tree_stochastic(zt_bits, parent, x, uniforms, temperature, return_margins=False):
    """Sampling walk over bf16 logits (p = softmax(z / T) in fp64);
    uniforms [B,N+1] fp32.  Returns (out_tokens, accepted_nodes, num_accepted
    [, min_margin [B]])."""
    zt_bits = np.asarray(zt_bits)
    B, N1, V = zt_bits.shape
    u = np.asarray(uniforms, dtype=np.float32).reshape(B, N1).astype(np.float64)
    res, mins = [], np.full(B, np.inf)
    for b in range(B):
        P = [softmax64(zt_bits[b, i], temperature) for i in range(N1)]
        mg = [] if return_margins else None
        res.append(walk(P, parent[b], x[b], u[b], mg))
        if mg:
            mins[b] = min(mg)
    out = _pack(B, N1 - 1, res)
    return (*out, mins) if return_margins else out


# ------------------------------------------------------------------ exact law

def tree_emitted_law(P_rows, parent, x):
    """Exact distribution {emitted token tuple: probability} of `walk` for
    Fraction probability rows, by running `walk` itself on one representative
    of every region of the uniforms on which its output is constant: node n's
    test compares u[n] with one threshold (the rejected set before n is fixed
    by the tree: every earlier sibling was rejected), and the final draw u[N]
    is constant between consecutive cumulative breakpoints of every residual
    the walk can sample from."""
    N = len(parent)
    P = [np.array([Fraction(v) for v in row], dtype=object) for row in P_rows]
    V = len(P[0])
    thresholds, cuts = [], {Fraction(0), Fraction(1)}
    for p in [-1] + list(range(N)):
        rej, S = set(), Fraction(0)
        for n in children(parent, p):
            xv = int(x[n])
            valid = 0 <= xv < V and xv not in rej
            px = P[p + 1][xv] if valid else Fraction(0)
            t = px / (1 - S) if (1 - S) > 0 else Fraction(0)
            thresholds.append((n, min(t, Fraction(1))))
            if valid:
                rej.add(xv)
                S += px
            for dist in (P[p + 1], np.array([0 if v in rej else P[p + 1][v] for v in range(V)], dtype=object)):
                tot = sum(dist)
                acc = Fraction(0)
                if tot > 0:
                    for d in dist:
                        acc += d
                        cuts.add(acc / tot)
        if not children(parent, p):
            tot = sum(P[p + 1])
            acc = Fraction(0)
            for d in P[p + 1]:
                acc += d
                cuts.add(acc / tot)
    thr = dict(thresholds)
    cuts = sorted(cuts)
    law = {}
    for bits in itertools.product((0, 1), repeat=N):
        u = [None] * (N + 1)
        w = Fraction(1)
        for n in range(N):
            t = thr[n]
            if bits[n]:
                w *= t
                u[n] = t / 2            # inside [0, t): accepted if tested
            else:
                w *= 1 - t
                u[n] = (t + 1) / 2      # inside [t, 1): rejected if tested
            if w == 0:
                break
        if w == 0:
            continue
        for a, b in zip(cuts, cuts[1:]):
            u[N] = (a + b) / 2
            toks, _ = walk(P, parent, x, u)
            key = tuple(toks)
            law[key] = law.get(key, Fraction(0)) + w * (b - a)
    return law


def marginal_first(law):
    out = {}
    for seq, pr in law.items():
        out[seq[0]] = out.get(seq[0], Fraction(0)) + pr
    return out


def conditional_next(law, first):
    """Law of the second token given the first (only sequences of length >= 2)."""
    out, tot = {}, Fraction(0)
    for seq, pr in law.items():
        if seq[0] == first and len(seq) >= 2:
            out[seq[1]] = out.get(seq[1], Fraction(0)) + pr
            tot += pr
    return {v: pr / tot for v, pr in out.items()} if tot > 0 else {}


__all__ = ["children", "walk", "walk_greedy", "accept_tree_greedy", "accept_tree_stochastic",
           "tree_emitted_law", "marginal_first", "conditional_next", "target_argmax"]


def tree_attention_mask(parent):
    """Ancestor masks and depths of one sequence's tree (N <= 64 nodes).

    The target model scores every node in one pass: the row of node n may
    attend to the prefix, the last accepted token (the root) and the nodes on
    the path from the root to n, itself included; no other node (a sibling
    branch is another continuation).  Returned per node: the set of those
    tree nodes as bits of an integer (bit j = node j), and the depth (the
    number of nodes on the path, so node n sits depth positions after the
    root).  A node whose chain of parents leaves {-1, 0, .., n-1} at any step
    is unreachable: mask 0, depth 0.
    """
    N = len(parent)
    masks, depths = [], []
    for n in range(N):
        m, d, cur, ok = 0, 0, n, True
        while cur != -1:
            p = int(parent[cur])
            if p < -1 or p >= cur:
                ok = False
                break
            m |= 1 << cur
            d += 1
            cur = p
        masks.append(m if ok else 0)
        depths.append(d if ok else 0)
    return masks, depths


def tree_attention_masks(parents):
    """tree_attention_mask for a batch: parents int [B, N] -> (masks uint64
    [B, N], depths int32 [B, N])."""
    parents = np.asarray(parents)
    B, N = parents.shape
    masks = np.zeros((B, N), np.uint64)
    depths = np.zeros((B, N), np.int32)
    for b in range(B):
        m, d = tree_attention_mask(parents[b])
        masks[b] = np.array(m, dtype=np.uint64)
        depths[b] = d
    return masks, depths
