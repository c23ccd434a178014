"""Exact law of the tokens emitted by `accept.accept_chain`, by enumeration.

For tiny vocabularies the oracle's own decision function is run, in exact
Fraction arithmetic, on every draft chain x (weight prod_i q_i(x_i)) and on
one representative of every region of the uniforms u on which its output is
constant, weighted by the region's length:

  * u_i (i < k) enters only through u_i * q_i(x_i) < p_i(x_i), i.e. through
    the threshold t_i = p_i(x_i) / q_i(x_i): the regions are [0, min(t_i,1))
    and [min(t_i,1), 1).
  * u_k enters only through inverse-CDF sampling from one of the candidate
    distributions (the residual at a rejected position, or p_k).  The union of
    all their cumulative breakpoints partitions [0,1) into intervals on each
    of which every candidate draw is constant.

The result is the exact distribution of the emitted token sequence, which the
tests compare with the target law (the losslessness of speculative sampling,
paper §3.1 EAGLE) and with the closed-form expected acceptance length.
"""

from __future__ import annotations

import itertools
from fractions import Fraction

import numpy as np

from .accept import accept_chain


def _obj(v):
    return np.array([Fraction(t) for t in v], dtype=object)


def _breakpoints(dist):
    tot = sum(dist)
    if tot <= 0:
        return []
    cum, acc = [], Fraction(0)
    for d in dist:
        acc += d
        cum.append(acc / tot)
    return cum


def emitted_law(p, q, draft_support=None):
    """Exact distribution {emitted token tuple: probability} (Fractions).

    p: k+1 probability vectors (Fractions) of equal length V; q: k vectors.
    draft_support: optional list of k iterables restricting drafts (defaults
    to every v with q_i(v) > 0).
    """
    k = len(q)
    V = len(p[0])
    P = [_obj(v) for v in p]
    Q = [_obj(v) for v in q]
    # candidate distributions for the final draw and their breakpoints
    cuts = {Fraction(0), Fraction(1)}
    cands = [P[k]] + [np.maximum(P[i] - Q[i], 0) for i in range(k)] + [P[i] for i in range(k)]
    for d in cands:
        cuts.update(_breakpoints(list(d)))
    cuts = sorted(c for c in cuts if 0 <= c <= 1)
    uk_regions = [((a + b) / 2, b - a) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]

    if draft_support is None:
        draft_support = [[v for v in range(V) if Q[i][v] > 0] for i in range(k)]
    law = {}
    for x in itertools.product(*draft_support):
        wx = Fraction(1)
        for i in range(k):
            wx *= Q[i][x[i]]
        if wx == 0:
            continue
        # regions of each u_i
        ui_regions = []
        for i in range(k):
            t = min(P[i][x[i]] / Q[i][x[i]], Fraction(1))
            regs = []
            if t > 0:
                regs.append((t / 2, t))
            if t < 1:
                regs.append(((t + 1) / 2, 1 - t))
            ui_regions.append(regs)
        for combo in itertools.product(*ui_regions):
            wu = wx
            for _, w in combo:
                wu *= w
            for uk, wk in uk_regions:
                u = [c[0] for c in combo] + [uk]
                toks, _ = accept_chain(P, Q, list(x), u)
                key = tuple(int(t) for t in toks)
                law[key] = law.get(key, Fraction(0)) + wu * wk
    return law


def conditional_token_law(law, prefix):
    """Law of the token emitted right after `prefix`, given that it is reached.

    Returns {token: probability} over emitted sequences that extend `prefix`
    with at least one more token.
    """
    n = len(prefix)
    sub = {}
    tot = Fraction(0)
    for seq, pr in law.items():
        if len(seq) > n and tuple(seq[:n]) == tuple(prefix):
            sub[seq[n]] = sub.get(seq[n], Fraction(0)) + pr
            tot += pr
    if tot == 0:
        return {}
    return {t: pr / tot for t, pr in sub.items()}


def expected_accepted_exact(law):
    """E[a] = E[len(emitted) - 1] under the enumerated law."""
    return sum((len(seq) - 1) * pr for seq, pr in law.items())
