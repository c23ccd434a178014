"""Checks of a device acceptance result that hold for every sequence, also
those whose decisions lie too close to a boundary for an exact comparison.

The device evaluates the speculative-sampling rule from fp32 statistics; the
oracle evaluates it in fp64.  Where a decision lies within ~1e-6 (relative)
of its boundary the two may legitimately differ.  These helpers replay the
device's own walk in fp64 and require:
  * every accept test the device took is the fp64 decision, unless it lies
    within DEC_TOL (relative to p) of the boundary u * q = p;
  * the emitted token carries positive residual mass and sits at the
    inverse-CDF position of u * R, up to CDF_TOL * R of cumulative mass.
"""

import numpy as np

from oracle import accept as oa

DEC_TOL = 1e-6
CDF_TOL = 1e-5


def _decision_ok(took_accept: bool, lhs: float, px: float) -> bool:
    """lhs = u * q (or u * (1 - S)); accept iff lhs < px in exact arithmetic."""
    if took_accept == (lhs < px):
        return True
    return px > 0 and abs(lhs - px) <= DEC_TOL * px


def _sample_ok(v: int, r: np.ndarray, P: np.ndarray, uk: float) -> bool:
    if not r.sum() > 0:
        r = P
    cum = np.cumsum(r)
    R = cum[-1]
    t = uk * R
    if not (0 <= v < len(r)) or not r[v] > 0:
        return False
    lo = cum[v - 1] if v > 0 else 0.0
    return lo <= t + CDF_TOL * R and cum[v] >= t - CDF_TOL * R


def check_chain(out, num, zt, zd, x, u, T):
    """Chain verification (spec_verify_accept), every sequence b.
    zt [B,k+1,V] and zd [B,k,V] (or None: one-hot drafts) bf16 bits."""
    B, k1, V = zt.shape
    k = k1 - 1
    u = np.asarray(u, np.float32).astype(np.float64)
    for b in range(B):
        a = int(num[b])
        assert 0 <= a <= k, (b, a)
        np.testing.assert_array_equal(out[b, :a], x[b, :a])
        assert np.all(out[b, a + 1:] == -1), b
        for i in range(min(a + 1, k)):
            xi = int(x[b, i])
            valid = 0 <= xi < V
            p = oa.softmax64(zt[b, i], T)
            px = p[xi] if valid else 0.0
            qx = (1.0 if zd is None else oa.softmax64(zd[b, i], T)[xi]) if valid else 0.0
            assert _decision_ok(i < a, u[b, i] * qx, px), (b, i, u[b, i] * qx, px)
        P = oa.softmax64(zt[b, a], T)
        if a < k:
            xa = int(x[b, a])
            if zd is None:
                r = P.copy()
                if 0 <= xa < V:
                    r[xa] = 0.0
            else:
                r = np.maximum(P - oa.softmax64(zd[b, a], T), 0.0)
        else:
            r = P
        assert _sample_ok(int(out[b, a]), r, P, u[b, k]), (b, a, int(out[b, a]))


def check_tree(out, nodes, num, zt, parent, x, u, T):
    """Tree verification (spec_verify_accept_tree), every sequence b: the
    device's path is replayed node by node (children in index order)."""
    B, N1, V = zt.shape
    N = N1 - 1
    u = np.asarray(u, np.float32).astype(np.float64)
    for b in range(B):
        a = int(num[b])
        path = [int(n) for n in nodes[b, :a]]
        assert np.all(nodes[b, a:] == -1), b
        cur = -1
        step = 0
        while True:
            P = oa.softmax64(zt[b, cur + 1], T)
            nxt = path[step] if step < a else None
            rejected = set()
            S = 0.0
            moved = False
            for n in [m for m in range(N) if int(parent[b, m]) == cur]:
                xv = int(x[b, n])
                valid = 0 <= xv < V and xv not in rejected
                px = P[xv] if valid else 0.0
                took = n == nxt
                assert _decision_ok(took, u[b, n] * (1.0 - S), px), (b, n, u[b, n] * (1.0 - S), px)
                if took:
                    assert int(out[b, step]) == xv, (b, step)
                    moved = True
                    break
                if valid:
                    rejected.add(xv)
                    S += px
            if moved:
                cur = nxt
                step += 1
                continue
            assert nxt is None, (b, "path continues past a node whose children were all rejected")
            r = P.copy()
            for v in rejected:
                r[v] = 0.0
            assert _sample_ok(int(out[b, a]), r, P, u[b, N]), (b, a, int(out[b, a]))
            assert np.all(out[b, a + 1:] == -1), b
            break
