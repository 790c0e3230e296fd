"""Oracle pins: exhaustive enumeration on tiny N in exact rational arithmetic.

Every vector on a small rational grid (N <= 5) is routed by the fp64 oracle and by an
exact Fraction evaluation of the same rule (Algorithm 1 with the cap of Section 2.1, the
curve flipped to run from (0,0) to (1,1) as in Section 2.3).  With eps equal to the exact
binary value of 1e-8 no two deviations tie exactly, so the fp64 oracle must agree on e, k
and the ids for every vector.  A second, geometric evaluation (depth below the chord by a
cross product, eps = 0) checks the exact evaluation itself wherever its maximum is clear.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O

EPS = Fraction(1e-8)   # exact value of the double nearest 1e-8


def exact_rule(p, K):
    N = len(p)
    order = sorted(range(N), key=lambda j: (-p[j], j))
    s = [p[j] for j in order]
    R = s[0] - s[-1]
    D = [(s[0] - s[i]) / (R + EPS) - Fraction(i, N - 1) for i in range(N)]
    e = 0
    for i in range(1, N):
        if D[i] > D[e]:
            e = i
    return e, min(e + 1, K), order


def chord_depth_argmax(p):
    """argmax of the depth of sorted point (i, s_i) below the chord from the first to the
    last sorted point, via the cross product (chord vector) x (point vector).  Returns the
    argmax and the gap to the runner-up (in depth units)."""
    s = sorted(p, reverse=True)
    N = len(s)
    cx, cy = N - 1, s[-1] - s[0]
    depth = []
    for i in range(N):
        px, py = i, s[i] - s[0]
        depth.append(cx * py - cy * px)   # >0 above the chord ... negative below it
    depth = [-x for x in depth]
    best = max(range(N), key=lambda i: (depth[i], -i))
    others = [depth[i] for i in range(N) if i != best]
    return best, depth[best] - max(others), depth


def _grid(N, G):
    for v in itertools.product(range(G + 1), repeat=N):
        yield [Fraction(x, G) for x in v]


@pytest.mark.parametrize("N,G", [(2, 6), (3, 6), (4, 6), (5, 5)])
def test_bruteforce_exact(N, G):
    vecs = list(_grid(N, G))
    P = np.array([[float(x) for x in v] for v in vecs])
    for K in sorted({1, 2, N}):
        r = O.route_from_probs(P, K=K)
        for t, v in enumerate(vecs):
            e, k, order = exact_rule(v, K)
            assert r.e[t] == e, (v, K)
            assert r.k[t] == k, (v, K)
            assert list(r.ids[t, :k]) == order[:k], (v, K)
            assert list(r.ids[t, k:]) == [-1] * (K - k)
            assert np.array_equal(r.w[t, :k], P[t, order[:k]])


@pytest.mark.parametrize("N,G", [(3, 6), (4, 6), (5, 5)])
def test_exact_rule_matches_chord_geometry(N, G):
    """Where the chord-depth maximum is clear (gap far above the eps effect), the exact
    rule picks the same index."""
    checked = 0
    for v in _grid(N, G):
        best, gap, depth = chord_depth_argmax(v)
        s = sorted(v, reverse=True)
        R = s[0] - s[-1]
        if R == 0 or gap <= R * (N - 1) * Fraction(1, 10 ** 6):
            continue
        e, _, _ = exact_rule(v, N)
        assert e == best, v
        checked += 1
    assert checked > 100


def test_bruteforce_renormalised_weights():
    vecs = list(_grid(4, 4))
    vecs = [v for v in vecs if sum(v) > 0]
    P = np.array([[float(x) for x in v] for v in vecs])
    r = O.route_from_probs(P, K=3, renorm=True)
    for t, v in enumerate(vecs):
        e, k, order = exact_rule(v, 3)
        sel = sum(v[j] for j in order[:k])
        if sel == 0:
            continue
        want = [float(v[j] / sel) for j in order[:k]]
        assert np.allclose(r.w[t, :k], want, rtol=1e-15, atol=0)
