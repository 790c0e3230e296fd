"""Pins of the oracle's elbow angle (Section 2.3) and tail randomisation (Section 2.2):
closed forms, exact rational arithmetic, geometric bounds and special cases that reduce to
the plain routing."""
from fractions import Fraction
import math

import numpy as np
import pytest
from scipy.special import softmax

from oracle import oracle as O


# ------------------------------------------------------------------------------ elbow angle
@pytest.mark.parametrize("N,m", [(4, 1), (8, 3), (16, 5), (64, 2), (64, 7), (64, 30)])
def test_angle_step_curve_closed_form(N, m):
    """m equal head probabilities over a flat tail, eps = 0: the elbow is the first tail
    point, (x', p') = (m / (N-1), 1), so v1 = (-x', -1), v2 = (1 - x', 0) and
    theta = 90 deg + atan(x')."""
    p = np.full(N, 0.01)
    p[:m] = (1.0 - 0.01 * (N - m)) / m
    e, th = O.elbow_angle_from_probs(p, eps=0.0)
    assert e[0] == m
    assert abs(th[0] - (90.0 + math.degrees(math.atan(m / (N - 1))))) < 1e-9


def _exact_cos(p, eps):
    """cos theta at the elbow in exact rational arithmetic (argmax by exact D)."""
    q = [Fraction(v) for v in p]
    order = sorted(range(len(q)), key=lambda i: (-q[i], i))
    s = [q[i] for i in order]
    n = len(s)
    R = s[0] - s[-1] + Fraction(eps)
    D = [(s[0] - s[i]) / R - Fraction(i, n - 1) for i in range(n)]
    e = max(range(n), key=lambda i: (D[i], -i))
    x, y = Fraction(e, n - 1), (s[0] - s[e]) / R
    dot = (-x) * (1 - x) + (-y) * (1 - y)
    n1sq, n2sq = x * x + y * y, (1 - x) ** 2 + (1 - y) ** 2
    return e, dot, n1sq, n2sq


@pytest.mark.parametrize("p", [
    [0.5, 0.2, 0.15, 0.1, 0.05],
    [0.4, 0.3, 0.1, 0.08, 0.06, 0.04, 0.02, 0.0],
    [0.9] + [0.1 / 63] * 63,
    [0.25, 0.25, 0.2, 0.1, 0.1, 0.05, 0.05],
])
def test_angle_exact_rational(p):
    """The angle from exact rational cos^2 (and the sign of the dot product)."""
    e, dot, n1sq, n2sq = _exact_cos(p, 0)
    eo, th = O.elbow_angle_from_probs(np.array(p), eps=0.0)
    assert eo[0] == e
    c = float(dot) / math.sqrt(float(n1sq) * float(n2sq))
    assert abs(th[0] - math.degrees(math.acos(c))) < 1e-9


def test_angle_worked_example_value():
    """p = (.5, .2, .15, .1, .05): e = 1, (x', p') = (1/4, 2/3), cos = -59 / sqrt(7081)."""
    e, th = O.elbow_angle_from_probs(np.array([0.5, 0.2, 0.15, 0.1, 0.05]), eps=0.0)
    assert e[0] == 1
    assert abs(th[0] - math.degrees(math.acos(-59.0 / math.sqrt(7081.0)))) < 1e-9


@pytest.mark.parametrize("p", [0.5 - np.arange(8) / 64.0, np.full(16, 1 / 16),
                               np.array([0.4, 0.35, 0.25])])
def test_angle_no_elbow_is_180(p):
    """A linear sorted curve (dyadic steps, so every D_i is exactly 0), a concave one
    (nothing below the chord) or a uniform one: the elbow is the first point and the angle
    is taken as 180 degrees."""
    e, th = O.elbow_angle_from_probs(p, eps=0.0)
    assert e[0] == 0 and th[0] == 180.0


def test_angle_bounds_and_consistency():
    """Every elbow point lies in the unit square, inside the circle on the diagonal
    (0,0)-(1,1), so 90 <= theta <= 180 (Thales); e is the routing's uncapped index."""
    lg = np.random.default_rng(3).standard_normal((4000, 64)).astype(np.float32) * 1.5
    e, th = O.elbow_angle(lg)
    assert (th >= 90.0 - 1e-9).all() and (th <= 180.0).all()
    r = O.route(lg, K=64)
    assert np.array_equal(e, r.e)
    assert np.array_equal(np.minimum(e + 1, 64), r.k)


# ------------------------------------------------------------------------------ tail random
def _ranked_logits(T, N, rng):
    """Logits whose descending order is the expert id order (rank(c) = c), with random
    gaps; the elbow varies per token."""
    gaps = rng.exponential(1.0, (T, N)) * rng.uniform(0.1, 1.0, (T, 1))
    return (-np.cumsum(gaps, axis=1)).astype(np.float32)


def test_tail_random_increasing_draw_is_top_k():
    """Draws increasing with rank pick ranks k..K-1 in order: exactly fixed top-K routing."""
    rng = np.random.default_rng(0)
    T, N, K = 500, 64, 8
    lg = _ranked_logits(T, N, rng)
    rand = np.tile(np.arange(N, dtype=np.float32) / N, (T, 1))
    k, ids, w = O.route_tail_random(lg, rand, K)
    top = O.route(lg, K, mode=O.MODE_TOPK)
    assert np.array_equal(ids, top.ids)
    np.testing.assert_allclose(w, top.w, rtol=0, atol=0)
    assert np.array_equal(k, O.route(lg, K).k)


def test_tail_random_decreasing_draw_takes_the_last_ranks():
    rng = np.random.default_rng(1)
    T, N, K = 300, 64, 8
    lg = _ranked_logits(T, N, rng)
    rand = np.tile(1.0 - np.arange(N, dtype=np.float32) / N, (T, 1))
    k, ids, w = O.route_tail_random(lg, rand, K)
    for t in range(T):
        assert list(ids[t, :k[t]]) == list(range(k[t]))
        assert list(ids[t, k[t]:]) == list(range(N - 1, N - 1 - (K - k[t]), -1))


def test_tail_random_invariants():
    rng = np.random.default_rng(2)
    T, N, K = 2000, 64, 8
    lg = (rng.standard_normal((T, N)) * 1.2).astype(np.float32)
    rand = rng.random((T, N), dtype=np.float32)
    k, ids, w = O.route_tail_random(lg, rand, K)
    r = O.route(lg, K)
    p = softmax(lg.astype(np.float64), axis=1)
    assert np.array_equal(k, r.k)
    for t in range(T):
        kt = k[t]
        assert list(ids[t, :kt]) == list(r.ids[t, :kt])          # the elbow's experts first
        assert len(set(ids[t])) == K                              # K distinct experts
        assert not set(ids[t, kt:]) & set(ids[t, :kt])            # tail from outside them
        tail = ids[t, kt:]
        assert (np.diff(rand[t, tail]) >= 0).all()                # increasing draw order
        others = np.setdiff1d(np.arange(N), ids[t])
        if len(tail) and len(others):
            assert rand[t, tail].max() <= rand[t, others].min()   # the smallest draws
    np.testing.assert_allclose(w, p[np.arange(T)[:, None], ids], rtol=1e-12)
    _, _, wr = O.route_tail_random(lg, rand, K, renorm=True)
    np.testing.assert_allclose(wr.sum(axis=1), 1.0, rtol=1e-12)


def test_tail_random_is_uniform_over_the_rest():
    """With uniform draws, a given non-selected expert joins the tail with probability
    (K - k) / (N - k): compare the observed count with its expectation."""
    rng = np.random.default_rng(4)
    T, N, K = 20000, 64, 8
    lg = _ranked_logits(T, N, rng)
    rand = rng.random((T, N), dtype=np.float32)
    k, ids, _ = O.route_tail_random(lg, rand, K)
    expect = np.zeros(N)
    seen = np.zeros(N)
    for t in range(T):
        kt = k[t]
        expect[kt:] += (K - kt) / (N - kt)     # rank(c) = c for these logits
        seen[ids[t, kt:]] += 1
    z = (seen - expect) / np.sqrt(np.maximum(expect, 1.0))
    assert np.abs(z[expect > 50]).max() < 5.0
    assert abs(seen.sum() - expect.sum()) < 1e-6 * expect.sum() + 1


def test_tail_random_invalid_shape():
    with pytest.raises(ValueError):
        O.route_tail_random(np.zeros((3, 8), np.float32), np.zeros((3, 7), np.float32), 4)
