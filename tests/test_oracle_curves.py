"""Oracle pins: hand-worked curves and closed-form curve families.

The routing rule is Algorithm 1 (Appendix A.1) with the cap of Section 2.1; the expected
values come from tests/golden/elbow_curves.txt (worked by hand in exact fractions) and
from closed forms that hold for whole families of curves.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "elbow_curves.txt")


def _fixtures():
    out = []
    for line in open(GOLDEN):
        if not line.strip() or line.lstrip().startswith("#"):
            continue
        name, p, K, e, k, mg = [s.strip() for s in line.split("|")]
        p = [Fraction(s) for s in p.split(",")]
        out.append((name, p, int(K), int(e), int(k), Fraction(mg)))
    return out


@pytest.mark.parametrize("case", _fixtures(), ids=lambda c: c[0])
def test_hand_worked_curve(case):
    name, p, K, e, k, mg = case
    r = O.route_from_probs(np.array([float(x) for x in p]), K=K)
    assert r.e[0] == e
    assert r.k[0] == k
    # ids: the descending order of p (ties -> lower index), first k of it
    order = sorted(range(len(p)), key=lambda j: (-p[j], j))
    assert list(r.ids[0, :k]) == order[:k]
    assert all(i == -1 for i in r.ids[0, k:])
    assert np.allclose(r.w[0, :k], [float(p[j]) for j in order[:k]], rtol=0, atol=0)
    assert abs(r.margin[0] - float(mg)) < 1e-6


@pytest.mark.parametrize("N", [4, 8, 16, 64, 128])
@pytest.mark.parametrize("K", [1, 2, 8])
def test_step_curve_puts_elbow_at_step(N, K):
    """m equal head probabilities over a flat tail: e = m, k = min(m + 1, K)."""
    if K > N:
        pytest.skip("K > N")
    for m in range(1, N - 1):
        p = np.array([1.0] * m + [0.5] * (N - m))   # scale is irrelevant to the rule
        r = O.route_from_probs(p, K=K)
        assert r.e[0] == m, (N, m)
        assert r.k[0] == min(m + 1, K)


@pytest.mark.parametrize("N", [3, 8, 64])
def test_linear_curve_has_no_interior_deviation(N):
    """p_(i) = a - b i: every point lies on the chord, so e = 0 and k = 1."""
    b = 2.0 ** -4
    p = np.array([(N - i) * b for i in range(N)])   # exact binary fractions
    r = O.route_from_probs(p, K=min(8, N))
    assert r.e[0] == 0 and r.k[0] == 1
    assert r.margin[0] < 1e-6   # a tie up to eps: reported as a near-tie
    # with eps = 0 every D_i is exactly 0 (dyadic values): the first index wins the tie
    r0 = O.route_from_probs(p, K=min(8, N), eps=0.0)
    assert r0.e[0] == 0 and r0.k[0] == 1 and r0.margin[0] == 0.0


@pytest.mark.parametrize("N", [2, 8, 64])
def test_uniform_and_concave_curves_select_one(N):
    r = O.route_from_probs(np.full(N, 1.0 / N), K=min(8, N))
    assert r.k[0] == 1 and r.e[0] == 0
    # concave: every point is above the chord
    p = np.array([1.0 - (i / (N - 1)) ** 2 * 0.9 for i in range(N)])
    r = O.route_from_probs(p, K=min(8, N))
    assert r.k[0] == 1


@pytest.mark.parametrize("N", [8, 16, 64])
def test_convex_kink_family(N):
    """Convex piecewise-linear curve with one kink at index m (slope s1 then s2, s1 > chord
    slope > s2): D is increasing before m and decreasing after, so e = m."""
    rng = np.random.default_rng(N)
    for _ in range(200):
        m = int(rng.integers(1, N - 1))
        s2 = float(rng.uniform(0.01, 0.1))
        s1 = s2 * float(rng.uniform(2.0, 50.0)) * (N - 1) / max(m, 1)
        i = np.arange(N)
        p = np.where(i <= m, 10.0 - s1 * i, 10.0 - s1 * m - s2 * (i - m))
        chord = (p[0] - p[-1]) / (N - 1)
        if not (s1 > chord * (1 + 1e-6) and s2 < chord * (1 - 1e-6)):
            continue
        r = O.route_from_probs(p, K=8)
        assert r.e[0] == m
        assert r.k[0] == min(m + 1, 8)


def test_one_dominant_expert():
    p = np.array([0.9] + [0.1 / 63] * 63)
    r = O.route_from_probs(p, K=8)
    assert r.k[0] == 2 and list(r.ids[0, :2]) == [0, 1]


def test_step_curve_from_logits():
    """Same step curves through the softmax: equal logits give equal probabilities."""
    N = 64
    for m in range(1, 12):
        lg = np.full((1, N), -1.0, np.float32)
        idx = np.random.default_rng(m).permutation(N)[:m]
        lg[0, idx] = 3.0
        r = O.route(lg, K=8)
        assert r.k[0] == min(m + 1, 8)
        # head experts in id order, then the lowest-id tail expert
        expect = sorted(idx.tolist()) + [j for j in range(N) if j not in idx]
        assert list(r.ids[0, :r.k[0]]) == expect[:r.k[0]]


def test_eps_only_matters_for_tiny_range():
    """With a flat-ish curve (range ~1e-9) the eps term dominates the normaliser."""
    p = np.array([1.0 + 1e-9, 1.0, 1.0, 1.0])
    r0 = O.route_from_probs(p, K=4, eps=0.0)
    r1 = O.route_from_probs(p, K=4, eps=1e-8)
    assert r0.k[0] == 2          # exact: a one-point step
    assert r1.k[0] == 1          # eps >> range: D_1 = 1e-9/1.1e-8 - 1/3 < 0


def test_invalid_arguments_rejected():
    with pytest.raises(ValueError):
        O.route(np.zeros((2, 4), np.float32), K=5)      # K > N
    with pytest.raises(ValueError):
        O.route(np.zeros((2, 1), np.float32), K=1)      # N < 2
    with pytest.raises(ValueError):
        O.route(np.full((1, 4), -np.inf, np.float32), K=2)  # no finite logit
