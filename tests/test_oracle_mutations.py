"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a temporary copy of oracle.c (a textual substitution,
compiled with gcc into a scratch directory; the oracle itself is untouched) and checks
that at least one pin of the oracle suite fails on the mutant, while the unmodified
source passes all of them.
"""
import os
import tempfile
from fractions import Fraction

import numpy as np
import pytest
from scipy.special import expit, softmax

from oracle import oracle as O
from paper_2608_04401_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "elbow_curves.txt")

MUTATIONS = {
    # the orientation printed in Algorithm 1 (k = 1 for every token)
    "unflipped_curve": ("double pn = (p_max - p[sigma[i]]) / denom;",
                        "double pn = (p[sigma[i]] - p_min) / denom;"),
    "last_index_wins_ties": ("if (D[i] > D[e]) e = i;", "if (D[i] >= D[e]) e = i;"),
    "zero_based_count": ("k = e + 1 < K ? e + 1 : K;", "k = e < K ? (e > 0 ? e : 1) : K;"),
    "no_cap": ("k = e + 1 < K ? e + 1 : K;", "k = e + 1;"),
    "index_over_N": ("double xn = (double)i / (double)(N - 1);",
                     "double xn = (double)i / (double)N;"),
    "dropped_p_min": ("double denom = p_max - p_min + eps;", "double denom = p_max + eps;"),
    "ties_to_higher_id": ("(key[prev] == key[cur] && prev < cur)",
                          "(key[prev] == key[cur] && prev > cur)"),
    "unnormalised_softmax": ("for (int j = 0; j < N; ++j) p[j] /= s;\n        /* descending",
                             "for (int j = 0; j < N; ++j) p[j] /= 1.0;\n        /* descending"),
    "gate_up_swapped": ("const float *wg = Wgu + (long)i * d;",
                        "const float *wg = Wgu + (long)(m + i) * d;"),
    "silu_sign": ("return z / (1.0 + exp(-z));", "return z / (1.0 + exp(z));"),
    "weight_dropped": ("acc[c] += w[r * K + j] * o[c];", "acc[c] += o[c];"),
    "residual_dropped": ("acc[c] = residual ? (double)residual[t * d + c] : 0.0;",
                         "acc[c] = 0.0;"),
    # elbow angle (Section 2.3)
    "angle_v2_reversed": ("v2x = 1.0 - xe, v2y = 1.0 - ye;", "v2x = xe - 1.0, v2y = ye - 1.0;"),
    "angle_in_radians": ("th = acos(c) * (180.0 / acos(-1.0));", "th = acos(c);"),
    "angle_last_index_wins": ("if (yi - xi > best)", "if (yi - xi >= best)"),
    "angle_point_unflipped": ("double ye = (hi - p[sigma[e]]) / R;",
                              "double ye = (p[sigma[e]] - lo) / R;"),
    # tail randomisation (Section 2.2)
    "tail_largest_draws": ("if (c < 0 || rand[t * N + q] < rand[t * N + c]) c = q;",
                           "if (c < 0 || rand[t * N + q] > rand[t * N + c]) c = q;"),
    "tail_may_repeat": ("                if (used[q]) continue;\n", ""),
    "down_transposed": ("const float *wd = Wd + (long)r * m;\n        for (int i = 0; i < m; ++i) acc += (double)wd[i] * h[i];",
                        "for (int i = 0; i < m; ++i) acc += (double)Wd[(long)i * d + r] * h[i];"),
}


def _golden():
    for line in open(GOLDEN):
        if line.strip() and not line.lstrip().startswith("#"):
            name, p, K, e, k, mg = [s.strip() for s in line.split("|")]
            yield [Fraction(x) for x in p.split(",")], int(K), int(e), int(k), Fraction(mg)


def _ffn_np(x, Wgu, Wd):
    m = Wd.shape[1]
    g = Wgu[:m].astype(np.float64) @ x.astype(np.float64)
    u = Wgu[m:].astype(np.float64) @ x.astype(np.float64)
    return Wd.astype(np.float64) @ (g * expit(g) * u)


def run_pins(orc) -> list:
    """A compact copy of the oracle pins; returns the names of those that fail."""
    failed = []

    def check(name, fn):
        try:
            ok = fn()
        except Exception:
            ok = False
        if not ok:
            failed.append(name)

    def golden():
        for p, K, e, k, mg in _golden():
            r = orc.route_from_probs(np.array([float(x) for x in p]), K=K)
            order = sorted(range(len(p)), key=lambda j: (-p[j], j))
            if r.e[0] != e or r.k[0] != k or list(r.ids[0, :k]) != order[:k]:
                return False
            if abs(r.margin[0] - float(mg)) > 1e-6:
                return False
        return True

    def bruteforce():
        import itertools
        eps = Fraction(1e-8)
        vecs = [[Fraction(x, 4) for x in v] for v in itertools.product(range(5), repeat=4)]
        P = np.array([[float(x) for x in v] for v in vecs])
        r = orc.route_from_probs(P, K=4)
        for t, v in enumerate(vecs):
            order = sorted(range(4), key=lambda j: (-v[j], j))
            s = [v[j] for j in order]
            D = [(s[0] - s[i]) / (s[0] - s[-1] + eps) - Fraction(i, 3) for i in range(4)]
            e = max(range(4), key=lambda i: (D[i], -i))
            if r.k[t] != min(e + 1, 4) or list(r.ids[t, :r.k[t]]) != order[:r.k[t]]:
                return False
        return True

    def invariants():
        lg = synth.planted_logits(512, 16, seed=1, m_max=12)
        lg[:, 5] = lg[:, 9]                       # exact ties
        r = orc.route(lg, K=4)
        order = np.argsort(-lg.astype(np.float64), axis=1, kind="stable")
        p = softmax(lg.astype(np.float64), axis=1)
        for t in range(lg.shape[0]):
            k = r.k[t]
            if not 1 <= k <= 4 or list(r.ids[t, :k]) != list(order[t, :k]):
                return False
            if not np.allclose(r.w[t, :k], p[t, r.ids[t, :k]], rtol=1e-12):
                return False
        return True

    def ffn():
        L = synth.moe_layer(16, 24, 4, 40, dtype="f32", seed=2)
        resid = synth.gaussian_logits(16, 24, seed=6)
        res = orc.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=3, residual=resid)
        for t in range(16):
            ref = resid[t].astype(np.float64).copy()
            for j in range(res.routing.k[t]):
                e = res.routing.ids[t, j]
                ref += res.routing.w[t, j] * _ffn_np(L.x[t], L.W_gu[e], L.W_down[e])
            if not np.allclose(res.y[t], ref, rtol=1e-9, atol=1e-12):
                return False
        return True

    def exact_ties():
        p = np.array([(8 - i) * 2.0 ** -4 for i in range(8)])   # linear: D_i == 0 exactly
        r = orc.route_from_probs(p, K=8, eps=0.0)
        return r.e[0] == 0 and r.k[0] == 1

    def angle():
        import math
        for N, m in ((8, 3), (64, 7)):
            p = np.full(N, 0.01)
            p[:m] = (1.0 - 0.01 * (N - m)) / m
            e, th = orc.elbow_angle_from_probs(p, eps=0.0)
            if e[0] != m or abs(th[0] - (90 + math.degrees(math.atan(m / (N - 1))))) > 1e-9:
                return False
        e, th = orc.elbow_angle_from_probs(np.array([0.5, 0.2, 0.15, 0.1, 0.05]), eps=0.0)
        if e[0] != 1 or abs(th[0] - math.degrees(math.acos(-59 / math.sqrt(7081)))) > 1e-9:
            return False
        lin = np.array([(8 - i) * 2.0 ** -4 for i in range(8)])   # linear: D_i == 0 exactly
        e, th = orc.elbow_angle_from_probs(lin, eps=0.0)
        return e[0] == 0 and th[0] == 180.0

    def tail_random():
        rng = np.random.default_rng(5)
        T, N, K = 200, 32, 6
        lg = (-np.cumsum(rng.exponential(1.0, (T, N)), axis=1)).astype(np.float32)  # rank = id
        k, ids, w = orc.route_tail_random(lg, np.tile(np.arange(N, dtype=np.float32), (T, 1)), K)
        if not np.array_equal(ids, orc.route(lg, K, mode=O.MODE_TOPK).ids):
            return False
        rand = rng.random((T, N), dtype=np.float32)
        k, ids, w = orc.route_tail_random(lg, rand, K)
        for t in range(T):
            tail = ids[t, k[t]:]
            others = np.setdiff1d(np.arange(N), ids[t])
            if len(set(ids[t])) != K:
                return False
            if len(tail) and rand[t, tail].max() > rand[t, others].min():
                return False
        return True

    check("angle", angle)
    check("tail_random", tail_random)
    check("exact_ties", exact_ties)
    check("golden", golden)
    check("bruteforce", bruteforce)
    check("invariants", invariants)
    check("ffn", ffn)
    return failed


@pytest.fixture(scope="module")
def workdir():
    with tempfile.TemporaryDirectory(prefix="orc_mut_") as d:
        yield d


def test_unmodified_oracle_passes(workdir):
    assert run_pins(O.OracleLib(O.build())) == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutant_is_caught(name, workdir):
    src = open(O.SRC).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, "mutation anchor not found: %s" % name
    path = os.path.join(workdir, name + ".c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = O.compile_source(path, os.path.join(workdir, "lib%s.so" % name))
    failed = run_pins(O.OracleLib(lib))
    assert failed, "no pin caught mutation %s" % name
