"""Oracle pins: invariants, symmetries, library special cases and the load-balance theorem.

* Section 2.1: 1 <= k <= K; the selected set is a prefix of the descending order and a
  subset of the top-K set (monotone pruning; Appendix A.3 proof of Theorem 1);
  k under cap K equals min(k uncapped, K).
* Permuting a token's logits permutes the ids and leaves k unchanged; a constant shift of
  the logits leaves the probabilities, hence k, unchanged (up to near-ties).
* Special cases that reduce to library routines: K = 1 is argmax; top-K ids are the first
  K of a stable descending argsort; weights are scipy's softmax.
* Theorem 1 and Corollaries 1-2 (Appendix A.3) hold on any finite batch, and the paper's
  printed arithmetic (delta = 0.05 gives about 0.10 and about 7 for N = 64) is reproduced.
"""
import numpy as np
import pytest
from scipy.special import softmax

from oracle import oracle as O
from paper_2608_04401_amd import stats, synth

NEAR = 1e-6


@pytest.fixture(scope="module")
def planted():
    return synth.planted_logits(T=8192, N=64, seed=3)


def _topk_order(lg):
    return np.argsort(-lg.astype(np.float64), axis=1, kind="stable")


def test_bounds_prefix_subset(planted):
    K = 8
    r = O.route(planted, K=K)
    rt = O.route(planted, K=K, mode=O.MODE_TOPK)
    assert r.k.min() >= 1 and r.k.max() <= K
    order = _topk_order(planted)
    for t in range(planted.shape[0]):
        k = r.k[t]
        assert list(r.ids[t, :k]) == list(order[t, :k])          # prefix, rank order
        assert set(r.ids[t, :k]) <= set(rt.ids[t])                # subset of top-K
        assert len(set(r.ids[t, :k])) == k                        # distinct
        assert (r.ids[t, k:] == -1).all() and (r.w[t, k:] == 0).all()
    assert (rt.k == K).all()
    assert np.array_equal(rt.ids, order[:, :K])


def test_cap_commutes(planted):
    full = O.route(planted, K=64)
    for K in (1, 2, 4, 8, 16):
        r = O.route(planted, K=K)
        assert np.array_equal(r.k, np.minimum(full.k, K))


def test_k1_is_argmax():
    lg = synth.gaussian_logits(4096, 16, seed=5)
    lg[:100, 3] = lg[:100, 7] = 9.0          # exact ties -> lowest id
    r = O.route(lg, K=1)
    assert (r.k == 1).all()
    assert np.array_equal(r.ids[:, 0], np.argmax(lg, axis=1))


def test_weights_are_softmax(planted):
    r = O.route(planted, K=8)
    p = softmax(planted.astype(np.float64), axis=1)
    for t in range(0, planted.shape[0], 7):
        k = r.k[t]
        np.testing.assert_allclose(r.w[t, :k], p[t, r.ids[t, :k]], rtol=1e-14, atol=0)


def test_permutation_invariance(planted):
    rng = np.random.default_rng(11)
    lg = planted[:2048]
    r = O.route(lg, K=8)
    perm = rng.permutation(64)
    lp = lg[:, perm]                      # new expert j holds old expert perm[j]
    rp = O.route(lp, K=8)
    assert np.array_equal(r.k, rp.k)
    for t in range(lg.shape[0]):
        k = r.k[t]
        assert list(perm[rp.ids[t, :k]]) == list(r.ids[t, :k])


def test_shift_invariance_up_to_near_ties(planted):
    lg = planted[:4096]
    r = O.route(lg, K=8)
    rs = O.route((lg.astype(np.float64) + 0.75).astype(np.float32), K=8)
    diff = r.k != rs.k
    assert (r.margin[diff] < NEAR).all()
    assert diff.sum() <= 2


def test_theorem1_and_corollaries_hold_on_batches():
    for seed in range(4):
        for gen in ("planted", "gauss"):
            lg = (synth.planted_logits(4096, 64, seed=seed) if gen == "planted"
                  else synth.gaussian_logits(4096, 64, seed=seed, std=0.9))
            K = 8
            re = O.route(lg, K=K)
            rt = O.route(lg, K=K, mode=O.MODE_TOPK)
            ce = np.bincount(re.ids[re.ids >= 0], minlength=64)
            ct = np.bincount(rt.ids.ravel(), minlength=64)
            assert ce.sum() == re.k.sum() and ct.sum() == K * 4096
            rep = stats.load_balance_report(ce, ct, K=K, T=4096)
            assert rep["l1"] <= rep["l1_bound"] + 1e-12
            assert rep["top1_abs_change"] <= rep["top1_bound"] + 1e-12
            assert rep["cv2_abs_change"] <= rep["cv2_bound"] + 1e-12


def test_theorem_bound_is_tight_in_the_worst_case():
    """Worst case of the proof: removed mass disjoint from the kept mass gives equality."""
    # 2 experts, K = 2; half the tokens keep both, half keep only expert 0
    ct = np.array([100, 100])
    ce = np.array([100, 50])
    rep = stats.load_balance_report(ce, ct, K=2, T=100)
    # delta = 1 - 1.5/2 = 0.25, bound 2*0.25/0.75 = 2/3; l1 = |2/3-1/2| + |1/3-1/2| = 1/3
    assert abs(rep["delta"] - 0.25) < 1e-15
    assert abs(rep["l1_bound"] - 2 / 3) < 1e-15
    assert abs(rep["l1"] - 1 / 3) < 1e-15


def test_paper_printed_bound_arithmetic():
    """Appendix A.3, Discussion: delta = 0.05 -> 2 delta/(1-delta) ~ 0.10 and
    2 N delta/(1-delta)^2 ~ 7 for OLMoE's N = 64 experts."""
    assert abs(stats.theorem1_bound(0.05) - 0.10) < 0.006
    assert abs(stats.corollary2_bound(64, 0.05) - 7.0) < 0.1
    # Section 2.4: E[k] ~ 7.6 at K = 8 is a pruning rate of 0.05
    assert abs(stats.pruning_rate(7.6, 8) - 0.05) < 1e-12


def test_table1_sign_convention():
    """Table 1: % change = (top-K value - elbow value) / top-K value * 100, so an increase
    under elbow routing is negative."""
    ct = np.array([10, 10, 10, 10])
    ce = np.array([10, 9, 8, 7])       # elbow routing more skewed
    rep = stats.load_balance_report(ce, ct, K=4, T=10)
    assert rep["top1_share_change_pct"] < 0
    assert rep["cv_change_pct"] <= 0


def test_cv_hand_value_and_textbook_definition():
    """Appendix A.3, Corollary 2 writes CV^2 = N ||q||^2 - 1 for a utilisation vector q.  Hand
    value: counts (2, 1, 1, 0) give q = (1/2, 1/4, 1/4, 0), mean 1/4, population variance
    ((1/4)^2 + 0 + 0 + (1/4)^2) / 4 = 1/32, so CV^2 = (1/32) / (1/4)^2 = 1/2.  On random
    vectors the value must equal the textbook ratio of numpy's population standard deviation
    to the mean, and it must be 0 for uniform load."""
    q = stats.utilization([2, 1, 1, 0])
    assert np.array_equal(q, [0.5, 0.25, 0.25, 0.0])
    assert abs(stats.cv2(q) - 0.5) < 1e-15
    assert abs(stats.cv(q) - np.sqrt(0.5)) < 1e-15
    assert stats.cv(stats.utilization([7, 7, 7, 7, 7])) < 1e-7  # sqrt of a rounding residue
    rng = np.random.default_rng(5)
    for N in (2, 3, 8, 64):
        c = rng.integers(0, 1000, N) + 1
        qq = stats.utilization(c)
        assert abs(stats.cv(qq) - np.std(qq) / np.mean(qq)) < 1e-12
    # Table 1 sign on a case where both CVs are non-zero: the elbow routing's more skewed load
    # (CV 0.5 vs 0.25) is a negative % change of -100
    ct, ce = np.array([5, 3, 3, 5]), np.array([2, 1, 1, 0])
    rep = stats.load_balance_report(ce, ct, K=4, T=4)
    assert abs(rep["cv_top"] - 0.25) < 1e-15 and abs(rep["cv_elbow"] - np.sqrt(0.5)) < 1e-15
    assert abs(rep["cv_change_pct"] - (0.25 - np.sqrt(0.5)) / 0.25 * 100) < 1e-9
