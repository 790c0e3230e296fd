"""Oracle pins for the dispatch view of a routing (expert-major token lists).

Every (token, rank < k_t) assignment appears exactly once; counts sum to sum_t k_t
(the dispatch invariant the method's load statistics rest on, Appendix A.3: an expert's
load is the number of tokens routed to it); a hand-worked example fixes the order.
"""
import numpy as np

from oracle import oracle as O
from paper_2608_04401_amd import synth


def test_hand_worked_dispatch():
    # 4 tokens, N = 3, K = 2
    k = np.array([2, 1, 2, 1])
    ids = np.array([[2, 0], [1, -1], [0, 1], [2, -1]])
    counts, offsets, row_token, inv = O.dispatch(k, ids, 3)
    assert list(counts) == [2, 2, 2]
    assert list(offsets) == [0, 2, 4, 6]
    # expert 0: tokens 0, 2; expert 1: tokens 1, 2; expert 2: tokens 0, 3
    assert list(row_token) == [0, 2, 1, 2, 0, 3]
    assert inv.tolist() == [[4, 0], [2, -1], [1, 3], [5, -1]]


def test_dispatch_invariants_on_routing():
    lg = synth.planted_logits(3000, 64, seed=4)
    r = O.route(lg, K=8)
    counts, offsets, row_token, inv = O.dispatch(r.k, r.ids, 64)
    assert counts.sum() == r.k.sum() == offsets[-1] == len(row_token)
    assert np.array_equal(counts, np.bincount(r.ids[r.ids >= 0], minlength=64))
    assert np.array_equal(offsets[1:], np.cumsum(counts))
    for e in range(64):
        toks = row_token[offsets[e]:offsets[e + 1]]
        assert np.all(np.diff(toks) > 0)                         # increasing, distinct
        assert set(toks) == set(np.nonzero((r.ids == e).any(axis=1))[0])
    T, K = r.ids.shape
    for t in range(T):
        for j in range(K):
            if j < r.k[t]:
                row = inv[t, j]
                assert row_token[row] == t
                assert offsets[r.ids[t, j]] <= row < offsets[r.ids[t, j] + 1]
            else:
                assert inv[t, j] == -1
