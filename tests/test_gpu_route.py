"""GPU parity: routing kernel (softmax, descending sort, elbow, cap, weights) vs the oracle,
from identical seeded fp32 logits, through the C ABI."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

from helpers import compare_routing, cpu, to_gpu

pytestmark = pytest.mark.gpu


def _run(lg, K, **kw):
    k, ids, w = B.elb_route(to_gpu(lg), K=K, **kw)
    torch.cuda.synchronize()
    return k, ids, w


def test_route_planted_65536x64():
    """Routing-only workload: T=65536, N=64, K=8, planted head of 1..8 experts."""
    lg = synth.planted_logits(T=65536, N=64, seed=0)
    k, ids, w = _run(lg, 8)
    compare_routing(k, ids, w, O.route(lg, K=8), "planted 65536x64 elbow")


def test_route_planted_2p20x64():
    """The routing-only workload at T = 2^20 (the largest size the benchmark times, 4096 blocks of
    16 waves per SIMD): every token against the oracle."""
    lg = synth.planted_logits(T=1 << 20, N=64, seed=1)
    k, ids, w = _run(lg, 8)
    compare_routing(k, ids, w, O.route(lg, K=8), "planted 2^20x64 elbow")


def test_route_planted_topk_is_exact_everywhere():
    lg = synth.planted_logits(T=65536, N=64, seed=1)
    k, ids, w = _run(lg, 8, mode=B.MODE_TOPK)
    r = O.route(lg, K=8, mode=O.MODE_TOPK)
    assert np.array_equal(cpu(k), r.k) and np.array_equal(cpu(ids), r.ids)
    np.testing.assert_allclose(cpu(w), r.w, rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("N", [2, 3, 5, 8, 13, 16, 17, 31, 32, 33, 50, 63, 64])
def test_route_sizes(N):
    rng = np.random.default_rng(N)
    for T in (1, 63, 64, 65, 1000):
        for K in sorted({1, 2, min(8, N), min(N, 16)}):
            for gen in ("planted", "gauss_small", "gauss_big"):
                if gen == "planted":
                    lg = synth.planted_logits(T, N, seed=int(rng.integers(1 << 30)),
                                              m_max=min(8, N))
                else:
                    std = 0.2 if gen == "gauss_small" else 5.0
                    lg = synth.gaussian_logits(T, N, seed=int(rng.integers(1 << 30)), std=std)
                for mode in (B.MODE_ELBOW, B.MODE_TOPK):
                    k, ids, w = _run(lg, K, mode=mode)
                    compare_routing(k, ids, w, O.route(lg, K=K, mode=mode),
                                    "N=%d T=%d K=%d %s mode=%d" % (N, T, K, gen, mode))


@pytest.mark.parametrize("renorm", [False, True])
@pytest.mark.parametrize("eps", [0.0, 1e-8, 1e-3])
def test_route_eps_and_renormalize(eps, renorm):
    lg = synth.planted_logits(5000, 64, seed=7)
    k, ids, w = _run(lg, 8, eps=eps, renormalize=renorm)
    compare_routing(k, ids, w, O.route(lg, K=8, eps=eps, renorm=renorm),
                    "eps=%g renorm=%d" % (eps, renorm))


def test_route_exact_ties():
    """Quantised logits: many exactly equal values -> ids ordered by lower expert id."""
    rng = np.random.default_rng(3)
    lg = (np.round(rng.standard_normal((4096, 64)) * 2) / 2).astype(np.float32)
    lg[:64] = 1.5                              # all equal: k = 1, id 0
    for K in (1, 8, 16):
        for mode in (B.MODE_ELBOW, B.MODE_TOPK):
            k, ids, w = _run(lg, K, mode=mode)
            compare_routing(k, ids, w, O.route(lg, K=K, mode=mode), "ties K=%d" % K)
    k, ids, _ = _run(lg[:64], 8)
    assert (cpu(k) == 1).all() and (cpu(ids)[:, 0] == 0).all()


def test_route_step_curves():
    """m equal head logits over a flat tail: k = min(m + 1, K), head ids in id order."""
    N, T = 64, 64 * 12
    lg = np.full((T, N), -2.0, np.float32)
    rng = np.random.default_rng(5)
    ms = np.arange(T) % 12 + 1
    for t in range(T):
        lg[t, rng.permutation(N)[:ms[t]]] = 1.0
    k, ids, w = _run(lg, 8)
    assert np.array_equal(cpu(k), np.minimum(ms + 1, 8))
    compare_routing(k, ids, w, O.route(lg, K=8), "step curves")


def test_route_neg_inf_and_unaligned():
    lg = synth.planted_logits(2048, 64, seed=9)
    lg[::3, 5] = -np.inf
    lg[::7, :40] = -np.inf
    # an unaligned view: the logits start 4 bytes into the buffer
    buf = torch.empty(lg.size + 1, dtype=torch.float32, device="cuda:0")
    view = buf[1:].view(lg.shape)
    view.copy_(torch.from_numpy(lg))
    assert view.data_ptr() % 16 == 4
    k, ids, w = B.elb_route(view, K=8)
    torch.cuda.synchronize()
    compare_routing(k, ids, w, O.route(lg, K=8), "-inf, unaligned")


def test_route_empty():
    k, ids, w = B.elb_route(torch.empty((0, 64), dtype=torch.float32, device="cuda:0"), K=8)
    assert k.numel() == 0
