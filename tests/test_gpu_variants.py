"""GPU parity of the routing variants against the oracle, through the C ABI: caps above 16
up to the uncapped elbow routing (K = N), tail randomisation (Section 2.2) and the elbow
angle (Section 2.3), on identical seeded fp32 logits and draws.

Comparison rules as for the main routing: k, e and ids bit-exact except on near-ties (the
oracle's deviation margin below NEAR_TIE), weights to relative 1e-5.  Angles: within
ANGLE_TOL degrees where e agrees.  The kernel forms the elbow point in fp32 from
exp2-based u and the scaled deviation; the point's coordinates carry a relative error of a
few 1e-7 (of 1 - u) on these curves, and theta = atan2(|v1 x v2|, v1 . v2) moves by at
most |dP| / min(|v1|, |v2|) radians, below 1e-4 degrees for elbow points at distance
>= 1 / 63 from both ends (every e >= 1 at N = 64); ANGLE_TOL keeps a 20x margin.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

from helpers import NEAR_TIE, RTOL_BF16, compare_routing, cpu, rel_err_rows, to_gpu

pytestmark = pytest.mark.gpu
ANGLE_TOL = 2e-3


def _logits(gen, T, N, seed):
    if gen == "planted":
        return synth.planted_logits(T, N, seed=seed, m_max=min(8, N))
    return synth.gaussian_logits(T, N, seed=seed, std=0.2 if gen == "gauss_small" else 5.0)


# ------------------------------------------------------------------------- caps above 16
@pytest.mark.parametrize("N", [17, 33, 50, 64])
def test_route_caps_above_16(N):
    rng = np.random.default_rng(100 + N)
    for T in (1, 63, 64, 65, 1000):
        for K in sorted({17, (17 + N) // 2, N}):
            for gen in ("planted", "gauss_small", "gauss_big"):
                lg = _logits(gen, T, N, int(rng.integers(1 << 30)))
                for mode in (B.MODE_ELBOW, B.MODE_TOPK):
                    k, ids, w = B.elb_route(to_gpu(lg), K=K, mode=mode)
                    torch.cuda.synchronize()
                    compare_routing(k, ids, w, O.route(lg, K=K, mode=mode),
                                    "N=%d T=%d K=%d %s mode=%d" % (N, T, K, gen, mode))


@pytest.mark.parametrize("renorm", [False, True])
def test_route_uncapped_65536x64(renorm):
    """Elbow-N (K = N = 64) on the routing-only workload; every k is the elbow's own."""
    lg = synth.planted_logits(65536, 64, seed=11)
    k, ids, w = B.elb_route(to_gpu(lg), K=64, renormalize=renorm)
    torch.cuda.synchronize()
    ref = O.route(lg, K=64, renorm=renorm)
    compare_routing(k, ids, w, ref, "uncapped renorm=%d" % renorm)
    assert np.array_equal(ref.k, ref.e + 1)


def test_caps_kernel_matches_routing_kernel_bits():
    """At K = 16 the routing kernel serves elb_route; at K = 17 the variants kernel does.
    Both run the same arithmetic, so the uncapped ranks and weights agree bit for bit: the
    first 16 slots of a K = 17 top-K routing equal the K = 16 one."""
    lg = synth.planted_logits(5000, 64, seed=14)
    k16, i16, w16 = B.elb_route(to_gpu(lg), K=16, mode=B.MODE_TOPK)
    k17, i17, w17 = B.elb_route(to_gpu(lg), K=17, mode=B.MODE_TOPK)
    ke16, _, _ = B.elb_route(to_gpu(lg), K=16)
    ke17, _, _ = B.elb_route(to_gpu(lg), K=17)
    torch.cuda.synchronize()
    assert torch.equal(i17[:, :16], i16) and torch.equal(w17[:, :16], w16)
    assert torch.equal(torch.clamp(ke17, max=16), ke16)


def test_route_caps_ties_and_neg_inf():
    rng = np.random.default_rng(12)
    lg = (np.round(rng.standard_normal((2048, 64)) * 2) / 2).astype(np.float32)
    lg[:64] = 0.5
    lg[64::5, 3] = -np.inf
    lg[65::9, :40] = -np.inf
    for K in (24, 64):
        for mode in (B.MODE_ELBOW, B.MODE_TOPK):
            k, ids, w = B.elb_route(to_gpu(lg), K=K, mode=mode)
            torch.cuda.synchronize()
            compare_routing(k, ids, w, O.route(lg, K=K, mode=mode), "ties K=%d" % K)


def test_forward_uncapped_bf16():
    """The whole layer with the uncapped routing (K = N = 32): variable k up to 32 through
    dispatch, the grouped expert GEMMs and the combine."""
    L = synth.moe_layer(700, 128, 32, 128, dtype="bf16", seed=13)
    x, Wr, Wgu, Wd = (to_gpu(a, torch.bfloat16) for a in (L.x, L.W_router, L.W_gu, L.W_down))
    y, dbg = B.elb_moe_forward(x, Wr, Wgu, Wd, K=32, debug=True)
    torch.cuda.synchronize()
    ref = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=32)
    k, ids = cpu(dbg["k"]), cpu(dbg["ids"])
    same = (k == ref.routing.k) & (ids == ref.routing.ids).all(axis=1)
    assert (ref.routing.margin[~same] < NEAR_TIE).all()
    rel = rel_err_rows(cpu(y)[same], ref.y[same])
    print("uncapped forward: mean k %.3f, max k %d, max rel %.3e" % (k.mean(), k.max(),
                                                                     rel.max()))
    assert rel.max() < RTOL_BF16


# ------------------------------------------------------------------------- elbow angle
def _check_angle(lg, eps=1e-8, label=""):
    e, th = B.elb_elbow_angle(to_gpu(lg), eps=eps)
    torch.cuda.synchronize()
    e, th = cpu(e), cpu(th).astype(np.float64)
    eo, tho = O.elbow_angle(lg, eps=eps)
    margin = O.route(lg, K=lg.shape[1], eps=eps).margin
    near = margin < NEAR_TIE
    bad = (e != eo) & ~near
    assert not bad.any(), "%s: e differs outside near-ties at %s" % (
        label, np.nonzero(bad)[0][:8].tolist())
    ok = e == eo
    err = np.abs(th[ok] - tho[ok])
    print("%s: tokens %d, near-ties %d, e mismatches %d, max |dtheta| %.2e deg, "
          "mean theta %.3f" % (label, len(e), int(near.sum()), int((~ok).sum()),
                               err.max(), th.mean()))
    assert err.max() < ANGLE_TOL
    assert ((th >= 90.0 - 1e-3) & (th <= 180.0)).all()
    assert (th[e == 0] == 180.0).all()
    return e, th


def test_angle_planted_65536x64():
    _check_angle(synth.planted_logits(65536, 64, seed=20), label="planted 65536x64")


@pytest.mark.parametrize("N", [2, 3, 8, 17, 33, 64])
@pytest.mark.parametrize("gen", ["planted", "gauss_small", "gauss_big"])
def test_angle_sizes(N, gen):
    for T in (1, 65, 1000):
        _check_angle(_logits(gen, T, N, seed=N * 1000 + T), label="%s N=%d T=%d" % (gen, N, T))


@pytest.mark.parametrize("eps", [0.0, 1e-3])
def test_angle_eps(eps):
    _check_angle(synth.planted_logits(4096, 64, seed=21), eps=eps, label="eps=%g" % eps)


def test_angle_step_curve_closed_form():
    """m equal head logits over a flat tail, eps = 0: the elbow is the first tail point at
    (m / (N - 1), 1) and theta = 90 + atan(m / (N - 1)) degrees."""
    N, T = 64, 64 * 8
    ms = np.arange(T) % 30 + 1
    lg = np.full((T, N), -2.0, np.float32)
    rng = np.random.default_rng(22)
    for t in range(T):
        lg[t, rng.permutation(N)[:ms[t]]] = 1.0
    e, th = B.elb_elbow_angle(to_gpu(lg), eps=0.0)
    torch.cuda.synchronize()
    assert np.array_equal(cpu(e), ms)
    want = 90.0 + np.degrees(np.arctan(ms / (N - 1)))
    assert np.abs(cpu(th) - want).max() < 1e-4


def test_angle_optional_outputs_and_empty():
    lg = to_gpu(synth.planted_logits(300, 64, seed=23))
    e_full, th_full = B.elb_elbow_angle(lg)
    th_only = torch.empty(300, dtype=torch.float32, device=lg.device)
    assert B.lib().elb_elbow_angle(B._ptr(lg), 300, 64, 1e-8, None, B._ptr(th_only),
                                   B._stream()) == 0
    torch.cuda.synchronize()
    assert torch.equal(th_only, th_full)
    e, th = B.elb_elbow_angle(torch.empty((0, 64), dtype=torch.float32, device=lg.device))
    assert e.numel() == 0 and th.numel() == 0


# ------------------------------------------------------------------------- tail random
def _check_tail(lg, rand, K, renorm=False, label=""):
    k, ids, w = B.elb_route_tail_random(to_gpu(lg), to_gpu(rand), K=K, renormalize=renorm)
    torch.cuda.synchronize()
    k, ids, w = cpu(k), cpu(ids), cpu(w)
    ko, io, wo = O.route_tail_random(lg, rand, K, renorm=renorm)
    near = O.route(lg, K=K).margin < NEAR_TIE
    mism = (k != ko) | (ids != io).any(axis=1)
    bad = mism & ~near
    assert not bad.any(), "%s: %d mismatches outside near-ties, first %s" % (
        label, int(bad.sum()), np.nonzero(bad)[0][:8].tolist())
    ok = ~mism
    np.testing.assert_allclose(w[ok], wo[ok], rtol=1e-5, atol=1e-7)
    assert (ids >= 0).all() and (ids < lg.shape[1]).all()
    assert all(len(set(r)) == K for r in ids[: min(len(ids), 2000)])
    print("%s: tokens %d, near-ties %d, mismatches %d, mean k_elbow %.3f" % (
        label, len(k), int(near.sum()), int(mism.sum()), k.mean()))


@pytest.mark.parametrize("renorm", [False, True])
def test_tail_random_planted_65536x64(renorm):
    lg = synth.planted_logits(65536, 64, seed=30)
    _check_tail(lg, synth.uniform_draws(65536, 64, seed=30), 8, renorm,
                "planted 65536x64 renorm=%d" % renorm)


@pytest.mark.parametrize("N", [2, 5, 16, 33, 64])
def test_tail_random_sizes(N):
    rng = np.random.default_rng(31 + N)
    for T in (1, 65, 1000):
        for K in sorted({1, min(2, N), min(8, N), N}):
            for gen in ("planted", "gauss_small", "gauss_big"):
                s = int(rng.integers(1 << 30))
                _check_tail(_logits(gen, T, N, s), synth.uniform_draws(T, N, seed=s), K,
                            label="%s N=%d T=%d K=%d" % (gen, N, T, K))


def test_tail_random_tied_draws_and_topk_reduction():
    """Equal draws go to the lower expert id; draws increasing with the logit rank make the
    result the fixed top-K routing: bit-identical to the routing kernel's top-K ids and
    weights, with its elbow k."""
    lg = synth.planted_logits(4096, 64, seed=32)
    tied = np.round(synth.uniform_draws(4096, 64, seed=32) * 4) / 4
    _check_tail(lg, tied.astype(np.float32), 8, label="tied draws")
    order = np.argsort(np.lexsort((np.tile(np.arange(64), (4096, 1)), -lg)), axis=1)
    rank = order.astype(np.float32)            # rank of each expert (0 = largest logit)
    k, ids, w = B.elb_route_tail_random(to_gpu(lg), to_gpu(rank), K=8)
    kt, it, wt = B.elb_route(to_gpu(lg), K=8, mode=B.MODE_TOPK)
    ke, _, _ = B.elb_route(to_gpu(lg), K=8)
    torch.cuda.synchronize()
    # the variants kernel runs the routing kernel's arithmetic in the same order: the same bits
    assert torch.equal(ids, it) and torch.equal(w, wt) and torch.equal(k, ke)


def test_tail_random_topk_mode_has_no_tail():
    lg = synth.planted_logits(1000, 64, seed=33)
    rand = synth.uniform_draws(1000, 64, seed=33)
    k, ids, w = B.elb_route_tail_random(to_gpu(lg), to_gpu(rand), K=8, mode=B.MODE_TOPK)
    r = O.route(lg, K=8, mode=O.MODE_TOPK)
    torch.cuda.synchronize()
    assert (cpu(k) == 8).all() and np.array_equal(cpu(ids), r.ids)


@pytest.mark.parametrize("N", [16, 37, 64])
@pytest.mark.parametrize("K", [8, 16])
def test_tail_random_tied_and_neg_inf_logits(N, K):
    """Logits that tie at the selection boundary (quantised values, so rank k - 1 often has
    equal keys that only the lower-id rule separates) and -inf logits, for the caps that sort
    the keys alone (K <= 16): the elbow's experts and their weights must be the routing's."""
    if K > N:
        pytest.skip("K > N")
    rng = np.random.default_rng(N * 100 + K)
    T = 6000
    lg = (np.round(rng.standard_normal((T, N)) * 2) / 2).astype(np.float32)
    lg[:64] = 0.5                                # all equal: k = 1, the lowest id
    lg[64:128, : N // 2] = 1.0                   # a flat head of N / 2 equal logits
    lg[128::5, 3] = -np.inf
    lg[129::9, : N - 2] = -np.inf                # only two finite logits
    rand = (np.round(rng.random((T, N)) * 8) / 8).astype(np.float32)  # tied draws too
    for renorm in (False, True):
        _check_tail(lg, rand, K, renorm, "tied/-inf logits N=%d K=%d renorm=%d"
                    % (N, K, renorm))
