"""Oracle pins for the expert part of the layer.

The expert MLP is OLMoE's bias-free SwiGLU block (the model of the Implementation
Details section): FFN(x) = W_down (silu(W_gate x) * (W_up x)), and the layer output is the
routing-weighted sum over the selected experts (Section 2 with the cap of Section 2.1).
Pins: numpy fp64 matmuls with scipy's logistic function (library routines the oracle
does not use), a closed form when all experts are identical, and the residual identity.
"""
import numpy as np
import pytest
from scipy.special import expit

from oracle import oracle as O
from paper_2608_04401_amd import synth


def ffn_np(x, Wgu, Wd):
    m = Wd.shape[1]
    g = Wgu[:m].astype(np.float64) @ x.astype(np.float64)
    u = Wgu[m:].astype(np.float64) @ x.astype(np.float64)
    return Wd.astype(np.float64) @ (g * expit(g) * u)


@pytest.fixture(scope="module")
def tiny():
    return synth.tiny_layer(seed=0)


def test_router_logits_match_matmul(tiny):
    lg = O.router_logits(tiny.x, tiny.W_router)
    ref = tiny.x.astype(np.float64) @ tiny.W_router.astype(np.float64).T
    np.testing.assert_allclose(lg, ref, rtol=1e-12, atol=1e-14)


def test_experts_match_library_matmul(tiny):
    L = tiny
    r = O.route(O.router_logits(L.x, L.W_router).astype(np.float32), K=8)
    y = O.moe_experts(L.x, L.W_gu, L.W_down, r.k, r.ids, r.w)
    for t in range(0, L.T, 5):
        ref = np.zeros(L.d)
        for j in range(r.k[t]):
            ref += r.w[t, j] * ffn_np(L.x[t], L.W_gu[r.ids[t, j]], L.W_down[r.ids[t, j]])
        np.testing.assert_allclose(y[t], ref, rtol=1e-10, atol=1e-13)


def test_gate_and_up_are_not_interchangeable(tiny):
    """Non-symmetric check: swapping gate and up rows changes the output (so the pin above
    distinguishes them)."""
    L = tiny
    m = L.m
    Wsw = np.concatenate([L.W_gu[:, m:], L.W_gu[:, :m]], axis=1)
    k = np.ones(4, np.int32)
    ids = np.zeros((4, 1), np.int32)
    w = np.ones((4, 1))
    a = O.moe_experts(L.x, L.W_gu, L.W_down, k, ids, w, tokens=np.arange(4))
    b = O.moe_experts(L.x, Wsw, L.W_down, k, ids, w, tokens=np.arange(4))
    assert np.abs(a - b).max() > 1e-3


def test_identical_experts_closed_form():
    """All experts equal: y_t = (sum_j w_tj) FFN(x_t)."""
    L = synth.moe_layer(64, 32, 6, 48, dtype="f32", seed=9)
    Wgu = np.repeat(L.W_gu[:1], 6, axis=0)
    Wd = np.repeat(L.W_down[:1], 6, axis=0)
    res = O.moe_forward(L.x, L.W_router, Wgu, Wd, K=4)
    for t in range(L.T):
        ref = res.routing.w[t].sum() * ffn_np(L.x[t], Wgu[0], Wd[0])
        np.testing.assert_allclose(res.y[t], ref, rtol=1e-10, atol=1e-14)


def test_residual_and_token_subset(tiny):
    L = tiny
    resid = synth.gaussian_logits(L.T, L.d, seed=4)
    tok = np.array([5, 0, 255, 17])
    full = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=8)
    sub = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=8, tokens=tok, residual=resid)
    np.testing.assert_allclose(sub.y, full.y[tok] + resid[tok].astype(np.float64), rtol=1e-13,
                               atol=1e-13)
    assert np.array_equal(sub.routing.k, full.routing.k[tok])


def test_forward_routes_on_its_fp64_logits(tiny):
    L = tiny
    full = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=8)
    lg = O.router_logits(L.x, L.W_router)
    np.testing.assert_array_equal(full.logits, lg)
    # k from the fp64 logits equals k from the fp32-rounded logits except at near-ties
    r32 = O.route(lg.astype(np.float32), K=8)
    diff = r32.k != full.routing.k
    assert (full.routing.margin[diff] < 1e-6).all()


def test_topk_mode_layer(tiny):
    L = tiny
    res = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=2, mode=O.MODE_TOPK)
    assert (res.routing.k == 2).all()
    order = np.argsort(-res.logits, axis=1, kind="stable")
    assert np.array_equal(res.routing.ids, order[:, :2])
