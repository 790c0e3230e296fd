"""GPU: the fused router + routing kernel.  Its k, ids and w must be bit-identical to the
two-step path (router kernel, then routing kernel) and its optional logits identical to the
router kernel's; and, like the layer, its routing must match the oracle's on its own fp64
logits except on near-ties."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

from helpers import NEAR_TIE, RTOL_BF16, cpu, rel_err_rows, to_gpu

pytestmark = pytest.mark.gpu
BF = torch.bfloat16


def _case(T, d, N, K, seed, **kw):
    L = synth.moe_layer(T, d, N, 64, dtype="bf16", seed=seed)
    x, Wr = to_gpu(L.x, BF), to_gpu(L.W_router, BF)
    k, ids, w, lg = B.elb_router_route(x, Wr, K=K, with_logits=True, **kw)
    lg2 = B.elb_router_logits(x, Wr)
    k2, ids2, w2 = B.elb_route(lg2, K=K, **kw)
    torch.cuda.synchronize()
    assert torch.equal(lg, lg2)
    assert torch.equal(k, k2) and torch.equal(ids, ids2) and torch.equal(w, w2)
    # without the logits output: the same routing
    k3, ids3, w3, none = B.elb_router_route(x, Wr, K=K, **kw)
    torch.cuda.synchronize()
    assert none is None and torch.equal(k3, k) and torch.equal(ids3, ids) and torch.equal(w3, w)
    return L, k, ids, w


@pytest.mark.parametrize("T,d,N,K", [(4096, 2048, 64, 8), (37, 96, 50, 5), (300, 320, 64, 16),
                                     (5, 544, 3, 2), (64, 2048, 64, 8), (1, 64, 8, 8),
                                     (1000, 128, 16, 12), (33, 256, 33, 16), (1, 256, 64, 8),
                                     (17, 512, 64, 16), (4095, 256, 64, 8)])
@pytest.mark.parametrize("mode", [B.MODE_ELBOW, B.MODE_TOPK])
def test_fused_equals_two_step(T, d, N, K, mode):
    _case(T, d, N, K, seed=T + d + N, mode=mode)


@pytest.mark.parametrize("renorm", [False, True])
@pytest.mark.parametrize("eps", [0.0, 1e-3])
def test_fused_eps_renorm(eps, renorm):
    _case(1000, 512, 64, 8, seed=3, eps=eps, renormalize=renorm)


def test_fused_empty_batch():
    """T = 0: nothing is launched and the outputs are empty."""
    x = torch.empty((0, 2048), dtype=BF, device="cuda")
    Wr = torch.zeros((64, 2048), dtype=BF, device="cuda")
    k, ids, w, lg = B.elb_router_route(x, Wr, K=8, with_logits=True)
    torch.cuda.synchronize()
    assert k.shape == (0,) and ids.shape == (0, 8) and w.shape == (0, 8) and lg.shape == (0, 64)


def test_fused_vs_oracle_olmoe():
    L, k, ids, w = _case(4096, 2048, 64, 8, seed=0)
    ref = O.route(O.router_logits(L.x, L.W_router).astype(np.float32), K=8)
    k, ids = cpu(k), cpu(ids)
    same = (k == ref.k) & (ids == ref.ids).all(axis=1)
    assert (ref.margin[~same] < NEAR_TIE).all()
    print("fused vs oracle: %d tokens, %d near-tie differences, mean k %.4f" % (
        len(k), int((~same).sum()), k.mean()))


@pytest.mark.parametrize("T,d,K,mode", [(4096, 2048, 8, B.MODE_ELBOW), (1025, 512, 8, B.MODE_ELBOW),
                                        (4097, 512, 8, B.MODE_TOPK), (2048, 256, 16, B.MODE_ELBOW),
                                        (8256, 1024, 12, B.MODE_ELBOW), (3000, 768, 8, B.MODE_ELBOW),
                                        (8192, 512, 8, B.MODE_ELBOW), (8193, 256, 16, B.MODE_TOPK)])
def test_layer_split_router_equals_fused(T, d, K, mode):
    """Batches above 1024 tokens with N = 64 and d % 256 == 0.  Up to T = 4096 the layer (and
    elb_router_route) take the one-launch router + routing: 16 tokens per block, the four
    quarters of the contraction in its four waves, then the 16-lane routing and the dispatch
    histogram of the block's quarter of its 64-token group.  Above 4096 the layer computes the
    router in four blocks per 64 tokens (each a quarter of the contraction) and routes in a
    second launch, which also writes the dispatch histogram: up to T = 8192 16 tokens per
    block, one histogram per quarter of each group, which the dispatch adds up; from T = 8193
    (and T = 8256) one lane per token with one histogram and the dispatch's scan launch.  The
    layer's logits, k, ids and w must be the fused entry point's bits and the two-step path's
    (router kernel, then routing kernel; slices of 1, 2, 3, 4 and 8 64-column chunks; ragged
    T), its per-expert counts those of its routing, its output the bits of the expert stage
    run on the same routing (which counts the assignments itself), and the oracle's."""
    L = synth.moe_layer(T, d, 64, 128, dtype="bf16", seed=T + d)
    x, Wr, Wgu, Wd = (to_gpu(a, BF) for a in (L.x, L.W_router, L.W_gu, L.W_down))
    y, dbg = B.elb_moe_forward(x, Wr, Wgu, Wd, K=K, mode=mode, debug=True)
    k, ids, w, lg = B.elb_router_route(x, Wr, K=K, mode=mode, with_logits=True)
    lg2 = B.elb_router_logits(x, Wr)
    k2, ids2, w2 = B.elb_route(lg2, K=K, mode=mode)
    torch.cuda.synchronize()
    assert torch.equal(dbg["logits"], lg) and torch.equal(lg, lg2)
    assert torch.equal(dbg["k"], k) and torch.equal(dbg["ids"], ids) and torch.equal(dbg["w"], w)
    assert torch.equal(k, k2) and torch.equal(ids, ids2) and torch.equal(w, w2)
    kk, ii = cpu(k), cpu(ids)
    assert np.array_equal(cpu(dbg["counts"]), np.bincount(ii[ii >= 0], minlength=64))
    assert cpu(dbg["counts"]).sum() == kk.sum()
    y2 = B.elb_moe_experts(x, Wgu, Wd, k, ids, w)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    tok = np.sort(np.random.default_rng(T).choice(T, 256, replace=False))
    ref = O.moe_experts(L.x, L.W_gu, L.W_down, kk[tok], ii[tok],
                        cpu(w)[tok].astype(np.float64), tokens=tok)
    rel = rel_err_rows(cpu(y)[tok], ref)
    assert rel.max() < RTOL_BF16, rel.max()


@pytest.mark.parametrize("T,d,K,mode", [(64, 2048, 8, B.MODE_ELBOW), (5, 512, 8, B.MODE_TOPK),
                                        (1024, 256, 16, B.MODE_ELBOW), (333, 768, 12, B.MODE_ELBOW),
                                        (100, 320, 8, B.MODE_ELBOW), (777, 192, 12, B.MODE_TOPK),
                                        (1, 256, 8, B.MODE_ELBOW), (65, 1024, 8, B.MODE_TOPK)])
def test_layer_small_batch_router_equals_fused(T, d, K, mode):
    """Batches of at most 1024 tokens with N = 64: with d % 256 == 0 the layer takes the
    one-launch router + routing, otherwise one wave per (16 tokens, 16 experts, quarter of the
    contraction) and the quarters summed in the 16-lane split routing.  Its logits, k, ids and
    w must be the fused entry point's bits and the two-step path's, its per-expert counts those
    of its routing, and its output the expert stage's bits on the same routing."""
    L = synth.moe_layer(T, d, 64, 128, dtype="bf16", seed=T + d + 1)
    x, Wr, Wgu, Wd = (to_gpu(a, BF) for a in (L.x, L.W_router, L.W_gu, L.W_down))
    y, dbg = B.elb_moe_forward(x, Wr, Wgu, Wd, K=K, mode=mode, debug=True)
    k, ids, w, lg = B.elb_router_route(x, Wr, K=K, mode=mode, with_logits=True)
    lg2 = B.elb_router_logits(x, Wr)
    k2, ids2, w2 = B.elb_route(lg2, K=K, mode=mode)
    torch.cuda.synchronize()
    assert torch.equal(dbg["logits"], lg) and torch.equal(lg, lg2)
    assert torch.equal(dbg["k"], k) and torch.equal(dbg["ids"], ids) and torch.equal(dbg["w"], w)
    assert torch.equal(k, k2) and torch.equal(ids, ids2) and torch.equal(w, w2)
    kk, ii = cpu(k), cpu(ids)
    assert np.array_equal(cpu(dbg["counts"]), np.bincount(ii[ii >= 0], minlength=64))
    y2 = B.elb_moe_experts(x, Wgu, Wd, k, ids, w)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
