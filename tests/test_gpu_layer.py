"""GPU parity: dispatch, router GEMM, grouped SwiGLU expert GEMMs, combine and the whole
layer, through the C ABI, against the fp64 oracle on identical seeded inputs."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

from helpers import (NEAR_TIE, RTOL_BF16, RTOL_F32, compare_routing, cpu, rel_err_rows,
                     to_gpu)

pytestmark = pytest.mark.gpu
BF = torch.bfloat16


def _layer_gpu(L, dtype):
    return tuple(to_gpu(a, dtype) for a in (L.x, L.W_router, L.W_gu, L.W_down))


@pytest.fixture(scope="module")
def olmoe():
    """OLMoE-shaped prefill layer: T=4096, d=2048, N=64 experts, intermediate 1024, bf16."""
    L = synth.olmoe_layer(T=4096, seed=0)
    lg64 = O.router_logits(L.x, L.W_router)
    return L, lg64, _layer_gpu(L, BF)


# ------------------------------------------------------------------------------ dispatch
@pytest.mark.parametrize("T,N,K", [(65536, 64, 8), (1000, 64, 8), (777, 5, 3), (64, 8, 8),
                                   (1, 2, 1), (4096, 33, 16), (256, 64, 8), (257, 64, 8),
                                   (200, 64, 64), (130, 17, 5), (255, 3, 3), (8192, 64, 8),
                                   (8193, 64, 8), (5000, 64, 64), (8000, 7, 2)])
def test_dispatch_matches_oracle(T, N, K):
    """T <= 256 runs the single-block dispatch, larger T the three-launch one."""
    lg = synth.planted_logits(T, N, seed=T + N, m_max=min(8, N))
    r = O.route(lg, K=K)
    counts, offsets, row_token, inv = B.elb_dispatch(to_gpu(r.k, torch.int32),
                                                     to_gpu(r.ids, torch.int32), N)
    c0, o0, rt0, inv0 = O.dispatch(r.k, r.ids, N)
    assert np.array_equal(cpu(counts), c0)
    assert np.array_equal(cpu(offsets), o0)
    assert np.array_equal(cpu(row_token)[:len(rt0)], rt0)
    assert (cpu(row_token)[len(rt0):] == -1).all()        # rows past sum k untouched
    assert np.array_equal(cpu(inv), inv0)


def test_dispatch_small_and_large_agree():
    """The single-block path (T <= 256) and the three-launch path give the same lists for
    the first 256 tokens of a routing (the three-launch run sees 300 tokens, so its first
    256 tokens' rows precede the rest within each expert)."""
    lg = synth.planted_logits(300, 64, seed=5)
    r = O.route(lg, K=8)
    k, ids = to_gpu(r.k, torch.int32), to_gpu(r.ids, torch.int32)
    cs, os_, rts, invs = B.elb_dispatch(k[:256].contiguous(), ids[:256].contiguous(), 64)
    cl, ol, rtl, invl = B.elb_dispatch(k, ids, 64)
    c0, o0, rt0, inv0 = O.dispatch(r.k[:256], r.ids[:256], 64)
    assert np.array_equal(cpu(cs), c0) and np.array_equal(cpu(rts)[:len(rt0)], rt0)
    assert np.array_equal(cpu(invs), inv0)
    c1, o1, rt1, inv1 = O.dispatch(r.k, r.ids, 64)
    assert np.array_equal(cpu(cl), c1) and np.array_equal(cpu(invl), inv1)


def test_dispatch_topk_and_ids_outside_selection():
    lg = synth.gaussian_logits(3000, 64, seed=2)
    r = O.route(lg, K=8, mode=O.MODE_TOPK)
    out = B.elb_dispatch(to_gpu(r.k, torch.int32), to_gpu(r.ids, torch.int32), 64)
    ref = O.dispatch(r.k, r.ids, 64)
    for a, b in zip(out[:2], ref[:2]):
        assert np.array_equal(cpu(a), b)
    assert np.array_equal(cpu(out[3]), ref[3])


# ------------------------------------------------------------------------------ router
def test_router_logits_bf16(olmoe):
    L, lg64, (x, Wr, _, _) = olmoe
    lg = cpu(B.elb_router_logits(x, Wr))
    rel = rel_err_rows(lg, lg64)
    assert rel.max() < 1e-5, rel.max()


def test_router_logits_f32_tiny():
    L = synth.tiny_layer(seed=0)
    lg = cpu(B.elb_router_logits(to_gpu(L.x), to_gpu(L.W_router)))
    assert rel_err_rows(lg, O.router_logits(L.x, L.W_router)).max() < 1e-5


@pytest.mark.parametrize("T,d,N", [(37, 96, 50), (33, 32, 64), (300, 320, 64), (5, 544, 3)])
def test_router_ragged_tokens_and_experts(T, d, N):
    """Ragged token counts (not a multiple of 16), expert counts, and d with no whole 64-deep
    k-step (32), a trailing half step (96, 544) or fewer steps than the load ring (320)."""
    L = synth.moe_layer(T, d, N, 64, dtype="bf16", seed=T + d)
    lg = cpu(B.elb_router_logits(to_gpu(L.x, BF), to_gpu(L.W_router, BF)))
    assert rel_err_rows(lg, O.router_logits(L.x, L.W_router)).max() < 1e-5


# ------------------------------------------------------------------------------ experts
def _experts_case(L, dtype, K, mode, rtol, sample=None, residual=None, seed=0):
    """Expert part with the ORACLE's routing (from its fp64 logits) fed to both sides."""
    lg64 = O.router_logits(L.x, L.W_router)
    r = O.route(lg64.astype(np.float32), K=K, mode=mode)
    x, _, Wgu, Wd = _layer_gpu(L, dtype)
    res_g = None if residual is None else to_gpu(residual, dtype)
    y = B.elb_moe_experts(x, Wgu, Wd, to_gpu(r.k, torch.int32), to_gpu(r.ids, torch.int32),
                          to_gpu(r.w.astype(np.float32)), residual=res_g)
    torch.cuda.synchronize()
    tok = np.arange(L.T) if sample is None else np.sort(
        np.random.default_rng(seed).choice(L.T, sample, replace=False))
    ref = O.moe_experts(L.x, L.W_gu, L.W_down, r.k[tok], r.ids[tok],
                        r.w[tok].astype(np.float32).astype(np.float64), tokens=tok,
                        residual=residual)
    rel = rel_err_rows(cpu(y)[tok], ref)
    print("experts: dtype %s K %d mode %d: tokens %d, max rel %.3e, mean rel %.3e" % (
        dtype, K, mode, len(tok), rel.max(), rel.mean()))
    assert rel.max() < rtol, rel.max()
    return y


def test_experts_f32_tiny():
    _experts_case(synth.tiny_layer(seed=0), torch.float32, 8, O.MODE_ELBOW, RTOL_F32)


def test_experts_f32_ragged():
    L = synth.moe_layer(333, 48, 5, 80, dtype="f32", seed=4)
    _experts_case(L, torch.float32, 3, O.MODE_ELBOW, RTOL_F32)
    _experts_case(L, torch.float32, 5, O.MODE_TOPK, RTOL_F32)


def test_experts_bf16_ragged_with_residual():
    L = synth.moe_layer(300, 192, 16, 320, dtype="bf16", seed=5)
    res = synth.round_bf16(synth.gaussian_logits(300, 192, seed=6))
    _experts_case(L, BF, 4, O.MODE_ELBOW, RTOL_BF16, residual=res)


@pytest.mark.parametrize("T,d,N,m,K", [(1000, 192, 8, 128, 2), (1536, 320, 4, 256, 2)])
def test_experts_bf16_large_tiles_ragged(T, d, N, m, K):
    """Shapes on the 256-row tile path (>= 192 rows per expert on average) with a partial
    output tile in the down GEMM (d not a multiple of 256) and few k-tiles (d = 192: 3 in
    the gate/up GEMM; m = 128: 2 in the down GEMM), with a residual."""
    L = synth.moe_layer(T, d, N, m, dtype="bf16", seed=T + d)
    res = synth.round_bf16(synth.gaussian_logits(T, d, seed=7))
    _experts_case(L, BF, K, O.MODE_ELBOW, RTOL_BF16, residual=res)
    _experts_case(L, BF, K, O.MODE_TOPK, RTOL_BF16)


@pytest.mark.parametrize("rems", [[1, 9, 17, 32] * 4, [5] * 15 + [0], [32] * 8 + [33] * 8])
def test_experts_large_tiles_remainder_rows(rems):
    """Experts of 256 + r rows on the 256-row tile path.  Remainders of at most 32 rows go to
    the tail kernel when that saves a round of blocks (m = 2048: 16 tiles across per M-tile,
    so 16 M-tiles per round on 256 compute units): the first two cases take it (32 -> 16 and
    31 -> 16 M-tiles), the third does not (32 -> 24, still two rounds).  Every row is
    compared with the oracle."""
    N, d, m = 16, 128, 2048
    counts = np.array([256 + r for r in rems])
    T = int(counts.sum())
    L = synth.moe_layer(T, d, N, m, dtype="bf16", seed=int(counts[0]) + len(rems))
    rng = np.random.default_rng(int(counts.sum()))
    ids = rng.permutation(np.repeat(np.arange(N), counts)).astype(np.int32)[:, None]
    k = np.ones(T, np.int32)
    w = rng.uniform(0.2, 1.0, (T, 1)).astype(np.float32)
    x, _, Wgu, Wd = _layer_gpu(L, BF)
    y = B.elb_moe_experts(x, Wgu, Wd, to_gpu(k, torch.int32), to_gpu(ids, torch.int32),
                          to_gpu(w))
    torch.cuda.synchronize()
    ref = O.moe_experts(L.x, L.W_gu, L.W_down, k, ids, w.astype(np.float64))
    rel = rel_err_rows(cpu(y), ref)
    print("remainders %s: %d tokens, max rel %.3e" % (sorted(set(rems)), T, rel.max()))
    assert rel.max() < RTOL_BF16


@pytest.mark.parametrize("mode", [O.MODE_ELBOW, O.MODE_TOPK])
def test_experts_bf16_olmoe_all_tokens(olmoe, mode):
    """Expert stage of the headline layer on all 4096 tokens (every row of every M-tile,
    remainder blocks included)."""
    L = olmoe[0]
    _experts_case(L, BF, 8, mode, RTOL_BF16)


# ------------------------------------------------------------------------------ whole layer
def _forward_case(L, dtype, K, mode, rtol, sample=None, seed=0, label="forward", renorm=False):
    """The whole layer against the oracle on every token (or a seeded sample).

    Routing parity is taken on the GPU's OWN fp32 logits: the oracle routes the logits the
    layer returned, and k and ids must be bit-exact on every token whose oracle margin is at
    least NEAR_TIE; the layer output is compared on every token with the oracle's expert pass
    run on the GPU's routing.  The oracle's own end-to-end layer (fp64 logits) is compared
    too, on the tokens whose routing agrees with it."""
    x, Wr, Wgu, Wd = _layer_gpu(L, dtype)
    y, dbg = B.elb_moe_forward(x, Wr, Wgu, Wd, K=K, mode=mode, renormalize=renorm, debug=True)
    torch.cuda.synchronize()
    tok = np.arange(L.T) if sample is None else np.sort(
        np.random.default_rng(seed).choice(L.T, sample, replace=False))
    ref = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=K, mode=mode, renorm=renorm,
                        tokens=tok)
    lg = cpu(dbg["logits"])
    yy = cpu(y)
    # router logits (fp32 accumulation) against the fp64 definition
    assert rel_err_rows(lg[tok], ref.logits).max() < 1e-5
    # routing from the same fp32 logits: bit-exact outside near-ties
    r = O.route(lg, K=K, mode=mode, renorm=renorm)
    near, mism = compare_routing(dbg["k"], dbg["ids"], dbg["w"], r, label)
    k, ids, w = cpu(dbg["k"]), cpu(dbg["ids"]), cpu(dbg["w"])
    same = (k == r.k) & (ids == r.ids).all(axis=1)
    # outputs on every compared token: the oracle's experts on the GPU's routing (the oracle's
    # fp64 weights where the routing agrees, the GPU's on near-tie tokens that differ)
    wref = np.where(same[:, None], r.w, w.astype(np.float64))
    yref = O.moe_experts(L.x, L.W_gu, L.W_down, k[tok], ids[tok], wref[tok], tokens=tok)
    rel = rel_err_rows(yy[tok], yref)
    assert rel.max() < rtol, rel.max()
    # the oracle's end-to-end layer, routed on its fp64 logits: tokens routed differently may
    # only be those within the logits' own rounding of a tie (|dD| <= 16 max|dl| for a
    # perturbation dl of the logits, doubled here), or near-ties
    dl = float(np.abs(lg[tok] - ref.logits).max())
    tie64 = max(NEAR_TIE, 32.0 * dl)
    same64 = (k[tok] == ref.routing.k) & (ids[tok] == ref.routing.ids).all(axis=1)
    assert (ref.routing.margin[~same64] < tie64).all()
    rel64 = rel_err_rows(yy[tok][same64], ref.y[same64])
    assert rel64.max() < rtol, rel64.max()
    print("%s: T %d K %d mode %d: %d tokens compared, near-ties %d (GPU-logit routing "
          "mismatches %d), max rel err %.3e (fp64-logit layer: %d tokens routed differently, "
          "max rel err %.3e)" % (label, L.T, K, mode, len(tok), near, mism, rel.max(),
                                 int((~same64).sum()), rel64.max()))
    # counts output = assignments per expert of the routing the layer used
    counts = cpu(dbg["counts"])
    assert counts.sum() == k.sum()
    assert np.array_equal(counts, np.bincount(ids[ids >= 0], minlength=L.N))
    return y, dbg


@pytest.mark.parametrize("T", [768, 1024])
@pytest.mark.parametrize("mode", [O.MODE_ELBOW, O.MODE_TOPK])
def test_forward_bf16_olmoe_mid_batches_all_tokens(olmoe, T, mode):
    """The headline layer's weights at mid-sized batches (the first T of its tokens): 90 to
    128 rows per expert, where the 256-row tile kernel takes over from the 128-row one (most
    experts fill less than half of their one M-tile), on every token."""
    L = olmoe[0]
    Lt = synth.LayerInputs(L.x[:T].copy(), L.W_router, L.W_gu, L.W_down, L.dtype)
    _forward_case(Lt, BF, 8, mode, RTOL_BF16, label="olmoe T=%d" % T)


def test_forward_f32_tiny_all_tokens():
    _forward_case(synth.tiny_layer(seed=0), torch.float32, 8, O.MODE_ELBOW, RTOL_F32)
    _forward_case(synth.tiny_layer(seed=1), torch.float32, 2, O.MODE_ELBOW, RTOL_F32)


@pytest.mark.parametrize("mode", [O.MODE_ELBOW, O.MODE_TOPK])
def test_forward_bf16_olmoe_prefill_all_tokens(olmoe, mode):
    """The headline layer (T = 4096, d = 2048, N = 64, intermediate 1024, bf16): all 4096
    tokens, routing bit-exact from the layer's own fp32 logits."""
    L = olmoe[0]
    y, dbg = _forward_case(L, BF, 8, mode, RTOL_BF16, label="olmoe prefill")
    if mode == O.MODE_ELBOW:
        print("prefill mean k %.4f" % cpu(dbg["k"]).mean())


@pytest.mark.parametrize("T,d,N,m,K,mode", [(2048, 512, 32, 256, 4, O.MODE_ELBOW),
                                             (1500, 384, 16, 128, 6, O.MODE_TOPK),
                                             (3000, 256, 40, 128, 8, O.MODE_ELBOW)])
def test_forward_bf16_other_expert_counts_all_tokens(T, d, N, m, K, mode):
    """Whole bf16 layers with N = 32, 16 and 40 experts (the fused router with N < 64, the
    one-lane routing at NP = 32 / 16 / 64 with pads, the dispatch with N < 64 and the grouped
    GEMMs at other tile fills): every token against the oracle."""
    L = synth.moe_layer(T, d, N, m, dtype="bf16", seed=T + N)
    _forward_case(L, BF, K, mode, RTOL_BF16, label="bf16 N=%d" % N)


@pytest.mark.parametrize("mode", [O.MODE_ELBOW, O.MODE_TOPK])
def test_forward_bf16_olmoe_prefill_renormalized_all_tokens(olmoe, mode):
    """The headline layer with renormalised weights (the selected probabilities divided by
    their sum, as the paper's cap option allows): all 4096 tokens against the oracle."""
    _forward_case(olmoe[0], BF, 8, mode, RTOL_BF16, label="olmoe prefill renorm", renorm=True)


def test_forward_bf16_small_renormalized_all_tokens():
    """Renormalised weights through the one-kernel fused router (N = 64 at T > 1024 but d not
    a multiple of 256) and through the small-batch path (T <= 1024)."""
    _forward_case(synth.moe_layer(1200, 320, 64, 128, dtype="bf16", seed=7), BF, 8,
                  O.MODE_ELBOW, RTOL_BF16, label="fused renorm", renorm=True)
    _forward_case(synth.moe_layer(300, 256, 64, 128, dtype="bf16", seed=8), BF, 8,
                  O.MODE_ELBOW, RTOL_BF16, label="small renorm", renorm=True)


@pytest.mark.parametrize("K", [1, 2])
def test_forward_bf16_small_caps_all_tokens(K):
    """Caps K = 1 (the layer is argmax routing: k = 1 for every token) and K = 2 on an
    OLMoE-width layer at T = 2048 (the split router; few rows per expert, so the 128-row GEMM
    tiles): every token against the oracle."""
    L = synth.moe_layer(2048, 2048, 64, 256, dtype="bf16", seed=30 + K)
    y, dbg = _forward_case(L, BF, K, O.MODE_ELBOW, RTOL_BF16, label="K=%d" % K)
    if K == 1:
        assert (cpu(dbg["k"]) == 1).all()


def test_forward_bf16_decode_all_tokens():
    L = synth.olmoe_layer(T=64, seed=2)
    _forward_case(L, BF, 8, O.MODE_ELBOW, RTOL_BF16)


def test_forward_deterministic(olmoe):
    _, _, (x, Wr, Wgu, Wd) = olmoe
    y1 = B.elb_moe_forward(x, Wr, Wgu, Wd, K=8)
    y2 = B.elb_moe_forward(x, Wr, Wgu, Wd, K=8)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def test_forward_residual_stack_two_layers():
    """Two residual layers h <- h + MoE_l(h), compared layer by layer on the same input
    (teacher-forced): the input of layer 2 is the oracle's layer-1 output rounded to bf16."""
    T, d, N, m = 256, 128, 8, 64
    h = synth.round_bf16(synth.gaussian_logits(T, d, seed=21))
    for l in range(2):
        L = synth.moe_layer(T, d, N, m, dtype="bf16", seed=[21, l], with_x=False)
        hg = to_gpu(h, BF)
        y = B.elb_moe_forward(hg, to_gpu(L.W_router, BF), to_gpu(L.W_gu, BF),
                              to_gpu(L.W_down, BF), K=4, residual=hg)
        torch.cuda.synchronize()
        ref = O.moe_forward(h, L.W_router, L.W_gu, L.W_down, K=4, residual=h)
        rel = rel_err_rows(cpu(y), ref.y)
        near = ref.routing.margin < NEAR_TIE
        assert rel[~near].max() < RTOL_BF16
        h = synth.round_bf16(ref.y.astype(np.float32))


@pytest.mark.parametrize("dtype", [torch.float32, BF])
def test_forward_and_experts_empty_batch(dtype):
    """T = 0: the layer and the expert stage return at once with empty outputs (nothing is
    launched), and the dispatch writes all-zero counts and offsets, for both dtypes."""
    d, N, m, K = 128, 8, 64, 4
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    x = torch.empty((0, d), dtype=dtype, device="cuda")
    Wr = (torch.randn((N, d), generator=g, device="cuda") * 0.02).to(dtype)
    Wgu = (torch.randn((N, 2 * m, d), generator=g, device="cuda") * 0.02).to(dtype)
    Wd = (torch.randn((N, d, m), generator=g, device="cuda") * 0.02).to(dtype)
    y, dbg = B.elb_moe_forward(x, Wr, Wgu, Wd, K=K, debug=True)
    k = torch.empty(0, dtype=torch.int32, device="cuda")
    ids = torch.empty((0, K), dtype=torch.int32, device="cuda")
    w = torch.empty((0, K), dtype=torch.float32, device="cuda")
    y2 = B.elb_moe_experts(x, Wgu, Wd, k, ids, w)
    counts, offsets, row_token, inv = B.elb_dispatch(k, ids, N)
    torch.cuda.synchronize()
    assert y.shape == (0, d) and y2.shape == (0, d)
    assert dbg["k"].numel() == 0 and dbg["ids"].shape == (0, K)
    assert int(counts.abs().sum()) == 0 and int(offsets.abs().sum()) == 0
