"""GPU parity of the decode-sized expert path (weight-streaming grouped GEMMs, chosen when
an expert gets at most 16 rows on average) against the fp64 oracle, through the C ABI."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

from helpers import NEAR_TIE, RTOL_BF16, cpu, rel_err_rows, to_gpu

pytestmark = pytest.mark.gpu
BF = torch.bfloat16


def _gpu(L):
    return tuple(to_gpu(a, BF) for a in (L.x, L.W_router, L.W_gu, L.W_down))


@pytest.mark.parametrize("T", [1, 5, 64, 128])
@pytest.mark.parametrize("mode", [O.MODE_ELBOW, O.MODE_TOPK])
def test_forward_decode_olmoe_all_tokens(T, mode):
    L = synth.olmoe_layer(T=T, seed=40 + T)
    x, Wr, Wgu, Wd = _gpu(L)
    y, dbg = B.elb_moe_forward(x, Wr, Wgu, Wd, K=8, mode=mode, debug=True)
    torch.cuda.synchronize()
    ref = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=8, mode=mode)
    k, ids = cpu(dbg["k"]), cpu(dbg["ids"])
    same = (k == ref.routing.k) & (ids == ref.routing.ids).all(axis=1)
    assert (ref.routing.margin[~same] < NEAR_TIE).all()
    rel = rel_err_rows(cpu(y)[same], ref.y[same])
    print("decode T=%d mode %d: experts used %d, max rel %.3e" % (
        T, mode, len(np.unique(ids[ids >= 0])), rel.max()))
    assert rel.max() < RTOL_BF16


def _experts(L, k, ids, w, residual=None):
    x, _, Wgu, Wd = _gpu(L)
    res = None if residual is None else to_gpu(residual, BF)
    y = B.elb_moe_experts(x, Wgu, Wd, to_gpu(k, torch.int32), to_gpu(ids, torch.int32),
                          to_gpu(w), residual=res)
    torch.cuda.synchronize()
    ref = O.moe_experts(L.x, L.W_gu, L.W_down, k, ids, w.astype(np.float64),
                        residual=residual)
    return rel_err_rows(cpu(y), ref)


def test_experts_decode_crowded_expert_chunks():
    """One expert receives every token (100 rows: four 32-row chunks, the last ragged),
    the rest spread thinly; a residual is added."""
    T, N, K = 100, 64, 2
    L = synth.moe_layer(T, 256, N, 192, dtype="bf16", seed=41)
    rng = np.random.default_rng(41)
    ids = np.stack([np.full(T, 3), (np.arange(T) * 7 + 5) % N], axis=1).astype(np.int32)
    ids[ids[:, 1] == 3, 1] = 4
    k = np.where(np.arange(T) % 3 == 0, 1, 2).astype(np.int32)
    ids[k == 1, 1] = -1
    w = rng.uniform(0.1, 1.0, (T, K)).astype(np.float32)
    w[k == 1, 1] = 0
    res = synth.round_bf16(synth.gaussian_logits(T, 256, seed=42))
    rel = _experts(L, k, ids, w, residual=res)
    print("crowded expert: max rel %.3e" % rel.max())
    assert rel.max() < RTOL_BF16


@pytest.mark.parametrize("T,d,N,m,K", [(7, 64, 8, 64, 3), (33, 320, 16, 192, 4),
                                         (16, 128, 64, 64, 1)])
def test_experts_decode_shapes(T, d, N, m, K):
    """Small widths: m = 192 (six gate/up tasks of 32 columns), d = 320 (five down tasks of
    64 columns), a single 64-deep stage (d = 64 or m = 64), K = 1."""
    L = synth.moe_layer(T, d, N, m, dtype="bf16", seed=T + d)
    r = O.route(O.router_logits(L.x, L.W_router).astype(np.float32), K=K)
    rel = _experts(L, r.k, r.ids, r.w.astype(np.float32))
    print("shape T=%d d=%d N=%d m=%d K=%d: max rel %.3e" % (T, d, N, m, K, rel.max()))
    assert rel.max() < RTOL_BF16


@pytest.mark.parametrize("T", [1, 64, 128])
def test_forward_decode_packed_weights_bit_identical(T):
    """The packed copy of the weights gives the same bits as the row-major weights (same
    operands, same accumulation order), and parity with the oracle."""
    L = synth.olmoe_layer(T=T, seed=50 + T)
    x, Wr, Wgu, Wd = _gpu(L)
    packed = B.elb_pack_expert_weights(Wgu, Wd)
    assert packed.numel() == (Wgu.numel() + Wd.numel()) * 2
    y0 = B.elb_moe_forward(x, Wr, Wgu, Wd, K=8)
    y1, dbg = B.elb_moe_forward(x, Wr, Wgu, Wd, K=8, packed=packed, debug=True)
    torch.cuda.synchronize()
    assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
    ref = O.moe_forward(L.x, L.W_router, L.W_gu, L.W_down, K=8)
    k, ids = cpu(dbg["k"]), cpu(dbg["ids"])
    same = (k == ref.routing.k) & (ids == ref.routing.ids).all(axis=1)
    assert (ref.routing.margin[~same] < NEAR_TIE).all()
    assert rel_err_rows(cpu(y1)[same], ref.y[same]).max() < RTOL_BF16


@pytest.mark.parametrize("T,d,N,m,K", [(7, 64, 8, 64, 3), (33, 320, 16, 192, 4)])
def test_experts_decode_packed_small_widths(T, d, N, m, K):
    L = synth.moe_layer(T, d, N, m, dtype="bf16", seed=T + d + 1)
    r = O.route(O.router_logits(L.x, L.W_router).astype(np.float32), K=K)
    x, _, Wgu, Wd = _gpu(L)
    packed = B.elb_pack_expert_weights(Wgu, Wd)
    args = (to_gpu(r.k, torch.int32), to_gpu(r.ids, torch.int32),
            to_gpu(r.w.astype(np.float32)))
    y0 = B.elb_moe_experts(x, Wgu, Wd, *args)
    y1 = B.elb_moe_experts(x, Wgu, Wd, *args, packed=packed)
    torch.cuda.synchronize()
    assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
