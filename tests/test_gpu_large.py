"""GPU parity of the expert stage at sizes whose byte offsets pass 2^32.

The large-tile grouped GEMM adds a 32-bit per-lane byte offset to a 64-bit base.  These tests
run problems where a flat offset from the start of a tensor would wrap:
  - the down GEMM's H rows past 4 GiB (T K m 2 bytes > 2^32, on the large-tile path), and
  - gathered x rows past 4 GiB (T d 2 bytes > 2^32, which the library must hand to its
    64-bit-addressed kernel),
and compare the output rows whose operands lie beyond 2^32 bytes (plus a random sample)
with the fp64 oracle.  Inputs are drawn on the device from seeded generators; the oracle
reads host copies of the rows it checks."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_04401_amd import binding as B

from helpers import RTOL_BF16, cpu, rel_err_rows

pytestmark = pytest.mark.gpu
BF = torch.bfloat16


def _normal(shape, std, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device="cuda", dtype=torch.float32) * std).to(BF)


def _run(T, d, N, m, seed, pick):
    x = _normal((T, d), 1.0, seed)
    Wgu = _normal((N, 2 * m, d), 0.02, seed + 1)
    Wd = _normal((N, d, m), 0.02, seed + 2)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed + 3)
    ids = torch.randint(0, N, (T, 1), generator=g, device="cuda", dtype=torch.int32)
    k = torch.ones(T, dtype=torch.int32, device="cuda")
    w = torch.rand((T, 1), generator=g, device="cuda", dtype=torch.float32) * 0.8 + 0.2
    y = B.elb_moe_experts(x, Wgu, Wd, k, ids, w)
    torch.cuda.synchronize()
    ids_h = cpu(ids)[:, 0]
    tok = pick(ids_h)
    tok_t = torch.from_numpy(tok).cuda()
    xs = cpu(x.index_select(0, tok_t))
    ref = O.moe_experts(xs, cpu(Wgu), cpu(Wd), np.ones(len(tok), np.int32),
                        ids_h[tok, None].astype(np.int32),
                        cpu(w)[tok].astype(np.float64))
    rel = rel_err_rows(cpu(y.index_select(0, tok_t)), ref)
    del x, Wgu, Wd, y
    torch.cuda.empty_cache()
    return tok, rel


def test_down_gemm_h_rows_past_4gib():
    """d = 128, m = 4096, N = 8, K = 1, T = 600000: H holds T m bf16 = 4.9 GB, and the rows of
    the last expert (expert-major order) start past 2^31 / m = 524288 rows."""
    T, d, N, m = 600_000, 128, 8, 4096
    rng = np.random.default_rng(0)

    def pick(ids_h):
        last = np.nonzero(ids_h == N - 1)[0]       # every one of their H rows is past 2^32 B
        return np.unique(np.concatenate([rng.choice(last, 384, replace=False),
                                         rng.choice(T, 128, replace=False)]))
    tok, rel = _run(T, d, N, m, 11, pick)
    print("H past 4 GiB: %d tokens, max rel %.3e" % (len(tok), rel.max()))
    assert rel.max() < RTOL_BF16


def test_gate_up_gathered_x_past_4gib():
    """d = 2048, m = 128, N = 8, K = 1, T = 2^20 + 192: x holds T d bf16 > 2^32 bytes, so the
    last 192 tokens' rows start past 2^32 bytes; every one of them is checked."""
    T, d, N, m = (1 << 20) + 192, 2048, 8, 128
    rng = np.random.default_rng(1)

    def pick(ids_h):
        return np.unique(np.concatenate([np.arange(1 << 20, T),
                                         rng.choice(T, 128, replace=False)]))
    tok, rel = _run(T, d, N, m, 21, pick)
    print("x past 4 GiB: %d tokens, max rel %.3e" % (len(tok), rel.max()))
    assert rel.max() < RTOL_BF16
