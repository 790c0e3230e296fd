"""Shared helpers for the GPU parity tests (comparison rules of the parity contract).

Routing: k and expert ids must equal the oracle's bit for bit on every token whose oracle
deviation margin is at least NEAR_TIE (1e-6); tokens below it are near-ties, counted and
reported, and may differ.  Weights: relative 1e-5.  Layer outputs: per-token relative L2
error <= 1e-4 (fp32) or 2e-2 (bf16) against the fp64 oracle.
"""
import numpy as np
import torch

NEAR_TIE = 1e-6
RTOL_F32 = 1e-4
RTOL_BF16 = 2e-2


def dev():
    return torch.device("cuda:0")


def to_gpu(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev()).to(dtype)


def cpu(t):
    return t.detach().float().cpu().numpy() if t.is_floating_point() else t.cpu().numpy()


def compare_routing(k, ids, w, ref, label=""):
    """GPU (k, ids, w) vs an oracle Routing; returns (near-tie count, mismatches)."""
    k, ids, w = cpu(k), cpu(ids), cpu(w)
    near = ref.margin < NEAR_TIE
    mism = (k != ref.k) | (ids != ref.ids).any(axis=1)
    bad = mism & ~near
    assert not bad.any(), "%s: %d routing mismatches outside near-ties, first tokens %s" % (
        label, int(bad.sum()), np.nonzero(bad)[0][:8].tolist())
    ok = ~mism
    np.testing.assert_allclose(w[ok], ref.w[ok], rtol=1e-5, atol=1e-7)
    print("%s: tokens %d, near-ties %d, near-tie mismatches %d, mean k %.4f" % (
        label, len(k), int(near.sum()), int(mism.sum()), float(k.mean())))
    return int(near.sum()), int(mism.sum())


def rel_err_rows(y, ref):
    y = np.asarray(y, np.float64)
    num = np.linalg.norm(y - ref, axis=1)
    den = np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
    return num / den
