"""GPU parity of the 16-layer residual stack at full size: 16 OLMoE-shaped layers (d=2048,
N=64 experts, SwiGLU intermediate 1024, bf16), T=16384 tokens, h <- h + MoE_l(h), elbow
routing capped at K=8.  Every layer runs on all 16384 tokens; a seeded sample of tokens is
checked against the fp64 oracle layer by layer on the same input (teacher-forced: the oracle
layer gets the GPU's bf16 input rows, since tokens are independent through the stack and one
near-tie flip would change every later layer).  Weights are drawn on the device
(synth.device_stack_layer); the oracle reads host copies of the same tensors."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

from helpers import NEAR_TIE, RTOL_BF16, cpu, rel_err_rows

pytestmark = pytest.mark.gpu

T, D, N, M, K, LAYERS = 16384, 2048, 64, 1024, 8, 16


def test_residual_stack_16_layers_sampled():
    rng = np.random.default_rng(16)
    sample = np.sort(rng.choice(T, 24, replace=False))
    sample_t = torch.from_numpy(sample).cuda()
    h = synth.device_stack_input(T, D)
    worst, near_total, ks = 0.0, 0, []
    for l in range(LAYERS):
        Wr, Wgu, Wd = synth.device_stack_layer(l, D, N, M)
        y, dbg = B.elb_moe_forward(h, Wr, Wgu, Wd, K=K, residual=h, debug=True)
        torch.cuda.synchronize()
        k = cpu(dbg["k"])
        assert ((k >= 1) & (k <= K)).all()
        ks.append(float(k.mean()))
        hs = cpu(h.index_select(0, sample_t))
        ref = O.moe_forward(hs, cpu(Wr), cpu(Wgu), cpu(Wd), K=K, residual=hs)
        near = ref.routing.margin < NEAR_TIE
        rel = rel_err_rows(cpu(y.index_select(0, sample_t)), ref.y)
        assert rel[~near].max() < RTOL_BF16, "layer %d: max rel err %.3g" % (l, rel[~near].max())
        gk = k[sample]
        assert np.array_equal(gk[~near], ref.routing.k[~near]), "layer %d: k differs" % l
        worst = max(worst, float(rel[~near].max()))
        near_total += int(near.sum())
        h = y
        del Wr, Wgu, Wd, dbg
    print("16-layer stack: sampled tokens %d per layer, max rel err %.2e, near-ties %d, "
          "mean k per layer %s" % (len(sample), worst, near_total,
                                   " ".join("%.3f" % v for v in ks)))
