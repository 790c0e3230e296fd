"""GPU: the allocation-free entry point (elb_moe_forward_noalloc, the library's static scratch)
against elb_moe_forward with a caller workspace, through the C ABI.  The two share every
kernel, so the outputs and every debug output must be identical bit for bit; the calls run
in a row on one GPU, the second on a smaller input (the scratch keeps the first call's
contents), the third on the prefill-sized input again."""
import pytest
import torch

from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

pytestmark = pytest.mark.gpu


def _same(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a, b)


def _check(x, Wr, Wgu, Wd, mode, label):
    y_ref, d_ref = B.elb_moe_forward(x, Wr, Wgu, Wd, K=8, mode=mode, debug=True)
    y, d = B.elb_moe_forward_noalloc(x, Wr, Wgu, Wd, K=8, mode=mode, debug=True)
    torch.cuda.synchronize()
    assert _same(y, y_ref), label + ": y differs"
    for name in ("logits", "k", "ids", "w", "counts"):
        assert _same(d[name], d_ref[name]), "%s: %s differs" % (label, name)
    print("%s: T %d identical (mean k %.4f)" % (label, x.shape[0], d["k"].float().mean()))


def test_noalloc_matches_forward_on_consecutive_calls():
    """OLMoE-shaped layer (d = 2048, N = 64, intermediate 1024, bf16): T = 4096 (the largest
    input run here; 207 MB of the 256 MiB scratch), then T = 64 (the decode-sized kernels,
    reading a scratch that still holds the first call's data), then T = 4096 in top-8 mode."""
    Wr, Wgu, Wd = synth.device_stack_layer(0)
    x = synth.device_stack_input(4096, 2048)
    _check(x, Wr, Wgu, Wd, B.MODE_ELBOW, "prefill")
    _check(x[:64].contiguous(), Wr, Wgu, Wd, B.MODE_ELBOW, "decode")
    _check(x, Wr, Wgu, Wd, B.MODE_TOPK, "prefill top-8")


def test_noalloc_rejects_oversized_problem():
    Wr, Wgu, Wd = synth.device_stack_layer(1)
    x = synth.device_stack_input(8192, 2048)
    with pytest.raises(B.ElbError) as ei:
        B.elb_moe_forward_noalloc(x, Wr, Wgu, Wd, K=8)
    assert ei.value.status == 2
