"""GPU: the layer captured in a HIP graph (torch.cuda.CUDAGraph over the C-ABI calls) and
replayed.  No entry point allocates, synchronises or records a memset, so a captured call is
the same kernel sequence as an eager one: every replay must give the eager result bit for
bit.  Between replays the static input is overwritten in place and eager layer calls on
other inputs run on the same stream (they reuse the workspace the graph was captured with),
so each replay is checked against a fresh eager call on the new input.

Cases cover each path the forward takes by size: the OLMoE-shaped prefill layer (split
router, histogram-fed dispatch, large-tile GEMMs with remainder blocks), the decode-sized
layer (small-batch router, weight-streaming GEMMs, packed weights too), a mid-sized layer
with other expert counts (fused router + routing, count/scatter dispatch, 128-row GEMMs) and
the allocation-free entry point."""
import pytest
import torch

from paper_2608_04401_amd import binding as B
from paper_2608_04401_amd import synth

pytestmark = pytest.mark.gpu


def _same(a, b):
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def _replays(fwd, x, label, reps=3):
    """Capture fwd(x, out) once, then replay it on `reps` new inputs written into x."""
    T, d = x.shape
    inputs = [synth.device_normal_bf16((T, d), 100 + r, 1.0) for r in range(reps)]
    other = synth.device_normal_bf16((T, d), 99, 1.0)
    out = torch.empty_like(x)
    fwd(x, out)  # eager first: one-time per-device lookups happen outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fwd(x, out)
    torch.cuda.synchronize()
    for r in range(reps):
        x.copy_(inputs[r])
        g.replay()
        y_other = fwd(other, torch.empty_like(other))  # eager work between replays
        torch.cuda.synchronize()
        got = out.clone()
        ref = fwd(inputs[r].clone(), torch.empty_like(x))
        torch.cuda.synchronize()
        assert _same(got, ref), "%s: replay %d differs from the eager call" % (label, r)
        assert not _same(got, y_other), "%s: replay %d did not read the new input" % (label, r)
    print("%s: %d replays identical to eager calls (T %d)" % (label, reps, T))


def test_prefill_and_decode_layer_replay_in_a_graph():
    """OLMoE-shaped layer (d = 2048, N = 64, intermediate 1024, bf16): T = 4096 in elbow and
    top-8 mode, then T = 64 with row-major and with packed expert weights."""
    Wr, Wgu, Wd = synth.device_stack_layer(0)
    for mode, name in ((B.MODE_ELBOW, "elbow"), (B.MODE_TOPK, "top-8")):
        fwd = lambda xx, oo, mode=mode: B.elb_moe_forward(xx, Wr, Wgu, Wd, K=8, mode=mode,
                                                          out=oo)
        _replays(fwd, synth.device_stack_input(4096, 2048), "prefill " + name)
    fwd = lambda xx, oo: B.elb_moe_forward(xx, Wr, Wgu, Wd, K=8, out=oo)
    _replays(fwd, synth.device_stack_input(64, 2048), "decode")
    packed = B.elb_pack_expert_weights(Wgu, Wd)
    fwd = lambda xx, oo: B.elb_moe_forward(xx, Wr, Wgu, Wd, K=8, out=oo, packed=packed)
    _replays(fwd, synth.device_stack_input(64, 2048), "decode packed")


def test_mid_sized_layer_replays_in_a_graph():
    """T = 1000, d = 512, N = 32, m = 256, K = 4, bf16, with a residual."""
    T, d, N, m = 1000, 512, 32, 256
    Wr = synth.device_normal_bf16((N, d), 1, 0.02)
    Wgu = synth.device_normal_bf16((N, 2 * m, d), 2, 0.02)
    Wd = synth.device_normal_bf16((N, d, m), 3, 0.02)
    res = synth.device_normal_bf16((T, d), 4, 1.0)
    fwd = lambda xx, oo: B.elb_moe_forward(xx, Wr, Wgu, Wd, K=4, residual=res, out=oo)
    _replays(fwd, synth.device_normal_bf16((T, d), 5, 1.0), "mid-sized")


def test_noalloc_entry_point_replays_in_a_graph():
    """The allocation-free entry point (its static scratch) on the prefill-sized layer."""
    Wr, Wgu, Wd = synth.device_stack_layer(0)
    fwd = lambda xx, oo: B.elb_moe_forward_noalloc(xx, Wr, Wgu, Wd, K=8, out=oo)
    _replays(fwd, synth.device_stack_input(4096, 2048), "noalloc prefill")
