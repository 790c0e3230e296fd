"""GPU: the calibration kernels behind the bench's measured ceilings (not part of the layer).

The read stream reads every 16-byte chunk of its buffer exactly once, so the XOR of the words
it writes (one per wave) must equal the XOR of every 32-bit word of the buffer, whatever the
grid; sizes include a ragged tail past the four-loads-per-lane loop.  The MFMA loop must
return its instruction count and finite per-wave sums."""
import numpy as np
import pytest
import torch

from paper_2608_04401_amd import binding as B

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes,blocks", [(16, 1), (4096, 1), (1 << 20, 8),
                                           ((1 << 22) + 48, 37), ((1 << 26) + 16 * 1001, 2048)])
def test_read_stream_reads_every_chunk_once(nbytes, blocks):
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes)
    buf = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), generator=g, dtype=torch.int32,
                        device="cuda")
    out = torch.empty(blocks * 4, dtype=torch.int32, device="cuda")
    B.elb_calibrate_read_stream(buf, blocks, out)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(buf.cpu().numpy().view(np.uint32))
    assert got == want


def test_mfma_loop_counts_and_finishes():
    n = B.elb_calibrate_mfma_bf16(8, 10)
    torch.cuda.synchronize()
    assert n == 8 * 4 * 10 * 8
