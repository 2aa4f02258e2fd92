"""The measurement kernels behind the bench's measured ceilings compute what they
claim: the MFMA loop runs every round of its four chains (closed-form sum), the
streaming read sees every word (XOR of the sinks equals the buffer's XOR) and the
streaming copy moves every byte, for sizes that leave a ragged tail."""
import numpy as np
import pytest
import torch

import paper_2606_16824_amd as cwlib

pytestmark = pytest.mark.gpu


def test_mfma_loop_runs_every_round():
    wgs, iters = 300, 1000
    sink = torch.full((wgs * 8,), -1.0, dtype=torch.float32, device="cuda")
    flops = cwlib.ceiling_mfma_bf16(wgs, iters, sink)
    torch.cuda.synchronize()
    assert flops == wgs * 8 * iters * 131072
    # operands a = ((lane + e) & 7) / 1024, b = ((3 lane + e) & 7) / 1024: row r of A times
    # column 0 of B is 2 sum_e ((r + e) & 7) e / 2^20; lane 0 sums rows 0..3 of its four
    # chains (280 + 224 + 184 + 160 per round), exactly representable
    want = np.float32(848 * iters / 2.0 ** 20)
    got = sink.cpu().numpy()
    assert np.all(got == want), (got[:4], want)


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (64 << 20) + 16 * 7])
def test_stream_read_sees_every_word(nbytes):
    g = torch.Generator().manual_seed(nbytes)
    host = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g)
    src = host.cuda()
    sink = torch.zeros(16384, dtype=torch.int32, device="cuda")
    assert cwlib.ceiling_stream_read(src, sink) == nbytes
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(host.numpy().view(np.uint32))
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == want


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (64 << 20) + 16 * 7])
def test_stream_copy_moves_every_byte(nbytes):
    g = torch.Generator().manual_seed(nbytes + 1)
    host = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g)
    src = host.cuda()
    dst = torch.zeros(nbytes + 64, dtype=torch.uint8, device="cuda")
    assert cwlib.ceiling_stream_copy(src, dst[:nbytes]) == 2 * nbytes
    torch.cuda.synchronize()
    out = dst.cpu()
    assert torch.equal(out[:nbytes], host)
    assert int(out[nbytes:].sum()) == 0  # nothing written past the end
