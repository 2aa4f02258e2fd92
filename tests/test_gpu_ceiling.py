"""The measurement kernels behind the bench's measured ceilings compute what they
claim: the MFMA loop runs every round of its four chains (closed-form sum for the
low-entropy operands, a float64 product of the hashed operands for the random ones), the
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
    flops = cwlib.ceiling_mfma_bf16(wgs, iters, sink, random=False)
    torch.cuda.synchronize()
    assert flops == wgs * 8 * iters * 131072
    # operands a = ((lane + e) & 7) / 1024, b = ((3 lane + e) & 7) / 1024: row r of A times
    # column 0 of B is 2 sum_e ((r + e) & 7) e / 2^20; lane 0 sums rows 0..3 of its four
    # chains (280 + 224 + 184 + 160 per round), exactly representable
    want = np.float32(848 * iters / 2.0 ** 20)
    got = sink.cpu().numpy()
    assert np.all(got == want), (got[:4], want)


def _mix32(x):
    x = np.asarray(x, dtype=np.uint64)
    m = np.uint64(0xFFFFFFFF)
    x ^= x >> np.uint64(16)
    x = (x * np.uint64(0x7FEB352D)) & m
    x ^= x >> np.uint64(15)
    x = (x * np.uint64(0x846CA68B)) & m
    x ^= x >> np.uint64(16)
    return x


def _bf16_value(u):
    """Value of the bf16 whose bits are (u >> 31) << 15 | (123 + (u >> 8) % 6) << 7 | (u & 127)."""
    sign = np.where((u >> np.uint64(31)) & np.uint64(1), -1.0, 1.0)
    expo = 123 + ((u >> np.uint64(8)) % np.uint64(6)).astype(np.int64)
    mant = (u & np.uint64(127)).astype(np.float64)
    return sign * (1.0 + mant / 128.0) * 2.0 ** (expo - 127)


def test_mfma_loop_random_operands():
    wgs, iters = 37, 1000
    sink = torch.full((wgs * 8,), np.nan, dtype=torch.float32, device="cuda")
    assert cwlib.ceiling_mfma_bf16(wgs, iters, sink, random=True) == wgs * 8 * iters * 131072
    torch.cuda.synchronize()
    got = sink.cpu().numpy().astype(np.float64)
    # wave w's lane 0 is global lane 64 w; chain c's A row c sits in lanes c and c + 32
    # (k = 8 * half + e), B column 0 in lanes 0 and 32
    want = np.zeros(wgs * 8)
    scale = np.zeros(wgs * 8)
    w = np.arange(wgs * 8, dtype=np.uint64)
    for c in range(4):
        for half in range(2):
            for e in range(8):
                ga = 64 * w + np.uint64(c + 32 * half)
                gb = 64 * w + np.uint64(32 * half)
                a = _bf16_value(_mix32(np.uint64(64) * ga + np.uint64(8 * c + e)))
                hb = _mix32(np.uint64(64) * gb + np.uint64(8 * c + e))
                b = _bf16_value(_mix32(hb ^ np.uint64(0x9E3779B9)))
                want += iters * a * b
                scale += iters * np.abs(a * b)
    assert np.all(np.isfinite(got))
    assert np.all(np.abs(got - want) <= 2e-4 * scale + 1e-6), np.max(np.abs(got - want) / scale)


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
