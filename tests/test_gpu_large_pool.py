"""64-bit addressing: the same sequences with their pages moved to the top of a
pool larger than 4 GiB give bit-identical attention outputs (page-permutation
invariance) and write the new K/V to the same slots of the moved pages.  Covers
the extend kernel's DMA, the decode kernel, the fused page writes of both, the
stand-alone page write and the page swap."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import paper_2606_16824_amd as cwlib
from gpu_util import bits, to_gpu

pytestmark = pytest.mark.gpu

BIG_BYTES = 6 << 30  # each of the K and V pools


def _moved(dw, offset, num_big):
    """Pools of num_big pages holding dw's pages at ids + offset (the rest never read)."""
    kp = torch.empty((num_big,) + tuple(dw.k_pool.shape[1:]), dtype=dw.k_pool.dtype, device="cuda")
    vp = torch.empty_like(kp)
    n = dw.k_pool.shape[0]
    kp[offset:offset + n] = dw.k_pool
    vp[offset:offset + n] = dw.v_pool
    ks = vs = None
    if dw.k_scale is not None:
        ks = torch.ones((num_big,) + tuple(dw.k_scale.shape[1:]), dtype=torch.float32, device="cuda")
        vs = torch.ones_like(ks)
        ks[offset:offset + n] = dw.k_scale
        vs[offset:offset + n] = dw.v_scale
    bt = dw.block_table.clone()
    used = bt != torch.iinfo(torch.int32).max
    bt[used] += offset
    return kp, vp, ks, vs, bt


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_pages_past_4gib(kv):
    # two extends and two decodes: the step runs both kernels and fuses the page write
    spec = cw.custom_spec([3000, 700, 4000, 33], [50, 1, 130, 1], num_kv_heads=8, gqa_group=4,
                          head_dim=128, page_size=16, kv_dtype=kv, seed=77)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    page_bytes = dw.k_pool[0].numel() * dw.k_pool.element_size()
    num_big = BIG_BYTES // page_bytes
    offset = num_big - spec.num_pages
    print(f"\n[case] large pool {kv}: {num_big} pages of {page_bytes} B, pages moved by {offset}",
          flush=True)
    assert offset * page_bytes > (4 << 30)
    s = spec
    outs, pools = [], []
    for moved in (False, True):
        if moved:
            kp, vp, ks, vs, bt = _moved(dw, offset, num_big)
        else:
            kp, vp, ks, vs, bt = (dw.k_pool.clone(), dw.v_pool.clone(), dw.k_scale, dw.v_scale,
                                  dw.block_table)
        out = torch.full_like(dw.q, float("nan"))
        lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device="cuda")
        cwlib.step_attention(dw.q, dw.k_new, dw.v_new, kp, vp, bt, s.prefix_lens, s.suffix_lens,
                             s.gqa_group, s.softmax_scale, k_scale=ks, v_scale=vs, out=out, lse=lse)
        torch.cuda.synchronize()
        lo = offset if moved else 0
        outs.append((bits(out), lse.cpu().numpy().view(np.uint32)))
        pools.append((kp[lo:lo + s.num_pages].cpu(), vp[lo:lo + s.num_pages].cpu()))
        del kp, vp
        torch.cuda.empty_cache()
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    raw = lambda t: t.view(torch.uint8) if t.dtype != torch.uint8 else t
    assert torch.equal(raw(pools[0][0]), raw(pools[1][0]))
    assert torch.equal(raw(pools[0][1]), raw(pools[1][1]))


def test_swap_and_write_past_4gib():
    spec = cw.custom_spec([900, 20], [40, 3], num_kv_heads=8, gqa_group=4, head_dim=128,
                          page_size=16, kv_dtype="bf16", seed=78)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    page_bytes = dw.k_pool[0].numel() * dw.k_pool.element_size()
    num_big = BIG_BYTES // page_bytes
    offset = num_big - spec.num_pages
    print(f"\n[case] large pool write + swap: pages moved by {offset}", flush=True)
    kp, vp, _, _, bt = _moved(dw, offset, num_big)
    cwlib.kv_write_pages(dw.k_new, dw.v_new, kp, vp, bt, spec.prefix_lens, spec.suffix_lens)
    kw, vw = dw.k_pool.clone(), dw.v_pool.clone()
    cwlib.kv_write_pages(dw.k_new, dw.v_new, kw, vw, dw.block_table, spec.prefix_lens,
                         spec.suffix_lens)
    torch.cuda.synchronize()
    n = spec.num_pages
    assert torch.equal(kp[offset:offset + n].cpu().view(torch.int16), kw.cpu().view(torch.int16))
    assert torch.equal(vp[offset:offset + n].cpu().view(torch.int16), vw.cpu().view(torch.int16))
    # swap the moved pages out to a host pool and back into other high pages
    pages = (torch.arange(n, dtype=torch.int32) + offset).numpy()
    hk = torch.empty((n,) + tuple(kp.shape[1:]), dtype=kp.dtype).pin_memory()
    hv = torch.empty_like(hk).pin_memory()
    host = np.arange(n, dtype=np.int32)
    cwlib.kv_swap_out(kp, vp, hk, hv, pages, host)
    torch.cuda.synchronize()
    assert torch.equal(hk.view(torch.int16), kw.cpu().view(torch.int16))
    dst = (np.arange(n, dtype=np.int32) + offset - n)  # the n pages just below
    cwlib.kv_swap_in(hk, hv, kp, vp, host, dst)
    torch.cuda.synchronize()
    assert torch.equal(kp[offset - n:offset].cpu().view(torch.int16), kw.cpu().view(torch.int16))
    assert torch.equal(vp[offset - n:offset].cpu().view(torch.int16), vw.cpu().view(torch.int16))
