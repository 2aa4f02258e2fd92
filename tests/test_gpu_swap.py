"""GPU page swaps (cw_kv_swap_out / cw_kv_swap_in) against the oracle, bit for bit.

The host block pools are pinned host tensors, written and read by the kernel
over the host link."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_16824_amd as cwlib

pytestmark = pytest.mark.gpu

# (pool pages, host blocks, kv heads, head dim, page size, dtype, entries)
CASES = {
    "bf16_d128_p16": (300, 64, 8, 128, 16, "bf16", 50),
    "bf16_d64_p64": (97, 40, 3, 64, 64, "bf16", 40),
    "fp8_d128_p16": (200, 33, 2, 128, 16, "fp8", 33),
    "fp8_d64_p64": (50, 12, 1, 64, 64, "fp8", 7),
}


def _pools(n, hkv, d, p, dt, seed, pinned):
    g = np.random.default_rng(seed)
    elem = np.uint16 if dt == "bf16" else np.uint8
    k = g.integers(0, np.iinfo(elem).max + 1, size=(n, hkv, p, d), dtype=np.int64).astype(elem)
    v = g.integers(0, np.iinfo(elem).max + 1, size=(n, hkv, p, d), dtype=np.int64).astype(elem)
    ks = g.random((n, hkv), dtype=np.float32) if dt == "fp8" else None
    vs = g.random((n, hkv), dtype=np.float32) if dt == "fp8" else None

    def t(a):
        if a is None:
            return None
        x = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a)
        if dt == "bf16" and a.dtype == np.uint16:
            x = x.view(torch.bfloat16)
        return x.pin_memory() if pinned else x.cuda()
    return (k, v, ks, vs), tuple(t(a) for a in (k, v, ks, vs))


def _np(t):
    if t is None:
        return None
    t = t.cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


@pytest.mark.parametrize("name", list(CASES))
def test_swap_out_then_in_matches_oracle(name):
    n_pages, n_host, hkv, d, p, dt, n = CASES[name]
    print(f"\n[case] swap {name}: pool {n_pages}, host {n_host}, hkv {hkv}, D {d}, P {p}, {dt}, {n} entries",
          flush=True)
    g = np.random.default_rng(len(name))
    (k, v, ks, vs), (dk, dv, dks, dvs) = _pools(n_pages, hkv, d, p, dt, 1, pinned=False)
    (hk, hv, hks, hvs), (thk, thv, thks, thvs) = _pools(n_host, hkv, d, p, dt, 2, pinned=True)
    pages = g.choice(n_pages, size=n, replace=False)
    pages[1] = pages[0] if n > 2 else pages[1]  # a repeated source page is allowed
    host = g.permutation(n_host)[:n]
    cwlib.kv_swap_out(dk, dv, thk, thv, pages, host, k_scale=dks, v_scale=dvs, k_scale_host=thks,
                      v_scale_host=thvs)
    torch.cuda.synchronize()
    want = oracle.swap_out(k, v, ks, vs, pages, hk, hv, hks, hvs, host)
    for got, exp, what in zip((thk, thv, thks, thvs), want, ("K", "V", "K scale", "V scale")):
        if exp is None:
            continue
        nbad = int((_np(got) != exp).sum())
        print(f"[{name}] swap-out {what}: {nbad} differing elements", flush=True)
        assert nbad == 0
    # back into a different set of pool pages
    new_pages = g.choice(n_pages, size=n, replace=False)
    cwlib.kv_swap_in(thk, thv, dk, dv, host, new_pages, k_scale_host=thks, v_scale_host=thvs,
                     k_scale=dks, v_scale=dvs)
    torch.cuda.synchronize()
    want_in = oracle.swap_in(*want[:2], want[2], want[3], host, k, v, ks, vs, new_pages)
    for got, exp, what in zip((dk, dv, dks, dvs), want_in, ("K", "V", "K scale", "V scale")):
        if exp is None:
            continue
        nbad = int((_np(got) != exp).sum())
        print(f"[{name}] swap-in {what}: {nbad} differing elements", flush=True)
        assert nbad == 0


def test_turn_prefix_round_trip():
    # every prefix page of the turn workload (1024 pages of 8 kv heads, 32 KiB of
    # K and of V each) out to the host and back into a permuted set of pages
    import cw_workloads as cw
    spec = cw.spec_for("turn")
    w = cw.materialize(spec)
    n = int(spec.prefix_lens[0]) // spec.page_size
    pages = w.block_table[0, :n].numpy().astype(np.int32)
    print(f"\n[case] swap turn prefix: {n} pages", flush=True)
    dk, dv = w.k_pool.cuda(), w.v_pool.cuda()
    hk = torch.empty((n,) + tuple(dk.shape[1:]), dtype=dk.dtype).pin_memory()
    hv = torch.empty_like(hk).pin_memory()
    cwlib.kv_swap_out(dk, dv, hk, hv, pages, np.arange(n))
    torch.cuda.synchronize()
    idx = torch.from_numpy(pages).long()
    assert torch.equal(hk.view(torch.int16), w.k_pool[idx].view(torch.int16))
    assert torch.equal(hv.view(torch.int16), w.v_pool[idx].view(torch.int16))
    free = np.setdiff1d(np.arange(dk.shape[0]), w.block_table[0].numpy())[:n].astype(np.int32)
    assert len(free) == n
    cwlib.kv_swap_in(hk, hv, dk, dv, np.arange(n), free)
    torch.cuda.synchronize()
    fidx = torch.from_numpy(free).long().cuda()
    assert torch.equal(dk[fidx].cpu().view(torch.int16), w.k_pool[idx].view(torch.int16))
    assert torch.equal(dv[fidx].cpu().view(torch.int16), w.v_pool[idx].view(torch.int16))


def test_pageable_host_memory_is_rejected_before_launch():
    import paper_2606_16824_amd._lib as L
    lib = cwlib.library()
    dk = torch.zeros((4, 1, 16, 64), dtype=torch.bfloat16, device="cuda")
    pageable = np.zeros((4, 1, 16, 64), dtype=np.uint16)  # plain host memory, not device-mapped
    pages = np.array([0, 1], dtype=np.int32)
    host = np.array([2, 3], dtype=np.int32)
    ws = torch.empty(cwlib.swap_workspace_bytes(2), dtype=torch.uint8, device="cuda")
    st = lib.cw_kv_swap_out(dk.data_ptr(), dk.data_ptr(), None, None, 4, pageable.ctypes.data,
                            pageable.ctypes.data, None, None, 4, pages.ctypes.data, host.ctypes.data,
                            2, 1, 64, 16, 0, ws.data_ptr(), ws.numel(), None)
    assert st == L.CW_ERR_UNSUPPORTED, lib.cw_last_error_message()
    with pytest.raises(ValueError):  # the binding refuses unpinned host tensors itself
        cwlib.kv_swap_out(dk, dk, torch.zeros(4, 1, 16, 64, dtype=torch.bfloat16),
                          torch.zeros(4, 1, 16, 64, dtype=torch.bfloat16), [0], [0])
