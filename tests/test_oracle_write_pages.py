"""Pins of the oracle's page scatter: a hand-worked case, invariants, torch's fp8 cast."""
import numpy as np
import torch

import cw_workloads as cw
from conftest import paged_inputs
from oracle import PagedInputs, extend_attention_rowwise, write_pages


def test_hand_worked_scatter():
    # P=2, block table [3, 1, 4]; prefix 1, suffix 3 -> positions 1, 2, 3 land in
    # (page 3, slot 1), (page 1, slot 0), (page 1, slot 1).
    kp = np.zeros((5, 1, 2, 2), dtype=np.uint16)
    vp = np.zeros((5, 1, 2, 2), dtype=np.uint16) + 9
    kn = np.array([[[1, 2]], [[3, 4]], [[5, 6]]], dtype=np.uint16)
    vn = kn + 100
    inp = PagedInputs(np.zeros((3, 1, 2), np.uint16), kn, vn, kp, vp,
                      np.array([[3, 1, 4]], np.int32), np.array([1]), np.array([3]), 1, 1.0)
    k2, v2 = write_pages(inp)
    want_k = np.zeros_like(kp)
    want_k[3, 0, 1] = [1, 2]
    want_k[1, 0, 0] = [3, 4]
    want_k[1, 0, 1] = [5, 6]
    assert np.array_equal(k2, want_k)
    want_v = vp.copy()
    want_v[3, 0, 1] = [101, 102]
    want_v[1, 0, 0] = [103, 104]
    want_v[1, 0, 1] = [105, 106]
    assert np.array_equal(v2, want_v)
    assert np.array_equal(kp, np.zeros_like(kp))  # input untouched


def test_scatter_lands_where_gather_reads_and_nothing_else_changes():
    spec = cw.custom_spec([13, 0, 32, 7], [9, 5, 17, 1], num_kv_heads=2, gqa_group=2,
                          head_dim=8, page_size=8, seed=3)
    inp = paged_inputs(cw.materialize(spec, threads=1))
    k2, v2 = write_pages(inp)
    touched = np.zeros(inp.k_pool.shape[:1] + inp.k_pool.shape[2:3], dtype=bool)
    cu = inp.cu()
    for b in range(4):
        lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
        for i in range(ls):
            pos = lp + i
            pg, sl = inp.block_table[b, pos // 8], pos % 8
            assert not touched[pg, sl]  # write slots of different sequences are disjoint
            touched[pg, sl] = True
            assert np.array_equal(k2[pg, :, sl], inp.k_new[cu[b] + i])
            assert np.array_equal(v2[pg, :, sl], inp.v_new[cu[b] + i])
    mask = np.broadcast_to(touched[:, None, :, None], inp.k_pool.shape)
    assert np.array_equal(k2[~mask], inp.k_pool[~mask])
    assert np.array_equal(v2[~mask], inp.v_pool[~mask])


def test_written_pool_serves_as_longer_prefix():
    """Attention over (Lp, Ls) equals attention over (Lp+s, Ls-s) read from the written pool."""
    spec = cw.custom_spec([21], [14], num_kv_heads=1, gqa_group=3, head_dim=16, page_size=4, seed=8)
    inp = paged_inputs(cw.materialize(spec, threads=1))
    full, _ = extend_attention_rowwise(inp)
    k2, v2 = write_pages(inp)
    for s in (1, 3, 4, 13):
        moved = PagedInputs(inp.q[s:], inp.k_new[s:], inp.v_new[s:], k2, v2, inp.block_table,
                            inp.prefix_lens + s, inp.suffix_lens - s, 3, inp.softmax_scale)
        out, _ = extend_attention_rowwise(moved)
        np.testing.assert_allclose(out, full[s:], rtol=1e-13, atol=1e-15)


def test_fp8_quantise_on_write_matches_torch_cast():
    spec = cw.custom_spec([10, 3], [6, 12], num_kv_heads=2, gqa_group=1, head_dim=16,
                          page_size=4, kv_dtype="fp8", seed=12)
    w = cw.materialize(spec, threads=1)
    inp = paged_inputs(w)
    # push some values past the clamp: x / s beyond 448 must saturate, not become NaN
    inp.k_new[0, 0, :4] = torch.tensor([40.0, -40.0, 1e4, -1e4]).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    k2, v2 = write_pages(inp)
    cu = inp.cu()
    for b in range(2):
        lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
        for i in range(ls):
            pos = lp + i
            pg, sl = int(inp.block_table[b, pos // 4]), pos % 4
            for src, dst, sc in ((inp.k_new, k2, inp.k_scale), (inp.v_new, v2, inp.v_scale)):
                x = torch.from_numpy(src[cu[b] + i].view(np.int16)).view(torch.bfloat16).float()
                quot = (x / torch.from_numpy(sc[pg])[:, None]).clamp(-448, 448)
                ref = quot.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
                assert np.array_equal(dst[pg, :, sl], ref)
    assert k2[inp.block_table[0, 10 // 4], 0, 10 % 4, 2] == 0x7E  # +448
    assert k2[inp.block_table[0, 10 // 4], 0, 10 % 4, 3] == 0xFE  # -448
