"""Pins of the oracle's attention against independent references.

The paper prints no worked attention example, so every pin below comes from
mathematics or a library routine: pure-Python brute force on tiny inputs,
torch's scaled_dot_product_attention with an explicit bottom-right causal
mask, closed forms, and the invariances the paged layout must satisfy.
"""
import math
import struct

import numpy as np
import pytest
import torch

import cw_workloads as cw
from oracle import (PagedInputs, decode_attention, extend_attention_blocked,
                    extend_attention_rows, extend_attention_rowwise, extend_attention_token_blocks,
                    gather_sequence_kv)
from conftest import paged_inputs


def _bf16(bits):
    return struct.unpack("<f", struct.pack("<I", int(bits) << 16))[0]


def _fp8(code):
    return float(torch.tensor([int(code)], dtype=torch.uint8).view(torch.float8_e4m3fn).float()[0])


def brute_force(inp: PagedInputs):
    """Pure-Python loops, own page walk and own decoding; float64 via Python floats."""
    P = inp.k_pool.shape[2]
    T, HQ, D = inp.q.shape
    G = inp.gqa_group
    out = np.zeros((T, HQ, D))
    lse = np.zeros((T, HQ))
    row0 = 0
    for b in range(len(inp.prefix_lens)):
        lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
        for i in range(ls):
            for h in range(HQ):
                kvh = h // G
                qv = [_bf16(x) for x in inp.q[row0 + i, h]]
                keys, vals = [], []
                for j in range(lp + i + 1):
                    if j < lp:
                        pg, sl = int(inp.block_table[b][j // P]), j % P
                        if inp.kv_dtype == "bf16":
                            kv = [_bf16(x) for x in inp.k_pool[pg, kvh, sl]]
                            vv = [_bf16(x) for x in inp.v_pool[pg, kvh, sl]]
                        else:
                            ks, vs = float(inp.k_scale[pg, kvh]), float(inp.v_scale[pg, kvh])
                            kv = [_fp8(x) * ks for x in inp.k_pool[pg, kvh, sl]]
                            vv = [_fp8(x) * vs for x in inp.v_pool[pg, kvh, sl]]
                    else:
                        kv = [_bf16(x) for x in inp.k_new[row0 + j - lp, kvh]]
                        vv = [_bf16(x) for x in inp.v_new[row0 + j - lp, kvh]]
                    keys.append(kv)
                    vals.append(vv)
                sc = [inp.softmax_scale * sum(a * c for a, c in zip(qv, kv)) for kv in keys]
                m = max(sc)
                e = [math.exp(s - m) for s in sc]
                tot = sum(e)
                for d in range(D):
                    out[row0 + i, h, d] = sum(e[j] * vals[j][d] for j in range(len(e))) / tot
                lse[row0 + i, h] = m + math.log(tot)
        row0 += ls
    return out, lse


def small(lp, ls, g, d, p=4, hkv=2, kv_dtype="bf16", seed=0, shared=0):
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p,
                          kv_dtype=kv_dtype, seed=seed, shared_prefix_tokens=shared)
    return paged_inputs(cw.materialize(spec, threads=1))


@pytest.mark.parametrize("g", [1, 2, 3, 4])
@pytest.mark.parametrize("d", [4, 8])
def test_brute_force_tiny(g, d):
    inp = small([5, 0, 9, 12], [3, 7, 0, 4], g, d, p=4, seed=g * 10 + d)
    ref, ref_lse = brute_force(inp)
    for fn in (extend_attention_rowwise, extend_attention_blocked):
        out, lse = fn(inp)
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse, ref_lse, rtol=1e-12, atol=1e-12)


def test_brute_force_fp8_pool():
    inp = small([6, 11], [3, 2], 2, 8, p=4, kv_dtype="fp8", seed=3)
    ref, ref_lse = brute_force(inp)
    out, lse = extend_attention_rowwise(inp)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-12, atol=1e-12)
    out2, _ = extend_attention_blocked(inp)
    np.testing.assert_allclose(out2, ref, rtol=1e-12, atol=1e-12)


def _sdpa_reference(inp: PagedInputs):
    """torch SDPA (float64, CPU) per sequence on contiguous K/V, explicit mask."""
    T, HQ, D = inp.q.shape
    G = inp.gqa_group
    out = np.zeros((T, HQ, D))
    cu = inp.cu()
    P = inp.page_size
    for b in range(len(inp.prefix_lens)):
        lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
        if ls == 0:
            continue
        # contiguous K/V built with torch ops only (index_select of pages)
        kp = torch.from_numpy(inp.k_pool.view(np.int16)).view(torch.bfloat16).double()
        vp = torch.from_numpy(inp.v_pool.view(np.int16)).view(torch.bfloat16).double()
        pages = torch.from_numpy(inp.block_table[b, : (lp + P - 1) // P].astype(np.int64))
        kc = kp.index_select(0, pages).permute(0, 2, 1, 3).reshape(-1, kp.shape[1], D)[:lp]
        vc = vp.index_select(0, pages).permute(0, 2, 1, 3).reshape(-1, vp.shape[1], D)[:lp]
        kn = torch.from_numpy(inp.k_new.view(np.int16)).view(torch.bfloat16).double()[cu[b]:cu[b] + ls]
        vn = torch.from_numpy(inp.v_new.view(np.int16)).view(torch.bfloat16).double()[cu[b]:cu[b] + ls]
        k = torch.cat([kc, kn]).repeat_interleave(G, dim=1).transpose(0, 1)  # [HQ, N, D]
        v = torch.cat([vc, vn]).repeat_interleave(G, dim=1).transpose(0, 1)
        q = torch.from_numpy(inp.q.view(np.int16)).view(torch.bfloat16).double()[cu[b]:cu[b] + ls].transpose(0, 1)
        mask = torch.ones(ls, lp + ls, dtype=torch.bool).tril(diagonal=lp)  # bottom-right
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask,
                                                             scale=inp.softmax_scale)
        out[cu[b]:cu[b] + ls] = o.transpose(0, 1).numpy()
    return out


@pytest.mark.parametrize("g,d,p", [(1, 16, 4), (4, 32, 16), (3, 8, 8), (8, 64, 16)])
def test_matches_torch_sdpa(g, d, p):
    inp = small([40, 0, 17, 64], [25, 13, 1, 33], g, d, p=p, hkv=2, seed=100 + g)
    ref = _sdpa_reference(inp)
    out, _ = extend_attention_blocked(inp, block_tokens=8)
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-12)
    out1, _ = extend_attention_rowwise(inp)
    np.testing.assert_allclose(out1, ref, rtol=1e-10, atol=1e-12)


def test_sdpa_gqa_convention_is_h_div_g():
    # torch's own GQA broadcast (enable_gqa) maps query head h to kv head h // G,
    # the convention repeat_interleave reproduces in the reference above.
    torch.manual_seed(0)
    q = torch.randn(1, 8, 5, 16, dtype=torch.float64)
    k = torch.randn(1, 2, 5, 16, dtype=torch.float64)
    v = torch.randn(1, 2, 5, 16, dtype=torch.float64)
    a = torch.nn.functional.scaled_dot_product_attention(q, k, v, enable_gqa=True)
    b = torch.nn.functional.scaled_dot_product_attention(
        q, k.repeat_interleave(4, dim=1), v.repeat_interleave(4, dim=1))
    assert torch.allclose(a, b)


def test_single_visible_key_returns_its_value():
    inp = small([0, 0], [1, 5], 2, 16, p=4, seed=5)
    out, lse = extend_attention_rowwise(inp)
    vn = inp.v_new.astype(np.uint32) << 16
    vn = vn.view(np.float32).astype(np.float64)
    for r in (0, 1):  # first suffix row of each sequence sees only itself
        for h in range(out.shape[1]):
            assert np.array_equal(out[r, h], vn[r, h // 2])
    q = (inp.q.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    kn = (inp.k_new.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert lse[0, 0] == pytest.approx(inp.softmax_scale * float(q[0, 0] @ kn[0, 0]), rel=1e-12)


def test_zero_query_gives_mean_of_visible_values():
    """With q = 0 every visible key has weight 1/n; with V[j,:] = j, o_i = (Lp+i)/2."""
    inp = small([37, 10], [9, 6], 4, 8, p=8, hkv=1, seed=9)
    inp.q[:] = 0
    for b in range(2):
        lp = int(inp.prefix_lens[b])
        pg_count = (lp + 7) // 8
        for j in range(lp):
            pg, sl = inp.block_table[b, j // 8], j % 8
            inp.v_pool[pg, :, sl, :] = torch.tensor(float(j)).to(torch.bfloat16).view(torch.int16).item() & 0xFFFF
        c0 = int(inp.cu()[b])
        for i in range(int(inp.suffix_lens[b])):
            inp.v_new[c0 + i, :, :] = torch.tensor(float(lp + i)).to(torch.bfloat16).view(torch.int16).item() & 0xFFFF
    for fn in (extend_attention_rowwise, extend_attention_blocked):
        out, lse = fn(inp)
        for b in range(2):
            lp = int(inp.prefix_lens[b])
            c0 = int(inp.cu()[b])
            for i in range(int(inp.suffix_lens[b])):
                assert np.allclose(out[c0 + i], (lp + i) / 2.0, rtol=1e-14)
                assert np.allclose(lse[c0 + i], math.log(lp + i + 1), rtol=1e-14)


def _single_sequence(k_all, v_all, q_all, split, page_size, perm_seed, num_pages=None):
    """One sequence of N tokens with the first `split` keys cached in permuted pages."""
    n, hkv, d = k_all.shape
    n_pages = (n + page_size - 1) // page_size
    num_pages = num_pages or n_pages + 3
    rng = np.random.default_rng(perm_seed)
    ids = rng.permutation(num_pages)[:n_pages].astype(np.int32)
    kp = np.full((num_pages, hkv, page_size, d), 0x7FC0, dtype=np.uint16)
    vp = kp.copy()
    for j in range(split):
        kp[ids[j // page_size], :, j % page_size] = k_all[j]
        vp[ids[j // page_size], :, j % page_size] = v_all[j]
    return PagedInputs(q_all[split:].copy(), k_all[split:].copy(), v_all[split:].copy(), kp, vp,
                       ids[None, :], np.array([split]), np.array([n - split]),
                       q_all.shape[1] // hkv, 1 / math.sqrt(d))


def _random_bits(rng, shape):
    return torch.from_numpy(rng.standard_normal(shape, dtype=np.float32)).to(
        torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_split_point_and_page_permutation_invariance():
    rng = np.random.default_rng(11)
    n, hkv, g, d, P = 45, 2, 3, 16, 8
    k_all, v_all = _random_bits(rng, (n, hkv, d)), _random_bits(rng, (n, hkv, d))
    q_all = _random_bits(rng, (n, hkv * g, d))
    full, full_lse = extend_attention_rowwise(_single_sequence(k_all, v_all, q_all, 0, P, 0))
    for split in (0, 1, P - 1, P, P + 1, 30, n - 1):
        for perm_seed in (1, 2):
            out, lse = extend_attention_rowwise(_single_sequence(k_all, v_all, q_all, split, P, perm_seed))
            # same keys in the same order: identical to the all-suffix computation
            np.testing.assert_allclose(out, full[split:], rtol=1e-13, atol=1e-15)
            np.testing.assert_allclose(lse, full_lse[split:], rtol=1e-13)
        a, _ = extend_attention_rowwise(_single_sequence(k_all, v_all, q_all, split, P, 5))
        b, _ = extend_attention_rowwise(_single_sequence(k_all, v_all, q_all, split, P, 6))
        assert np.array_equal(a, b)  # page permutation: bit-identical


def test_gqa_equals_separate_mha_calls():
    inp = small([19, 7], [6, 11], 4, 16, p=4, hkv=2, seed=21)
    out, _ = extend_attention_rowwise(inp)
    for member in range(4):
        sub = PagedInputs(inp.q[:, member::4].copy(), inp.k_new, inp.v_new, inp.k_pool, inp.v_pool,
                          inp.block_table, inp.prefix_lens, inp.suffix_lens, 1, inp.softmax_scale)
        o1, _ = extend_attention_rowwise(sub)
        np.testing.assert_array_equal(o1, out[:, member::4])


def test_rows_and_decode_agree_with_full():
    inp = small([33, 4, 18], [1, 1, 1], 2, 8, p=4, seed=31)
    out, lse = extend_attention_blocked(inp)
    o2, l2 = decode_attention(inp.q, inp.k_new, inp.v_new, inp.k_pool, inp.v_pool, inp.block_table,
                              inp.prefix_lens, 2, inp.softmax_scale)
    np.testing.assert_allclose(o2, out, rtol=1e-12)
    rows = [(2, 3), (0, 0), (1, 1)]
    o3, l3 = extend_attention_rows(inp, rows)
    for k, (t, h) in enumerate(rows):
        np.testing.assert_allclose(o3[k], out[t, h], rtol=1e-12)
        assert l3[k] == pytest.approx(lse[t, h], rel=1e-12)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_token_blocks_against_brute_force(kv_dtype):
    # chosen suffix-token blocks (first, middle, ragged last, a whole short sequence)
    inp = small([7, 0, 12], [9, 5, 3], 3, 8, p=4, kv_dtype=kv_dtype, seed=57)
    ref, ref_lse = brute_force(inp)
    cu = inp.cu()
    blocks = [(0, 0, 4), (0, 4, 8), (0, 8, 9), (1, 0, 5), (2, 1, 3)]
    for (b, t0, t1), (out, lse) in zip(blocks, extend_attention_token_blocks(inp, blocks)):
        r0, r1 = int(cu[b]) + t0, int(cu[b]) + t1
        np.testing.assert_allclose(out, ref[r0:r1], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse, ref_lse[r0:r1], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_float32_blocked_matches_float64(kv_dtype):
    # the single-precision variant (timed as the CPU baseline) runs the same steps:
    # it agrees with the float64 checker to fp32 accumulation error
    inp = small([300, 0, 77], [40, 9, 64], 4, 64, p=16, kv_dtype=kv_dtype, seed=61)
    ref, ref_lse = extend_attention_blocked(inp)
    out, lse = extend_attention_blocked(inp, dtype=np.float32)
    assert out.dtype == np.float32 and lse.dtype == np.float32
    np.testing.assert_allclose(out, ref, rtol=0, atol=2e-5)
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=2e-5)


def test_fp8_gather_uses_page_scale():
    inp = small([13], [2], 1, 8, p=4, hkv=2, kv_dtype="fp8", seed=41)
    k, v = gather_sequence_kv(inp, 0)
    for j in range(13):
        pg, sl = int(inp.block_table[0, j // 4]), j % 4
        dec = torch.from_numpy(inp.k_pool[pg, :, sl]).view(torch.float8_e4m3fn).double().numpy()
        np.testing.assert_array_equal(k[j], dec * inp.k_scale[pg][:, None].astype(np.float64))
