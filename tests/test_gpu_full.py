"""Full-size parity: the named workloads at their real sizes, in the launch
configuration the benchmark times, checked on sampled rows the oracle computes
one by one (first and last suffix token of every sequence for every head, plus
seeded random rows), and the page scatter checked slot by slot.
"""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import BF16_MAX_ABS, BF16_MEAN_ABS, FP8_MAX_ABS, as_f64, assert_close, to_gpu

pytestmark = pytest.mark.gpu


def _sample_rows(spec, n_random=96, seed=0):
    cu = np.concatenate([[0], np.cumsum(spec.suffix_lens)])
    rows = []
    for b in range(spec.num_seqs):
        if spec.suffix_lens[b] == 0:
            continue
        for tok in {int(cu[b]), int(cu[b + 1] - 1)}:
            rows += [(tok, h) for h in range(spec.num_q_heads)]
    rng = np.random.default_rng(seed)
    t = rng.integers(0, spec.total_new_tokens, size=n_random)
    h = rng.integers(0, spec.num_q_heads, size=n_random)
    rows += list(zip(t.tolist(), h.tolist()))
    return rows


@pytest.mark.parametrize("name", ["turn", "batch16", "long", "mixed"])
def test_full_size_extend_sampled(name):
    w = cw.make(name)
    s = w.spec
    print(f"\n[case] full {name}: B={s.num_seqs} T={s.total_new_tokens} pages={s.num_pages} "
          f"kv={s.kv_dtype}", flush=True)
    dw = to_gpu(w)
    lse = torch.empty(dw.q.shape[0], dw.q.shape[1], device=dw.q.device)
    out = cwlib.extend_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                                 s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale,
                                 k_scale=dw.k_scale, v_scale=dw.v_scale, lse=lse)
    torch.cuda.synchronize()
    rows = _sample_rows(s)
    ref, ref_lse = oracle.extend_attention_rows(paged_inputs(w), rows)
    t_idx = torch.tensor([r for r, _ in rows])
    h_idx = torch.tensor([h for _, h in rows])
    got = as_f64(out.cpu()[t_idx, h_idx])
    got_lse = lse.cpu()[t_idx, h_idx].double().numpy()
    if s.kv_dtype == "bf16":
        assert_close(got, ref, BF16_MAX_ABS, BF16_MEAN_ABS, f"{name} sampled")
    else:
        assert_close(got, ref, FP8_MAX_ABS, None, f"{name} sampled")
    assert_close(got_lse, ref_lse, 1e-2, None, f"{name} lse")


@pytest.mark.parametrize("name", ["turn", "batch16", "mixed"])
def test_full_size_write_pages(name):
    w = cw.make(name)
    s = w.spec
    print(f"\n[case] full write_pages {name}", flush=True)
    dw = to_gpu(w)
    before_k = dw.k_pool.clone()
    cwlib.kv_write_pages(dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                         s.prefix_lens, s.suffix_lens, k_scale=dw.k_scale, v_scale=dw.v_scale)
    torch.cuda.synchronize()
    # destination of every new token: page and slot from the block table
    p = s.page_size
    pages, slots = [], []
    bt = w.block_table.numpy()
    for b in range(s.num_seqs):
        pos = s.prefix_lens[b] + np.arange(s.suffix_lens[b])
        pages.append(bt[b, pos // p])
        slots.append(pos % p)
    pages = torch.from_numpy(np.concatenate(pages).astype(np.int64)).to(dw.k_pool.device)
    slots = torch.from_numpy(np.concatenate(slots).astype(np.int64)).to(dw.k_pool.device)
    written = dw.k_pool[pages, :, slots, :]  # [T, Hkv, D]
    if s.kv_dtype == "bf16":
        assert torch.equal(written.view(torch.int16), dw.k_new.view(torch.int16))
    else:
        # sampled tokens against the oracle's quantise-on-write
        rng = np.random.default_rng(1)
        toks = rng.integers(0, s.total_new_tokens, size=64)
        sc = w.k_scale.numpy()
        kn = w.np_bits(w.k_new)
        pg_np, sl_np = pages.cpu().numpy(), slots.cpu().numpy()
        got = written.cpu().numpy()
        for tk in toks:
            x = oracle.bf16_bits_to_f64(kn[tk]).astype(np.float32)
            q = np.clip(x / sc[pg_np[tk]].astype(np.float32)[:, None], -448, 448)
            assert np.array_equal(got[tk], oracle.e4m3fn_encode_rne(q.astype(np.float64)))
    # nothing else changed
    mask = torch.ones(dw.k_pool.shape[0], dw.k_pool.shape[2], dtype=torch.bool, device=dw.k_pool.device)
    mask[pages, slots] = False
    keep = mask[:, None, :, None].expand(dw.k_pool.shape)
    raw = (lambda t: t.view(torch.int16)) if dw.k_pool.dtype == torch.bfloat16 else (lambda t: t)
    assert torch.equal(raw(dw.k_pool)[keep], raw(before_k)[keep])
