"""Full-size parity: the named workloads at their real sizes, in the launch
configuration the benchmark times (one cw_step_attention: the page write fused
into the extend launch, decodes on the decode kernel), against the oracle:
the named workloads, and a chunked-prefill step (32 chunks of at most 512
tokens and 32 decodes).

Outputs start as NaN and must all be finite afterwards.  The turn is compared
row by row in full.  For batch16, long and mixed, whole query tiles of the
extend kernel are compared, every head: the first, a middle and the last
(ragged) tile of every sequence (a tile is 256 packed rows = 256 / G tokens),
and for mixed also every decode row.  The page scatter is checked slot by slot.
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

TILE_ROWS = 256  # packed query rows per extend work item


def _tile_blocks(spec):
    """(sequence, t0, t1) of the first, a middle and the last query tile of every
    sequence (one block per decode sequence)."""
    tt = TILE_ROWS // spec.gqa_group
    blocks = []
    for b in range(spec.num_seqs):
        ls = int(spec.suffix_lens[b])
        if ls == 0:
            continue
        n_t = (ls + tt - 1) // tt
        for i in sorted({0, n_t // 2, n_t - 1}):
            blocks.append((b, i * tt, min(ls, (i + 1) * tt)))
    return blocks


def _run_step(dw):
    s = dw.spec
    out = torch.full_like(dw.q, float("nan"))
    lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
    cwlib.step_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                         s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale,
                         k_scale=dw.k_scale, v_scale=dw.v_scale, out=out, lse=lse)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("name", ["turn", "batch16", "long", "mixed", "chunked"])
def test_full_size_step(name):
    w = cw.make(name)
    s = w.spec
    print(f"\n[case] full {name}: B={s.num_seqs} T={s.total_new_tokens} pages={s.num_pages} "
          f"kv={s.kv_dtype}", flush=True)
    out, lse = _run_step(to_gpu(w))
    n_bad = int((~torch.isfinite(out)).sum()) + int((~torch.isfinite(lse)).sum())
    assert n_bad == 0, f"{n_bad} outputs not written or not finite"
    out_c, lse_c = out.cpu(), lse.cpu()
    inp = paged_inputs(w)
    if name == "turn":
        ref, ref_lse = oracle.extend_attention_blocked(inp)
        got, got_lse = as_f64(out_c), lse_c.double().numpy()
    else:
        blocks = _tile_blocks(s)
        res = oracle.extend_attention_token_blocks(inp, blocks)
        cu = np.concatenate([[0], np.cumsum(s.suffix_lens)])
        rows = np.concatenate([np.arange(cu[b] + t0, cu[b] + t1) for b, t0, t1 in blocks])
        ref = np.concatenate([o for o, _ in res])
        ref_lse = np.concatenate([l for _, l in res])
        idx = torch.from_numpy(rows)
        got, got_lse = as_f64(out_c[idx]), lse_c[idx].double().numpy()
        print(f"[{name}] {len(blocks)} tiles, {len(rows)} tokens x {s.num_q_heads} heads checked",
              flush=True)
    if s.kv_dtype == "bf16":
        assert_close(got, ref, BF16_MAX_ABS, BF16_MEAN_ABS, f"full {name}")
    else:
        assert_close(got, ref, FP8_MAX_ABS, None, f"full {name}")
    assert_close(got_lse, ref_lse, 1e-2, None, f"full {name} lse")


@pytest.mark.parametrize("name", ["turn", "batch16", "mixed", "chunked"])
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
        # every new token against the oracle's quantise-on-write
        sc = w.k_scale.numpy()
        kn = w.np_bits(w.k_new)
        pg_np = pages.cpu().numpy()
        got = written.cpu().numpy()
        x = oracle.bf16_bits_to_f64(kn).astype(np.float32)
        q = np.clip(x / sc[pg_np].astype(np.float32)[:, :, None], -448, 448)
        assert np.array_equal(got, oracle.e4m3fn_encode_rne(q.astype(np.float64)))
    # nothing else changed
    mask = torch.ones(dw.k_pool.shape[0], dw.k_pool.shape[2], dtype=torch.bool, device=dw.k_pool.device)
    mask[pages, slots] = False
    keep = mask[:, None, :, None].expand(dw.k_pool.shape)
    raw = (lambda t: t.view(torch.int16)) if dw.k_pool.dtype == torch.bfloat16 else (lambda t: t)
    assert torch.equal(raw(dw.k_pool)[keep], raw(before_k)[keep])


def test_chunked_step_one_launch_matches_two():
    """The chunked-prefill step through one extend launch (decodes as one-token
    extends) gives the rows of the two-kernel step within 2 bf16 ulps."""
    from gpu_util import assert_within_bf16_ulps
    w = cw.make("chunked")
    s = w.spec
    print("\n[case] chunked one launch vs step", flush=True)
    dw = to_gpu(w)
    two, _ = _run_step(dw)
    one = cwlib.write_extend_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                                       s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale)
    torch.cuda.synchronize()
    assert_within_bf16_ulps(as_f64(one), as_f64(two), 2, "chunked one launch vs two")
