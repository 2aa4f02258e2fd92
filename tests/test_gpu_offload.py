"""The offload serving loop on the GPU: the KV block manager with a host pool
admits requests; each admission's page copies run through cw_kv_swap_out then
cw_kv_swap_in (pinned host pools), and each step runs cw_step_attention over
the admitted requests (their prefix pages read from the pool, their suffix
written into it).  Every step's output is checked against the oracle over the
sessions' own K/V (not the pool's), and the pool pages of every admitted request
are checked bit for bit against the K/V of its tokens: a wrong swap list, a
copy in the wrong order or a wrong page write fails it."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from gpu_util import BF16_MAX_ABS, BF16_MEAN_ABS, as_f64, assert_close, bits
from test_offload import BLOCK, DEVICE_BLOCKS, HOST_BLOCKS, MAX_CTX, logical_kv, run_loop

pytestmark = pytest.mark.gpu

HKV, G, D = 2, 4, 64


def _bf16_bits(x):
    return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("seed", [1, 2])
def test_offload_serving_loop_matches_oracle(seed):
    print(f"\n[case] offload serving loop, seed {seed}", flush=True)
    kv = _bf16_bits(logical_kv(seed, 2 * HKV * D)).reshape(-1, MAX_CTX, 2, HKV, D)
    lk, lv = kv[:, :, 0], kv[:, :, 1]  # [session, position, head, dim] bf16 bits
    dev = torch.device("cuda:0")
    as_bf16 = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    kp = torch.zeros(DEVICE_BLOCKS, HKV, BLOCK, D, dtype=torch.bfloat16, device=dev)
    vp = torch.zeros_like(kp)
    kh = torch.zeros(HOST_BLOCKS, HKV, BLOCK, D, dtype=torch.bfloat16).pin_memory()
    vh = torch.zeros_like(kh).pin_memory()
    gen = torch.Generator().manual_seed(seed)
    scale = 1.0 / np.sqrt(D)
    counts = {"steps": 0, "out": 0, "in": 0}

    def apply_swaps(outs, ins):
        if outs:
            cwlib.kv_swap_out(kp, vp, kh, vh, [d for d, _ in outs], [h for _, h in outs])
            counts["out"] += len(outs)
        if ins:
            cwlib.kv_swap_in(kh, vh, kp, vp, [h for h, _ in ins], [d for _, d in ins])
            counts["in"] += len(ins)

    def after_step(rows):
        lp = np.asarray([c for _, _, c, _ in rows], np.int64)
        ls = np.asarray([e - c for _, _, c, e in rows], np.int64)
        stride = max(len(t) for _, t, _, _ in rows)
        bt = np.full((len(rows), stride), cw.BT_UNUSED, dtype=np.int32)
        for b, (_, t, _, _) in enumerate(rows):
            bt[b, :len(t)] = t
        kn = np.concatenate([lk[s, c:e] for s, _, c, e in rows])
        vn = np.concatenate([lv[s, c:e] for s, _, c, e in rows])
        q = torch.randn(int(ls.sum()), HKV * G, D, generator=gen).to(torch.bfloat16)
        out = torch.full(tuple(q.shape), float("nan"), dtype=torch.bfloat16, device=dev)
        cwlib.step_attention(q.to(dev), as_bf16(kn).to(dev), as_bf16(vn).to(dev), kp, vp,
                             torch.from_numpy(bt).to(dev), lp, ls, G, scale, out=out)
        torch.cuda.synchronize()
        # the oracle reads each prefix from the sessions' own K/V
        rk = np.zeros((DEVICE_BLOCKS, HKV, BLOCK, D), np.uint16)
        rv = np.zeros_like(rk)
        for s, t, c, _ in rows:
            for p in range(c):
                rk[t[p // BLOCK], :, p % BLOCK] = lk[s, p]
                rv[t[p // BLOCK], :, p % BLOCK] = lv[s, p]
        inp = oracle.PagedInputs(q=q.view(torch.int16).numpy().view(np.uint16), k_new=kn, v_new=vn,
                                 k_pool=rk, v_pool=rv, block_table=bt, prefix_lens=lp, suffix_lens=ls,
                                 gqa_group=G, softmax_scale=scale)
        ref, _ = oracle.extend_attention_blocked(inp)
        assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, f"offload step {counts['steps']}")
        gk, gv = bits(kp), bits(vp)
        for s, t, _, e in rows:
            for p in range(e):
                assert np.array_equal(gk[t[p // BLOCK], :, p % BLOCK], lk[s, p]), (counts["steps"], s, p)
                assert np.array_equal(gv[t[p // BLOCK], :, p % BLOCK], lv[s, p]), (counts["steps"], s, p)
        counts["steps"] += 1

    totals = run_loop(seed, apply_swaps, after_step)
    print(f"[offload] {counts['steps']} steps, {counts['out']} swap-outs, {counts['in']} swap-ins, "
          f"{totals['evicted']} evictions, {totals['hit']} cached tokens", flush=True)
    assert counts["out"] > 0 and counts["in"] > 0
