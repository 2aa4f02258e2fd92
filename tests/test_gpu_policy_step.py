"""A serving step produced by the KV block manager, run on the GPU against the
oracle.  Sessions of two shared-prefix groups and two private sessions run
requests through the manager on a small node (so blocks are shared, evicted and
reused), then one step admits four of them at once; their block tables (shared
prefix blocks aliased across the group's rows) and (prefix, suffix) lengths go
straight to cw_step_attention, with pools and new tokens drawn at random."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from gpu_util import BF16_MAX_ABS, BF16_MEAN_ABS, as_f64, assert_close, bits
from paper_2606_16824_amd import policy

pytestmark = pytest.mark.gpu

B, M, HKV, G, D = 16, 160, 2, 4, 128
SHARED = 128  # 8 shared blocks per group


def _policy_step():
    bm = policy.BlockManager(M, B)
    groups = [0, 1, 0, 1, -1, -1]
    for s, g in enumerate(groups):
        bm.add_session(s, g, SHARED if g >= 0 else 0)
    ctx = [0] * 6
    # earlier requests, one at a time (values: larger evicts first)
    first = [(300, 20), (260, 40), (180, 8), (400, 16), (350, 30), (500, 12)]
    values = [1.0, 9.0, 2.0, 8.0, 12.0, 6.0]  # group 0 needed soonest, session 4 last
    for s, (tin, tout) in enumerate(first):
        bm.admit(s, ctx[s], tin, tout)
        ctx[s] += tin + tout
        bm.release(s, values[s])
    # a second turn for sessions 1 and 5 (evicts what no longer fits)
    for s, tin in ((1, 700), (5, 300)):
        bm.admit(s, ctx[s], tin, 10)
        ctx[s] += tin + 10
        bm.release(s, values[s])
    # the step: four sessions' next requests admitted together (the group's
    # shared blocks are resident before it: no request of the step allocates a
    # block another one reads as prefix)
    step = [(0, 333), (2, 77), (4, 129), (5, 256)]
    rows, lp, ls = [], [], []
    for s, tin in step:
        table, cached, _ = bm.admit(s, ctx[s], tin, 0)
        rows.append(table)
        lp.append(cached)
        ls.append(ctx[s] + tin - cached)
    return groups, step, rows, np.asarray(lp), np.asarray(ls), bm


def test_block_manager_step_matches_oracle():
    groups, step, rows, lp, ls, bm = _policy_step()
    print(f"\n[case] policy step: Lp={lp.tolist()} Ls={ls.tolist()} "
          f"blocks={[len(r) for r in rows]} {bm.stats()}", flush=True)
    # the group-0 members' shared prefix is resident and aliased in both rows
    assert list(rows[0][:SHARED // B]) == list(rows[1][:SHARED // B])
    assert lp[0] >= SHARED and lp[1] >= SHARED  # aliased pages lie inside both prefixes
    assert (lp > 0).any() and (ls > 0).all()
    stride = max(len(r) for r in rows)
    bt = np.full((len(rows), stride), cw.BT_UNUSED, dtype=np.int32)
    for b, r in enumerate(rows):
        bt[b, :len(r)] = r
    T = int(ls.sum())
    g = torch.Generator().manual_seed(7)
    rnd = lambda *shape: torch.randn(*shape, generator=g).to(torch.bfloat16)
    q, kn, vn = rnd(T, HKV * G, D), rnd(T, HKV, D), rnd(T, HKV, D)
    kp, vp = rnd(M, HKV, B, D), rnd(M, HKV, B, D)
    dev = torch.device("cuda:0")
    dq, dkn, dvn, dkp, dvp = (t.to(dev) for t in (q, kn, vn, kp, vp))
    dbt = torch.from_numpy(bt).to(dev)
    scale = 1.0 / np.sqrt(D)
    out = torch.full_like(dq, float("nan"))
    cwlib.step_attention(dq, dkn, dvn, dkp, dvp, dbt, lp, ls, G, scale, out=out)
    torch.cuda.synchronize()
    u16 = lambda t: t.view(torch.int16).numpy().view(np.uint16)
    inp = oracle.PagedInputs(q=u16(q), k_new=u16(kn), v_new=u16(vn), k_pool=u16(kp), v_pool=u16(vp),
                             block_table=bt, prefix_lens=lp.astype(np.int64),
                             suffix_lens=ls.astype(np.int64), gqa_group=G, softmax_scale=scale)
    ref, _ = oracle.extend_attention_blocked(inp)
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "policy step")
    want_k, want_v = oracle.write_pages(inp)
    assert np.array_equal(bits(dkp), want_k) and np.array_equal(bits(dvp), want_v)
