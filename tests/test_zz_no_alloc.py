"""cw_extend_attention_noalloc (the entry point for callers that cannot allocate)
against cw_extend_attention, through the C ABI: bit-identical outputs on two
calls in a row, the second with a smaller input, no pinned allocation during
the calls, and the size cap and the init requirement enforced before anything
is enqueued."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import BF16_MAX_ABS, BF16_MEAN_ABS, as_f64, assert_close, bits, to_gpu

pytestmark = pytest.mark.gpu


def _both(dw):
    s = dw.spec
    nan = lambda: torch.full_like(dw.q, float("nan"))
    nan_lse = lambda: torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
    out_a, lse_a, out_b, lse_b = nan(), nan_lse(), nan(), nan_lse()
    args = (dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table, s.prefix_lens,
            s.suffix_lens, s.gqa_group, s.softmax_scale)
    cwlib.extend_attention(*args, k_scale=dw.k_scale, v_scale=dw.v_scale, out=out_a, lse=lse_a)
    torch.cuda.synchronize()
    n0 = cwlib.pinned_allocations()
    cwlib.extend_attention_noalloc(*args, k_scale=dw.k_scale, v_scale=dw.v_scale, out=out_b, lse=lse_b)
    torch.cuda.synchronize()
    assert cwlib.pinned_allocations() == n0
    return out_a, lse_a, out_b, lse_b


def test_noalloc_matches_extend_on_two_calls():
    fresh = cwlib.pinned_allocations() == 0
    spec_big = cw.custom_spec([700, 90, 3000], [150, 64, 300], num_kv_heads=2, gqa_group=4,
                              head_dim=128, page_size=16, seed=21)
    w_big = cw.materialize(spec_big)
    dw_big = to_gpu(w_big)
    if fresh:  # nothing has set up this device yet in this process
        print("\n[case] noalloc before cw_init", flush=True)
        out = torch.full_like(dw_big.q, float("nan"))
        with pytest.raises(cwlib.CWError) as ei:
            cwlib.extend_attention_noalloc(dw_big.q, dw_big.k_new, dw_big.v_new, dw_big.k_pool,
                                           dw_big.v_pool, dw_big.block_table, spec_big.prefix_lens,
                                           spec_big.suffix_lens, 4, spec_big.softmax_scale, out=out)
        assert ei.value.status == 8  # CW_ERR_INIT
        torch.cuda.synchronize()
        assert bool(torch.isnan(out).all())
    cwlib.init()
    spec_small = cw.custom_spec([40, 0], [9, 30], num_kv_heads=2, gqa_group=4, head_dim=128,
                                page_size=16, seed=22)
    w_small = cw.materialize(spec_small)
    for name, w, dw in (("big", w_big, dw_big), ("small", w_small, to_gpu(w_small))):
        print(f"\n[case] noalloc {name}: Lp={w.spec.prefix_lens.tolist()} Ls={w.spec.suffix_lens.tolist()}",
              flush=True)
        out_a, lse_a, out_b, lse_b = _both(dw)
        assert np.array_equal(bits(out_a), bits(out_b)), name
        assert np.array_equal(lse_a.cpu().numpy().view(np.uint32), lse_b.cpu().numpy().view(np.uint32)), name
        ref, _ = oracle.extend_attention_blocked(paged_inputs(w))
        assert_close(as_f64(out_b), ref, BF16_MAX_ABS, BF16_MEAN_ABS, f"noalloc {name}")


def test_noalloc_rejects_a_plan_larger_than_the_scratch():
    cwlib.init()
    w = cw.make("turn")
    s = w.spec
    dw = to_gpu(w)
    print("\n[case] noalloc over the scratch size (turn, one-tile split-K chunks)", flush=True)
    out = torch.full_like(dw.q, float("nan"))
    cwlib.set_tuning(0, 1)  # about 35k partial slots of 64 KiB: far above the cap
    try:
        need = cwlib.extend_workspace_bytes(s.prefix_lens, s.suffix_lens, s.num_kv_heads,
                                            s.gqa_group, s.head_dim, s.page_size)
        assert need > 64 << 20
        with pytest.raises(cwlib.CWError) as ei:
            cwlib.extend_attention_noalloc(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool,
                                           dw.block_table, s.prefix_lens, s.suffix_lens,
                                           s.gqa_group, s.softmax_scale, out=out)
        assert ei.value.status == 5  # CW_ERR_WORKSPACE
    finally:
        cwlib.set_tuning(0, 0)
    torch.cuda.synchronize()
    assert bool(torch.isnan(out).all())
