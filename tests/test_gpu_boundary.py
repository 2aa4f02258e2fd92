"""Boundary behaviour on the GPU: the binding's checks fire before any kernel is
launched, and no call allocates pinned memory after the one-time set-up."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import paper_2606_16824_amd as cwlib
from gpu_util import to_gpu

pytestmark = pytest.mark.gpu


def test_int64_block_table_and_short_out_are_rejected_before_launch():
    spec = cw.custom_spec([40, 7], [9, 3], num_kv_heads=2, gqa_group=4, head_dim=128, page_size=16,
                          seed=8)
    print("\n[case] binding rejects an int64 block table and a short out", flush=True)
    dw = to_gpu(cw.materialize(spec))
    out = torch.full_like(dw.q, float("nan"))
    with pytest.raises(ValueError, match="2-D int32"):
        cwlib.extend_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table.long(),
                               spec.prefix_lens, spec.suffix_lens, 4, spec.softmax_scale, out=out)
    with pytest.raises(ValueError, match="out has shape"):
        cwlib.extend_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                               spec.prefix_lens, spec.suffix_lens, 4, spec.softmax_scale, out=out[:-1])
    torch.cuda.synchronize()
    assert bool(torch.isnan(out).all())  # nothing was launched


def test_growing_plans_allocate_no_pinned_memory():
    cwlib.init()
    n0 = cwlib.pinned_allocations()
    assert n0 == 8  # the staging ring of the one device, allocated once
    print("\n[case] growing plans: extend, decode and step calls", flush=True)
    for n_seq in (1, 4, 16, 48):
        lp = [(311 * i) % 3000 for i in range(n_seq)]
        ls = [1 + (97 * i) % 300 for i in range(n_seq)]
        spec = cw.custom_spec(lp, ls, num_kv_heads=2, gqa_group=4, head_dim=128, page_size=16,
                              seed=n_seq)
        dw = to_gpu(cw.materialize(spec))
        cwlib.extend_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                               spec.prefix_lens, spec.suffix_lens, 4, spec.softmax_scale)
        cwlib.step_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                             spec.prefix_lens, spec.suffix_lens, 4, spec.softmax_scale)
        dspec = cw.custom_spec(lp, [1] * n_seq, num_kv_heads=2, gqa_group=4, head_dim=128,
                               page_size=16, seed=n_seq)
        dd = to_gpu(cw.materialize(dspec))
        cwlib.decode_attention(dd.q, dd.k_new, dd.v_new, dd.k_pool, dd.v_pool, dd.block_table,
                               dspec.prefix_lens, 4, dspec.softmax_scale)
        torch.cuda.synchronize()
        assert cwlib.pinned_allocations() == n0, n_seq
