"""GPU parity of cw_extend_attention / cw_decode_attention against the CPU oracle.

Every case prints its name and shape before touching the GPU.  Tolerances:
bf16 pool max-abs 2e-2 / mean-abs 2e-3 on N(0,1) inputs; fp8 pool max-abs
6e-2 against the oracle run on the same dequantised values.
"""
import zlib

import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import (BF16_MAX_ABS, BF16_MEAN_ABS, FP8_MAX_ABS, as_f64, assert_close,
                      assert_within_bf16_ulps, bits, run_extend, to_gpu)

pytestmark = pytest.mark.gpu


def _case(name, spec):
    print(f"\n[case] {name}: Lp={spec.prefix_lens.tolist()[:8]} Ls={spec.suffix_lens.tolist()[:8]} "
          f"B={spec.num_seqs} Hkv={spec.num_kv_heads} G={spec.gqa_group} D={spec.head_dim} "
          f"P={spec.page_size} kv={spec.kv_dtype}", flush=True)


SMALL_CASES = {
    # name: (prefix lens, suffix lens, Hkv, G, D, P, kv dtype)
    "tiny_shape": ([256], [64], 1, 4, 64, 16, "bf16"),
    "ragged_mha": ([0, 37, 200, 64], [70, 1, 129, 33], 2, 1, 128, 16, "bf16"),
    "gqa8_p64": ([100, 513], [45, 100], 2, 8, 128, 64, "bf16"),
    "gqa3_d64": ([31, 0, 95], [17, 40, 3], 3, 3, 64, 16, "bf16"),
    "empty_seq": ([40, 10, 0], [0, 20, 0], 1, 4, 128, 16, "bf16"),
    "long_tail": ([1000], [300], 2, 4, 128, 16, "bf16"),
    "gqa16": ([77], [9], 1, 16, 64, 64, "bf16"),
    "fp8_small": ([50, 300], [30, 60], 2, 4, 128, 16, "fp8"),
    "fp8_p64_d64": ([129, 64], [1, 77], 1, 2, 64, 64, "fp8"),
    "many_heads_mha": ([64, 130], [40, 17], 16, 1, 64, 16, "bf16"),
    "gqa16_d128_fp8": ([200, 17], [24, 3], 1, 16, 128, 16, "fp8"),
    "fp8_p64_d128": ([129, 64, 300], [33, 90, 1], 2, 4, 128, 64, "fp8"),
    "fp8_p16_d64": ([50, 130, 17], [20, 45, 3], 2, 4, 64, 16, "fp8"),
    # 263 query tiles of one (sequence, kv head): one round dealt across all XCDs,
    # the rest and the second sequence queued behind it
    "dealt_round": ([100, 30], [4200, 50], 1, 16, 64, 16, "bf16"),
    # 40 short ragged sequences: many bundles, idle padding in the XCD queues
    "many_seqs": ([(37 * i) % 301 for i in range(40)], [1 + (11 * i) % 40 for i in range(40)],
                  2, 4, 128, 16, "bf16"),
}


@pytest.mark.parametrize("name", list(SMALL_CASES))
def test_extend_small_against_oracle(name):
    lp, ls, hkv, g, d, p, dt = SMALL_CASES[name]
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p,
                          kv_dtype=dt, seed=zlib.crc32(name.encode()) % 1000)
    _case(name, spec)
    w = cw.materialize(spec)
    out, lse = run_extend(to_gpu(w))
    ref, ref_lse = oracle.extend_attention_blocked(paged_inputs(w))
    if dt == "bf16":
        assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, name)
    else:
        assert_close(as_f64(out), ref, FP8_MAX_ABS, None, name)
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, name + " lse")


def test_tiny_config_full():
    w = cw.make("tiny")
    _case("tiny", w.spec)
    out, lse = run_extend(to_gpu(w))
    ref, ref_lse = oracle.extend_attention_rowwise(paged_inputs(w))
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "tiny")
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, "tiny lse")


@pytest.mark.parametrize("chunk_tiles", [1, 2, 3, 7])
def test_forced_split_matches_unsplit(chunk_tiles):
    spec = cw.custom_spec([700, 90], [150, 64], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=16, seed=77)
    _case(f"split{chunk_tiles}", spec)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    base, base_lse = run_extend(dw)
    cwlib.set_tuning(0, chunk_tiles)
    try:
        out, lse = run_extend(dw)
    finally:
        cwlib.set_tuning(0, 0)
    ref, _ = oracle.extend_attention_blocked(paged_inputs(w))
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "split vs oracle")
    assert_within_bf16_ulps(as_f64(out), as_f64(base), 2, "split vs unsplit")
    # the row sums add the bf16-rounded weights (relative error <= 2^-9 each), so two
    # different splits of the keys may differ by up to 2 * 2^-9 in lse
    assert_close(lse.cpu().double().numpy(), base_lse.cpu().double().numpy(), 2 ** -8, None, "lse")


def _max_parts(items):
    real = items[items[:, 0] >= 0]
    _, counts = np.unique(real[:, :3], axis=0, return_counts=True)
    return int(counts.max())


def test_merge_of_few_partials():
    """64 query tiles with a target of 128 workgroups: one to three key chunks per
    tile, merged by the merge kernel's few-partials path (all loads of a row
    issued at once); the default plan splits them into more chunks (its
    many-partials path, slices merged through LDS).  Both against the oracle,
    and against each other within 2 bf16 ulps."""
    spec = cw.custom_spec([2000, 300], [1536, 512], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=16, seed=79)
    _case("few parts", spec)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    assert _max_parts(cwlib.plan_items(spec.prefix_lens, spec.suffix_lens, 2, 4, 128, 16)) > 4
    cwlib.set_tuning(1, 128)
    try:
        assert _max_parts(cwlib.plan_items(spec.prefix_lens, spec.suffix_lens, 2, 4, 128, 16)) <= 4
        out, lse = run_extend(dw)
    finally:
        cwlib.set_tuning(1, 0)
    base, base_lse = run_extend(dw)
    ref, _ = oracle.extend_attention_blocked(paged_inputs(w))
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "few parts vs oracle")
    assert_close(as_f64(base), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "many parts vs oracle")
    assert_within_bf16_ulps(as_f64(out), as_f64(base), 2, "few parts vs many parts")
    assert_close(lse.cpu().double().numpy(), base_lse.cpu().double().numpy(), 2 ** -8, None, "lse")


def test_page_permutation_bitwise():
    spec = cw.custom_spec([300, 45], [70, 130], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=16, seed=5)
    _case("perm", spec)
    w = cw.materialize(spec)
    out_a, _ = run_extend(to_gpu(w))
    # move every page to a new physical id and rewrite the block table
    rng = np.random.default_rng(9)
    perm = torch.from_numpy(rng.permutation(spec.num_pages).astype(np.int64))
    k2 = torch.empty_like(w.k_pool)
    v2 = torch.empty_like(w.v_pool)
    k2[perm] = w.k_pool
    v2[perm] = w.v_pool
    bt = w.block_table.clone()
    used = bt != cw.BT_UNUSED
    bt[used] = perm[bt[used].long()].to(torch.int32)
    w.k_pool, w.v_pool, w.block_table = k2, v2, bt
    out_b, _ = run_extend(to_gpu(w))
    assert np.array_equal(bits(out_a), bits(out_b))


def test_decode_equals_extend_with_suffix_one():
    spec = cw.custom_spec([2000, 17, 513, 64], [1, 1, 1, 1], num_kv_heads=2, gqa_group=4,
                          head_dim=128, page_size=16, seed=12)
    _case("decode", spec)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    ext, _ = run_extend(dw)
    dec = torch.full_like(dw.q, float("nan"))
    cwlib.decode_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                           spec.prefix_lens, spec.gqa_group, spec.softmax_scale, out=dec)
    torch.cuda.synchronize()
    ref, _ = oracle.extend_attention_rowwise(paged_inputs(w))
    assert_close(as_f64(dec), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "decode vs oracle")
    assert_within_bf16_ulps(as_f64(dec), as_f64(ext), 2, "decode vs extend")


def test_closed_form_single_key_and_mean():
    """Lp=0, first row sees only itself -> its v row exactly; q=0 -> mean of visible V."""
    spec = cw.custom_spec([0, 40], [5, 9], num_kv_heads=1, gqa_group=2, head_dim=64,
                          page_size=16, seed=3)
    _case("closed_form", spec)
    w = cw.materialize(spec)
    out, _ = run_extend(to_gpu(w))
    assert np.array_equal(bits(out)[0, 0], bits(w.v_new)[0, 0])
    assert np.array_equal(bits(out)[0, 1], bits(w.v_new)[0, 0])
    w.q.zero_()
    out0, _ = run_extend(to_gpu(w))
    ref, _ = oracle.extend_attention_rowwise(paged_inputs(w))
    assert_close(as_f64(out0), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "q=0")


@pytest.mark.parametrize("lp", [0, 100])
def test_forced_split_with_strongly_negative_scores(lp):
    """G = 1 and one-tile chunks: the first wave of a 256-row item sees none of the
    later chunks' keys; its empty partials must not outweigh real ones whose row
    maxima lie far below zero (scores about -128, i.e. -185 in log2 units)."""
    spec = cw.custom_spec([lp], [256], num_kv_heads=1, gqa_group=1, head_dim=64, page_size=16,
                          seed=31)
    _case(f"negative_split_lp{lp}", spec)
    w = cw.materialize(spec)
    g = torch.Generator().manual_seed(4)
    w.q = torch.full_like(w.q, -16.0)
    w.k_new = (1 + 0.05 * torch.randn(w.k_new.shape, generator=g)).to(torch.bfloat16)
    w.k_pool = (1 + 0.05 * torch.randn(w.k_pool.shape, generator=g)).to(torch.bfloat16)
    ref, ref_lse = oracle.extend_attention_blocked(paged_inputs(w))
    assert ref_lse.max() < -100.0  # every row's scores are strongly negative
    cwlib.set_tuning(0, 1)
    try:
        out, lse = run_extend(to_gpu(w))
    finally:
        cwlib.set_tuning(0, 0)
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "negative split")
    # the kernel rounds the scaled query to bf16 once (relative 2^-9); here every
    # element of q is the same, so every score moves by the same relative amount
    # and lse (about -128) by up to 128 * 2^-9 = 0.25
    assert_close(lse.cpu().double().numpy(), ref_lse, 0.5, None, "negative split lse")
