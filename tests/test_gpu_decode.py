"""GPU parity of cw_decode_attention (one new token per sequence) against the oracle."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import (BF16_MAX_ABS, BF16_MEAN_ABS, FP8_MAX_ABS, as_f64, assert_close,
                      assert_within_bf16_ulps, to_gpu)

pytestmark = pytest.mark.gpu


def _run_decode(dw):
    s = dw.spec
    out = torch.full_like(dw.q, float("nan"))
    lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
    cwlib.decode_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                           s.prefix_lens, s.gqa_group, s.softmax_scale, k_scale=dw.k_scale,
                           v_scale=dw.v_scale, out=out, lse=lse)
    torch.cuda.synchronize()
    return out, lse


CASES = {
    # name: (prefix lens, Hkv, G, D, P, kv)
    "mixed_lens_bf16": ([0, 1, 15, 16, 17, 31, 32, 33, 1023, 1024, 1025, 4000], 2, 4, 128, 16, "bf16"),
    "mixed_lens_fp8": ([0, 1, 15, 16, 17, 31, 32, 33, 1023, 1024, 1025, 4000], 2, 4, 128, 16, "fp8"),
    "p64_g8_bf16": ([63, 64, 65, 5000], 2, 8, 128, 64, "bf16"),
    "p64_g8_fp8": ([63, 64, 65, 5000], 2, 8, 128, 64, "fp8"),
    "d64_bf16": ([100, 2047, 2048, 2049], 3, 2, 64, 16, "bf16"),
    "d64_fp8_p64": ([100, 4095, 4096, 9000], 1, 16, 64, 64, "fp8"),
    "d64_fp8_p16": ([100, 2047, 2048, 2049], 2, 4, 64, 16, "fp8"),
    "d64_bf16_p64": ([63, 64, 65, 3000], 2, 2, 64, 64, "bf16"),
    "mqa_g1": ([300, 7], 1, 1, 128, 16, "bf16"),
}


@pytest.mark.parametrize("name", list(CASES))
def test_decode_against_oracle(name):
    lp, hkv, g, d, p, dt = CASES[name]
    spec = cw.custom_spec(lp, [1] * len(lp), num_kv_heads=hkv, gqa_group=g, head_dim=d,
                          page_size=p, kv_dtype=dt, seed=len(name) * 7)
    print(f"\n[case] decode {name}: Lp={lp} Hkv={hkv} G={g} D={d} P={p} {dt}", flush=True)
    w = cw.materialize(spec)
    out, lse = _run_decode(to_gpu(w))
    ref, ref_lse = oracle.extend_attention_rowwise(paged_inputs(w))
    if dt == "bf16":
        assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, name)
    else:
        assert_close(as_f64(out), ref, FP8_MAX_ABS, None, name)
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, name + " lse")


@pytest.mark.parametrize("chunk_tiles", [1, 2, 5])
@pytest.mark.parametrize("dt", ["bf16", "fp8"])
def test_decode_chunking_invariance(chunk_tiles, dt):
    spec = cw.custom_spec([3000, 64, 129], [1, 1, 1], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=16, kv_dtype=dt, seed=99)
    print(f"\n[case] decode chunk {chunk_tiles} {dt}", flush=True)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    base, base_lse = _run_decode(dw)
    cwlib.set_tuning(0, chunk_tiles)
    try:
        out, lse = _run_decode(dw)
    finally:
        cwlib.set_tuning(0, 0)
    assert_within_bf16_ulps(as_f64(out), as_f64(base), 2, "chunked vs default")
    assert_close(lse.cpu().double().numpy(), base_lse.cpu().double().numpy(), 1e-4, None, "lse")
    ref, _ = oracle.extend_attention_rowwise(paged_inputs(w))
    tol = BF16_MAX_ABS if dt == "bf16" else FP8_MAX_ABS
    assert_close(as_f64(out), ref, tol, None, "chunked vs oracle")


def test_decode_page_permutation_bitwise():
    spec = cw.custom_spec([2500, 33], [1, 1], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=16, kv_dtype="fp8", seed=5)
    w = cw.materialize(spec)
    a, _ = _run_decode(to_gpu(w))
    rng = np.random.default_rng(3)
    perm = torch.from_numpy(rng.permutation(spec.num_pages).astype(np.int64))
    for name in ("k_pool", "v_pool", "k_scale", "v_scale"):
        t = getattr(w, name)
        t2 = torch.empty_like(t)
        t2[perm] = t
        setattr(w, name, t2)
    bt = w.block_table.clone()
    used = bt != cw.BT_UNUSED
    bt[used] = perm[bt[used].long()].to(torch.int32)
    w.block_table = bt
    b, _ = _run_decode(to_gpu(w))
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("name", ["decode", "decode_bf16", "decode_long"])
def test_decode_full_size(name):
    """Every row of the full-size decode workloads against the oracle."""
    w = cw.make(name)
    s = w.spec
    print(f"\n[case] full {name}: B={s.num_seqs}", flush=True)
    out, lse = _run_decode(to_gpu(w))
    assert bool(torch.isfinite(out).all()) and bool(torch.isfinite(lse).all())
    ref, ref_lse = oracle.extend_attention_blocked(paged_inputs(w))
    tol = BF16_MAX_ABS if s.kv_dtype == "bf16" else FP8_MAX_ABS
    assert_close(as_f64(out), ref, tol, BF16_MEAN_ABS if s.kv_dtype == "bf16" else None, f"full {name}")
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, f"full {name} lse")


@pytest.mark.parametrize("n_seqs", [2048, 2049])
def test_decode_plan_upload_forms(n_seqs):
    """Decode plans are uploaded in compact form (rebuilt on the device) up to
    2048 sequences and as full work lists beyond: both against the oracle, and
    the compact upload switched off (CW_TUNE_COMPACT_DECODE 0) bit-identical."""
    rng = np.random.default_rng(n_seqs)
    lp = [int(x) for x in rng.integers(0, 200, size=n_seqs)]
    spec = cw.custom_spec(lp, [1] * n_seqs, num_kv_heads=2, gqa_group=4, head_dim=64, page_size=16,
                          kv_dtype="bf16", seed=n_seqs)
    print(f"\n[case] decode plan upload: {n_seqs} sequences", flush=True)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    out, lse = _run_decode(dw)
    cwlib.set_tuning(6, 0)
    try:
        out_full, lse_full = _run_decode(dw)
    finally:
        cwlib.set_tuning(6, 1)
    assert torch.equal(out.view(torch.int16), out_full.view(torch.int16))
    assert torch.equal(lse, lse_full)
    ref, ref_lse = oracle.extend_attention_rowwise(paged_inputs(w))
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, f"{n_seqs} sequences")
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, f"{n_seqs} sequences lse")
