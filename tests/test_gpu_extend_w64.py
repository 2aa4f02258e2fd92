"""GPU parity of the four-wave extend kernel (64 query rows per wave), selected with
CW_TUNE_EXTEND_KERNEL = 2, against the oracle and against the default eight-wave
kernel (bf16 pools).  Tolerances as in test_gpu_extend.py; the two kernels sum the
same bf16-rounded weights in another order, so they agree within 2 bf16 ulps."""
import zlib

import pytest

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import (BF16_MAX_ABS, BF16_MEAN_ABS, as_f64, assert_close, assert_within_bf16_ulps,
                      run_extend, to_gpu)

pytestmark = pytest.mark.gpu

KERNEL = cwlib._lib.CW_TUNE_EXTEND_KERNEL

CASES = {
    # name: (prefix lens, suffix lens, Hkv, G, D, P)
    "tiny_shape": ([256], [64], 1, 4, 64, 16),
    "ragged_mha": ([0, 37, 200, 64], [70, 1, 129, 33], 2, 1, 128, 16),
    "gqa8_p64": ([100, 513], [45, 100], 2, 8, 128, 64),
    "gqa3_d64": ([31, 0, 95], [17, 40, 3], 3, 3, 64, 16),
    "empty_seq": ([40, 10, 0], [0, 20, 0], 1, 4, 128, 16),
    "long_tail": ([1000], [300], 2, 4, 128, 16),
    "gqa16_p64_d64": ([77], [9], 1, 16, 64, 64),
    "odd_tiles_p64": ([96, 160, 33], [31, 65, 200], 2, 4, 128, 64),
    "many_seqs": ([(37 * i) % 301 for i in range(40)], [1 + (11 * i) % 40 for i in range(40)],
                  2, 4, 128, 16),
}


def _run(dw, kernel, chunk_tiles=0):
    cwlib.set_tuning(KERNEL, kernel)
    cwlib.set_tuning(0, chunk_tiles)
    try:
        return run_extend(dw)
    finally:
        cwlib.set_tuning(KERNEL, 0)
        cwlib.set_tuning(0, 0)


@pytest.mark.parametrize("name", list(CASES))
def test_w64_against_oracle_and_eight_wave(name):
    lp, ls, hkv, g, d, p = CASES[name]
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p,
                          seed=zlib.crc32(name.encode()) % 1000)
    print(f"\n[case] w64 {name}: Lp={lp[:8]} Ls={ls[:8]} Hkv={hkv} G={g} D={d} P={p}", flush=True)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    out, lse = _run(dw, 2)
    ref, ref_lse = oracle.extend_attention_blocked(paged_inputs(w))
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, f"w64 {name}")
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, f"w64 {name} lse")
    base, _ = _run(dw, 1)
    assert_within_bf16_ulps(as_f64(out), as_f64(base), 2, f"w64 vs eight-wave {name}")


@pytest.mark.parametrize("chunk_tiles", [1, 3])
def test_w64_forced_split(chunk_tiles):
    spec = cw.custom_spec([700, 90], [150, 64], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=64, seed=78)
    print(f"\n[case] w64 split{chunk_tiles}", flush=True)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    out, _ = _run(dw, 2, chunk_tiles)
    ref, _ = oracle.extend_attention_blocked(paged_inputs(w))
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "w64 split vs oracle")
    base, _ = _run(dw, 2)
    assert_within_bf16_ulps(as_f64(out), as_f64(base), 2, "w64 split vs unsplit")


def test_w64_full_turn():
    w = cw.make("turn")
    print("\n[case] w64 full turn", flush=True)
    dw = to_gpu(w)
    out, lse = _run(dw, 2)
    ref, ref_lse = oracle.extend_attention_blocked(paged_inputs(w))
    assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, "w64 full turn")
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, "w64 full turn lse")
