"""GPU cw_step_attention: a mixed chunked-prefill step (extends and decodes).

Decode rows must be bit-identical to cw_decode_attention of the decode
sequences alone, the other rows to cw_extend_attention of the extending
sequences alone, the pools to cw_kv_write_pages, and everything within the
tolerance of the oracle."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import BF16_MAX_ABS, BF16_MEAN_ABS, FP8_MAX_ABS, as_f64, assert_close, bits, to_gpu

pytestmark = pytest.mark.gpu

CASES = {
    "bf16_mixed": ([40, 0, 300, 17, 128, 999, 64], [1, 5, 1, 0, 70, 1, 33], 2, 4, 128, 16, "bf16"),
    "fp8_mixed_p64": ([65, 3, 500, 130], [1, 61, 1, 200], 2, 3, 64, 64, "fp8"),
    "fp8_mixed_p64_d128": ([700, 64, 129], [1, 150, 70], 2, 4, 128, 64, "fp8"),
    "decodes_only": ([100, 7, 250], [1, 1, 1], 1, 8, 128, 16, "bf16"),
    # the decode launch performs the page write; new tokens at page starts (Lp = 0, 16, 160, 64)
    "decodes_only_fp8": ([0, 16, 33, 160, 1023], [1, 1, 1, 1, 1], 2, 4, 128, 16, "fp8"),
    "decodes_only_fp8_p64_d64": ([64, 5, 700], [1, 1, 1], 3, 2, 64, 64, "fp8"),
    "decodes_only_bf16_p64": ([0, 64, 4100], [1, 1, 1], 2, 8, 128, 64, "bf16"),
    "extends_only": ([31, 200], [9, 40], 2, 2, 128, 16, "fp8"),
}


def _rows(spec, seqs):
    cu = np.concatenate([[0], np.cumsum(spec.suffix_lens)])
    return np.concatenate([np.arange(cu[b], cu[b + 1]) for b in seqs]).astype(np.int64) if len(seqs) else np.zeros(0, np.int64)


def _raw(t):
    t = t.detach().cpu()
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.view(torch.uint8).numpy()


def _check(spec, name, with_oracle=True):
    print(f"\n[case] step {name}: Lp={spec.prefix_lens.tolist()[:8]} Ls={spec.suffix_lens.tolist()[:8]} "
          f"{spec.kv_dtype}", flush=True)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    ls = spec.suffix_lens
    dec = [b for b in range(len(ls)) if ls[b] == 1]
    ext = [b for b in range(len(ls)) if ls[b] > 1]
    kp, vp = dw.k_pool.clone(), dw.v_pool.clone()
    out = torch.full_like(dw.q, float("nan"))
    lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
    cwlib.step_attention(dw.q, dw.k_new, dw.v_new, kp, vp, dw.block_table, spec.prefix_lens, ls,
                         spec.gqa_group, spec.softmax_scale, k_scale=dw.k_scale, v_scale=dw.v_scale,
                         out=out, lse=lse)
    torch.cuda.synchronize()
    # pools: the page write of the whole step
    kw, vw = dw.k_pool.clone(), dw.v_pool.clone()
    cwlib.kv_write_pages(dw.k_new, dw.v_new, kw, vw, dw.block_table, spec.prefix_lens, ls,
                         k_scale=dw.k_scale, v_scale=dw.v_scale)
    torch.cuda.synchronize()
    assert (_raw(kp) == _raw(kw)).all() and (_raw(vp) == _raw(vw)).all()
    # sub-batches through the single-kernel calls (on the unwritten pools)
    for seqs, kind in ((dec, "decode"), (ext, "extend")):
        if not seqs:
            continue
        rows = torch.from_numpy(_rows(spec, seqs)).cuda()
        sq, skn, svn = dw.q[rows].contiguous(), dw.k_new[rows].contiguous(), dw.v_new[rows].contiguous()
        sbt = dw.block_table[torch.tensor(seqs, device="cuda")].contiguous()
        o = torch.full_like(sq, float("nan"))
        l2 = torch.full((sq.shape[0], sq.shape[1]), float("nan"), device=sq.device)
        if kind == "decode":
            cwlib.decode_attention(sq, skn, svn, dw.k_pool, dw.v_pool, sbt, spec.prefix_lens[seqs],
                                   spec.gqa_group, spec.softmax_scale, k_scale=dw.k_scale,
                                   v_scale=dw.v_scale, out=o, lse=l2)
        else:
            cwlib.extend_attention(sq, skn, svn, dw.k_pool, dw.v_pool, sbt, spec.prefix_lens[seqs],
                                   ls[seqs], spec.gqa_group, spec.softmax_scale, k_scale=dw.k_scale,
                                   v_scale=dw.v_scale, out=o, lse=l2)
        torch.cuda.synchronize()
        n_out = int((bits(out[rows]) != bits(o)).sum())
        n_lse = int((lse[rows].cpu().numpy().view(np.uint32) != l2.cpu().numpy().view(np.uint32)).sum())
        print(f"[{name}] {kind} rows ({len(seqs)} seqs): differing out {n_out}, lse {n_lse}", flush=True)
        assert n_out == 0 and n_lse == 0
    if with_oracle:
        ref, _ = oracle.extend_attention_blocked(paged_inputs(w))
        if spec.kv_dtype == "bf16":
            assert_close(as_f64(out), ref, BF16_MAX_ABS, BF16_MEAN_ABS, name)
        else:
            assert_close(as_f64(out), ref, FP8_MAX_ABS, None, name)


@pytest.mark.parametrize("name", list(CASES))
def test_step_matches_single_kernel_calls_and_oracle(name):
    lp, ls, hkv, g, d, p, dt = CASES[name]
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p,
                          kv_dtype=dt, seed=31 + len(name))
    _check(spec, name)


def test_step_mixed_full_size():
    _check(cw.spec_for("mixed"), "mixed", with_oracle=False)


def test_step_decodes_full_size():
    _check(cw.spec_for("decode"), "decode", with_oracle=False)
