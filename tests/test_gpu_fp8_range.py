"""fp8 pools at the edges of the documented scale range, against the oracle on
the same dequantised values.

The extend kernel computes in fp16: V pages with scale 140 (stored values up to
448 x 140 = 62720, near the fp16 limit 65504) next to pages with scale 0.004, and K
pages with scales from 0.003 to 0.5.  The decode kernel applies the scales in fp32
and takes scale 1000 (values up to 448 000).  Outputs must be finite; the error
bound is relative to the largest |V| a row can see: bf16 rounding of the weights
and of the output and fp16 rounding of the values, 3 x 2^-9 of max |V|, and 1e-2
of it is asserted (with the 6e-2 fp8-pool bound as a floor)."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import FP8_MAX_ABS, as_f64, run_extend, to_gpu

pytestmark = pytest.mark.gpu


def _scales(w, k_vals, v_vals):
    n, h = w.k_scale.shape
    idx = np.arange(n * h).reshape(n, h)
    w.k_scale = torch.from_numpy(np.asarray(k_vals, np.float32)[idx % len(k_vals)]).contiguous()
    w.v_scale = torch.from_numpy(np.asarray(v_vals, np.float32)[idx % len(v_vals)]).contiguous()


def _check(got, ref, inp, what):
    assert np.isfinite(got).all(), what
    vmax = 0.0
    for b in range(len(inp.suffix_lens)):
        _, v = oracle.gather_sequence_kv(inp, b)
        vmax = max(vmax, float(np.abs(v).max()))
    bound = max(FP8_MAX_ABS, 1e-2 * vmax)
    err = float(np.abs(got - ref).max())
    print(f"[{what}] max |V| {vmax:.4g}, max err {err:.4g}, bound {bound:.4g}", flush=True)
    assert err <= bound, (what, err, bound)


def test_extend_fp8_scales_near_the_fp16_limit():
    spec = cw.custom_spec([300, 120, 64], [40, 70, 1], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=16, kv_dtype="fp8", seed=4242)
    print("\n[case] fp8 range: extend, V scales 140 / 0.004, K scales 0.003-0.5", flush=True)
    w = cw.materialize(spec)
    _scales(w, [0.02, 0.003, 0.5, 0.05], [140.0, 0.004, 0.05, 140.0, 0.03])
    # the largest code (448, 0x7E) in the first keys of sequence 0's first page,
    # scale 140: stored values of 62720
    pg = int(w.block_table[0, 0])
    w.v_scale[pg, :] = 140.0
    w.v_pool.view(torch.uint8)[pg, :, 0:4, 0:16] = 0x7E
    out, lse = run_extend(to_gpu(w))
    inp = paged_inputs(w)
    ref, ref_lse = oracle.extend_attention_blocked(inp)
    _check(as_f64(out), ref, inp, "extend")
    assert torch.isfinite(lse).all()
    l = lse.cpu().double().numpy()
    assert np.abs(l - ref_lse).max() <= 1e-2 * max(1.0, np.abs(ref_lse).max())


def test_decode_fp8_large_scales():
    spec = cw.custom_spec([300, 1000, 17], [1, 1, 1], num_kv_heads=2, gqa_group=4, head_dim=128,
                          page_size=16, kv_dtype="fp8", seed=4243)
    print("\n[case] fp8 range: decode, V scales up to 1000", flush=True)
    w = cw.materialize(spec)
    _scales(w, [0.02, 0.5, 0.003], [1000.0, 0.004, 0.05, 250.0])
    dw = to_gpu(w)
    out = torch.full_like(dw.q, float("nan"))
    lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
    cwlib.decode_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                           spec.prefix_lens, spec.gqa_group, spec.softmax_scale, k_scale=dw.k_scale,
                           v_scale=dw.v_scale, out=out, lse=lse)
    torch.cuda.synchronize()
    inp = paged_inputs(w)
    ref, ref_lse = oracle.extend_attention_rowwise(inp)
    _check(as_f64(out), ref, inp, "decode")
    l = lse.cpu().double().numpy()
    assert np.isfinite(l).all()
    assert np.abs(l - ref_lse).max() <= 1e-2 * max(1.0, np.abs(ref_lse).max())
