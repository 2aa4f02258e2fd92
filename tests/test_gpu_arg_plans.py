"""Plans in the kernel arguments, against plans uploaded through the staging ring.

Extend plans of up to 16 KB, and decode plans whose compact form (one record
per sequence, the order of the last chunks, the rebuild descriptor) fits in
16 KB, travel in the arguments of the attention and merge kernels, which rebuild
a compact decode plan's items and merge groups where they read them.
CW_TUNE_ARG_PLANS 0 uploads every plan instead.  Each case runs both ways,
bit-identical, and against the oracle: decode calls and steps of decodes only
(bf16 and fp8 pools, split and unsplit sequences, one and many chunks per
sequence), a decode call whose compact plan just fits the arguments (360
sequences) and one too large for them (400 sequences, uploaded either way),
extend calls and steps of extends only."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import BF16_MAX_ABS, BF16_MEAN_ABS, FP8_MAX_ABS, as_f64, assert_close, to_gpu

pytestmark = pytest.mark.gpu

ARG_PLANS = 7  # CW_TUNE_ARG_PLANS

# name: (entry point, prefix lens, suffix lens, Hkv, G, D, P, kv); every case's
# plan travels in the kernel arguments except decode_400's
CASES = {
    "decode_bf16": ("decode", [0, 1, 15, 300, 1023, 1025, 4000, 9000], None, 2, 4, 128, 16, "bf16"),
    "decode_fp8": ("decode", [0, 1, 15, 300, 1023, 1025, 4000, 9000], None, 2, 4, 128, 16, "fp8"),
    "decode_d64_p64": ("decode", [63, 64, 65, 5000, 20000], None, 2, 8, 64, 64, "fp8"),
    "decode_step_bf16": ("step", [5, 700, 2000, 33, 12000], [1, 1, 1, 1, 1], 2, 4, 128, 16, "bf16"),
    "decode_step_fp8": ("step", [5, 700, 2000, 33, 12000], [1, 1, 1, 1, 1], 2, 4, 128, 16, "fp8"),
    # 360 sequences: a compact plan of about 16 KB, the largest that fits the arguments
    "decode_360": ("decode", 360, None, 1, 4, 64, 16, "bf16"),
    "decode_400": ("decode", 400, None, 1, 4, 64, 16, "bf16"),
    "extend_bf16": ("extend", [700, 90, 3000], [150, 64, 300], 2, 4, 128, 16, "bf16"),
    "extend_step_fp8": ("step", [700, 0, 3000], [150, 64, 300], 2, 4, 128, 16, "fp8"),
}


def _run(kind, spec, dw):
    s = spec
    out = torch.full_like(dw.q, float("nan"))
    lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
    args = (dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table)
    kw = dict(k_scale=dw.k_scale, v_scale=dw.v_scale, out=out, lse=lse)
    if kind == "decode":
        cwlib.decode_attention(*args, s.prefix_lens, s.gqa_group, s.softmax_scale, **kw)
    elif kind == "extend":
        cwlib.extend_attention(*args, s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale, **kw)
    else:
        cwlib.step_attention(*args, s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale, **kw)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("name", list(CASES))
def test_arg_plan_matches_uploaded_plan(name):
    kind, lp, ls, hkv, g, d, p, dt = CASES[name]
    if isinstance(lp, int):
        lp = [int(x) for x in np.random.default_rng(lp).integers(0, 300, size=lp)]
    if ls is None:
        ls = [1] * len(lp)
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p, kv_dtype=dt,
                          seed=9300 + len(name))
    print(f"\n[case] arg plans {name}: {kind} B={len(lp)} Hkv={hkv} G={g} D={d} P={p} {dt}", flush=True)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    # a step of decodes only writes each new token into its page: start both runs from the same pools
    k0, v0 = dw.k_pool.clone(), dw.v_pool.clone()
    n0 = cwlib.arg_plan_calls()
    out_a, lse_a = _run(kind, spec, dw)
    assert cwlib.arg_plan_calls() - n0 == (0 if name == "decode_400" else 1), name
    dw.k_pool.copy_(k0)
    dw.v_pool.copy_(v0)
    cwlib.set_tuning(ARG_PLANS, 0)
    try:
        n0 = cwlib.arg_plan_calls()
        out_u, lse_u = _run(kind, spec, dw)
        assert cwlib.arg_plan_calls() == n0, name
    finally:
        cwlib.set_tuning(ARG_PLANS, 1)
    assert torch.equal(out_a.view(torch.int16), out_u.view(torch.int16)), name
    assert torch.equal(lse_a.view(torch.int32), lse_u.view(torch.int32)), name
    inp = paged_inputs(w)
    ref, ref_lse = oracle.extend_attention_rowwise(inp) if kind != "extend" and max(ls) == 1 \
        else oracle.extend_attention_blocked(inp)
    assert_close(as_f64(out_a), ref, BF16_MAX_ABS if dt == "bf16" else FP8_MAX_ABS,
                 BF16_MEAN_ABS if dt == "bf16" else None, name)
    assert_close(lse_a.cpu().double().numpy(), ref_lse, 1e-2, None, name + " lse")
