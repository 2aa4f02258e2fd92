"""Seeded random shapes against the oracle on the GPU: ragged lengths (empty
suffixes, empty prefixes, one-token suffixes, ragged page tails), GQA groups 1-16,
1-4 kv heads, D 64/128, P 16/64, bf16 and fp8 pools, through cw_step_attention
(decodes on the decode kernel, extends on the extend kernel, page write fused),
with the planner's tunings drawn too (forced chunk sizes, suffix weights, dealt
rounds).  Every case is printed before it runs; the list is fixed by its seed."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import BF16_MAX_ABS, BF16_MEAN_ABS, FP8_MAX_ABS, as_f64, assert_close, to_gpu

pytestmark = pytest.mark.gpu

N_CASES = 30


def _case(i):
    rng = np.random.default_rng(7000 + i)
    b = int(rng.integers(1, 7))
    lp = [int(x) for x in rng.choice([0, 1, 15, 16, 17, 63, 64, 65, 200, 777, 1500], size=b)]
    ls = [int(x) for x in rng.choice([0, 1, 1, 2, 31, 64, 65, 100, 257, 400], size=b)]
    if sum(ls) == 0:
        ls[0] = 5
    hkv = int(rng.choice([1, 2, 4]))
    g = int(rng.choice([1, 2, 3, 4, 8, 16]))
    d = int(rng.choice([64, 128]))
    p = int(rng.choice([16, 64]))
    dt = str(rng.choice(["bf16", "fp8"]))
    tune = (int(rng.choice([0, 0, 2, 5])), int(rng.choice([100, 125, 300])), int(rng.choice([0, 1])))
    return lp, ls, hkv, g, d, p, dt, tune


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_step_against_oracle(i):
    lp, ls, hkv, g, d, p, dt, (chunk, weight, deal) = _case(i)
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p,
                          kv_dtype=dt, seed=900 + i)
    print(f"\n[case] random {i}: Lp={lp} Ls={ls} Hkv={hkv} G={g} D={d} P={p} {dt} "
          f"chunk={chunk} weight={weight} deal={deal}", flush=True)
    w = cw.materialize(spec)
    dw = to_gpu(w)
    out = torch.full_like(dw.q, float("nan"))
    lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
    kp, vp = dw.k_pool.clone(), dw.v_pool.clone()
    cwlib.set_tuning(0, chunk)
    cwlib.set_tuning(5, weight)
    cwlib.set_tuning(3, deal)
    try:
        cwlib.step_attention(dw.q, dw.k_new, dw.v_new, kp, vp, dw.block_table, spec.prefix_lens,
                             spec.suffix_lens, g, spec.softmax_scale, k_scale=dw.k_scale,
                             v_scale=dw.v_scale, out=out, lse=lse)
        torch.cuda.synchronize()
    finally:
        cwlib.set_tuning(0, 0)
        cwlib.set_tuning(5, 125)
        cwlib.set_tuning(3, 1)
    inp = paged_inputs(w)
    ref, ref_lse = oracle.extend_attention_blocked(inp)
    got = as_f64(out)
    assert np.isfinite(got).all() and torch.isfinite(lse).all()
    if dt == "bf16":
        assert_close(got, ref, BF16_MAX_ABS, BF16_MEAN_ABS, f"random {i}")
    else:
        assert_close(got, ref, FP8_MAX_ABS, None, f"random {i}")
    assert_close(lse.cpu().double().numpy(), ref_lse, 1e-2, None, f"random {i} lse")
    # the pools hold exactly the oracle's page write
    wk, wv = oracle.write_pages(inp)
    raw = (lambda t: t.view(torch.int16).numpy()) if kp.dtype == torch.bfloat16 else (lambda t: t.view(torch.uint8).numpy())
    assert np.array_equal(raw(kp.cpu()), wk.view(np.int16) if kp.dtype == torch.bfloat16 else wk)
    assert np.array_equal(raw(vp.cpu()), wv.view(np.int16) if vp.dtype == torch.bfloat16 else wv)
