"""Plans read by the kernels straight from the pinned staging slot
(CW_TUNE_PLAN_DIRECT = 1) give the same bits as plans copied into the workspace
first: extend (split and unsplit), decode, the fused write + extend and mixed
steps, bf16 and fp8 pools; the pools written by the fused and step calls too.
Several calls in a row cycle through the staging ring."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import paper_2606_16824_amd as cwlib
from gpu_util import bits, to_gpu

pytestmark = pytest.mark.gpu

PLAN_DIRECT = 4  # tuning key

CASES = {
    # name: (prefix lens, suffix lens, Hkv, G, D, P, kv dtype)
    "split_bf16": ([700, 90], [150, 64], 2, 4, 128, 16, "bf16"),
    "mixed_bf16": ([40, 0, 300, 17, 128, 999, 64], [1, 5, 1, 0, 70, 1, 33], 2, 4, 128, 16, "bf16"),
    "mixed_fp8_p64": ([65, 3, 500, 130], [1, 61, 1, 200], 2, 3, 64, 64, "fp8"),
    "decodes_fp8": ([0, 16, 33, 160, 1023], [1, 1, 1, 1, 1], 2, 4, 128, 16, "fp8"),
    "many_seqs": ([(37 * i) % 301 for i in range(40)], [1 + (11 * i) % 40 for i in range(40)],
                  2, 4, 128, 16, "bf16"),
}


def _raw(t):
    t = t.detach().cpu()
    return t.view(torch.int16).numpy() if t.dtype == torch.bfloat16 else t.view(torch.uint8).numpy()


def _calls(dw, s):
    """(name, out, lse, k_pool, v_pool) of every entry point that takes the case."""
    res = []
    lp, ls = s.prefix_lens, s.suffix_lens
    kw = dict(k_scale=dw.k_scale, v_scale=dw.v_scale)

    def fresh():
        out = torch.full_like(dw.q, float("nan"))
        lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device)
        return out, lse

    out, lse = fresh()
    kp, vp = dw.k_pool.clone(), dw.v_pool.clone()
    cwlib.step_attention(dw.q, dw.k_new, dw.v_new, kp, vp, dw.block_table, lp, ls, s.gqa_group,
                         s.softmax_scale, out=out, lse=lse, **kw)
    res.append(("step", out, lse, kp, vp))
    if np.all(ls == 1):
        out, lse = fresh()
        cwlib.decode_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table, lp,
                               s.gqa_group, s.softmax_scale, out=out, lse=lse, **kw)
        res.append(("decode", out, lse, None, None))
    out, lse = fresh()
    cwlib.extend_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table, lp, ls,
                           s.gqa_group, s.softmax_scale, out=out, lse=lse, **kw)
    res.append(("extend", out, lse, None, None))
    out, lse = fresh()
    kp, vp = dw.k_pool.clone(), dw.v_pool.clone()
    cwlib.write_extend_attention(dw.q, dw.k_new, dw.v_new, kp, vp, dw.block_table, lp, ls,
                                 s.gqa_group, s.softmax_scale, out=out, lse=lse, **kw)
    res.append(("fused", out, lse, kp, vp))
    torch.cuda.synchronize()
    return res


@pytest.mark.parametrize("name", list(CASES))
def test_direct_plan_reads_match_copied_plans(name):
    lp, ls, hkv, g, d, p, dt = CASES[name]
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p,
                          kv_dtype=dt, seed=31)
    print(f"\n[case] plan direct {name}: B={spec.num_seqs} G={g} D={d} P={p} {dt}", flush=True)
    dw = to_gpu(cw.materialize(spec))
    copied = _calls(dw, spec)
    cwlib.set_tuning(PLAN_DIRECT, 1)
    try:
        direct = [_calls(dw, spec) for _ in range(3)]  # 12-15 calls: the ring wraps
    finally:
        cwlib.set_tuning(PLAN_DIRECT, 0)
    for run in direct:
        for (na, oa, la, ka, va), (nb, ob, lb, kb, vb) in zip(copied, run):
            assert na == nb
            assert np.array_equal(bits(oa), bits(ob)), na
            assert np.array_equal(la.cpu().numpy().view(np.int32), lb.cpu().numpy().view(np.int32)), na
            if ka is not None:
                assert np.array_equal(_raw(ka), _raw(kb)) and np.array_equal(_raw(va), _raw(vb)), na
