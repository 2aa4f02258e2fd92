"""GPU cw_kv_write_pages: the whole pool must equal the oracle scatter bit for bit."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
import paper_2606_16824_amd as cwlib
from conftest import paged_inputs
from gpu_util import to_gpu

pytestmark = pytest.mark.gpu

CASES = {
    "tiny": ([256], [64], 1, 64, 16, "bf16"),
    "ragged": ([13, 0, 32, 7, 100], [9, 5, 0, 1, 70], 2, 128, 16, "bf16"),
    "p64": ([65, 3], [200, 61], 3, 64, 64, "bf16"),
    "fp8": ([13, 0, 32, 7], [9, 5, 17, 1], 2, 128, 16, "fp8"),
    "fp8_p64": ([65, 3], [200, 61], 2, 64, 64, "fp8"),
}


def _pool_np(t):
    t = t.cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()


@pytest.mark.parametrize("name", list(CASES))
def test_write_pages_bit_exact(name):
    lp, ls, hkv, d, p, dt = CASES[name]
    spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=1, head_dim=d, page_size=p,
                          kv_dtype=dt, seed=len(name))
    print(f"\n[case] write_pages {name}: {spec.prefix_lens.tolist()} {spec.suffix_lens.tolist()}", flush=True)
    w = cw.materialize(spec)
    if dt == "fp8":
        # values far past 448 * scale must saturate to +-448
        w.k_new[0, 0, :2] = torch.tensor([1e4, -1e4]).to(torch.bfloat16)
    dw = to_gpu(w)
    cwlib.kv_write_pages(dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                         spec.prefix_lens, spec.suffix_lens, k_scale=dw.k_scale, v_scale=dw.v_scale)
    torch.cuda.synchronize()
    want_k, want_v = oracle.write_pages(paged_inputs(w))
    got_k, got_v = _pool_np(dw.k_pool), _pool_np(dw.v_pool)
    nk = int((got_k != want_k).sum())
    nv = int((got_v != want_v).sum())
    print(f"[{name}] mismatching elements: K {nk}, V {nv}", flush=True)
    assert nk == 0 and nv == 0
