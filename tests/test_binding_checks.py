"""The binding's marshalling checks: every tensor's dtype and shape is checked
against the call's lengths before any pointer reaches the library (the C side
cannot see tensor sizes).  The tensors here live on the CPU: a call whose
tensors pass every check stops at the device check instead, so each case shows
which check fired.  Runs without a GPU."""
import numpy as np
import pytest
import torch

import paper_2606_16824_amd as cwlib

LP, LS = [40, 0, 17], [5, 3, 1]
T, HKV, G, D, NP, P = sum(LS), 2, 4, 64, 16, 16


def _args(kv="bf16"):
    bf = torch.bfloat16
    pool_dt = bf if kv == "bf16" else torch.uint8
    a = dict(q=torch.zeros(T, HKV * G, D, dtype=bf), k_new=torch.zeros(T, HKV, D, dtype=bf),
             v_new=torch.zeros(T, HKV, D, dtype=bf),
             k_pool=torch.zeros(NP, HKV, P, D, dtype=pool_dt),
             v_pool=torch.zeros(NP, HKV, P, D, dtype=pool_dt),
             block_table=torch.zeros(3, 8, dtype=torch.int32),
             k_scale=None, v_scale=None, out=torch.zeros(T, HKV * G, D, dtype=bf),
             lse=torch.zeros(T, HKV * G, dtype=torch.float32))
    if kv == "fp8":
        a["k_scale"] = torch.ones(NP, HKV)
        a["v_scale"] = torch.ones(NP, HKV)
    return a


def _extend(a, fn=cwlib.extend_attention):
    return fn(a["q"], a["k_new"], a["v_new"], a["k_pool"], a["v_pool"], a["block_table"], LP, LS,
              G, 0.125, k_scale=a["k_scale"], v_scale=a["v_scale"], out=a["out"], lse=a["lse"])


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("fn", [cwlib.extend_attention, cwlib.write_extend_attention,
                                cwlib.step_attention])
def test_valid_shapes_reach_the_device_check(kv, fn):
    with pytest.raises(ValueError, match="on the GPU"):
        _extend(_args(kv), fn)


BAD = [
    ("block_table", lambda a: a["block_table"].long(), "block_table must be a 2-D int32"),
    ("block_table", lambda a: a["block_table"][:2], "rows for 3 sequences"),
    ("block_table", lambda a: a["block_table"].flatten(), "block_table must be a 2-D int32"),
    ("q", lambda a: a["q"][:-1], "q has shape"),
    ("q", lambda a: a["q"].float(), "q has dtype"),
    ("out", lambda a: a["out"][:, :4], "out has shape"),
    ("out", lambda a: a["out"].half(), "out has dtype"),
    ("k_new", lambda a: a["k_new"][:, :1], "k_new has shape"),
    ("v_new", lambda a: a["v_new"].float(), "v_new has dtype"),
    ("lse", lambda a: a["lse"][:-1], "lse has shape"),
    ("lse", lambda a: a["lse"].double(), "lse has dtype"),
    ("v_pool", lambda a: a["v_pool"][:-1], "v_pool has shape"),
    ("v_pool", lambda a: a["v_pool"].float(), "v_pool has dtype"),
    ("k_pool", lambda a: a["k_pool"][0], "k_pool must be a 4-D"),
    ("k_scale", lambda a: torch.ones(NP, HKV), "fp8 pools only"),
]


@pytest.mark.parametrize("name,bad,msg", BAD)
def test_bf16_call_rejects(name, bad, msg):
    a = _args("bf16")
    a[name] = bad(a)
    with pytest.raises(ValueError, match=msg):
        _extend(a)


FP8_BAD = [
    ("k_scale", lambda a: None, "needs k_scale and v_scale"),
    ("v_scale", lambda a: a["v_scale"].double(), "v_scale has dtype"),
    ("k_scale", lambda a: a["k_scale"][:, :1], "k_scale has shape"),
    ("v_pool", lambda a: a["v_pool"].view(torch.float8_e4m3fn), "v_pool has dtype"),
]


@pytest.mark.parametrize("name,bad,msg", FP8_BAD)
def test_fp8_call_rejects(name, bad, msg):
    a = _args("fp8")
    a[name] = bad(a)
    with pytest.raises(ValueError, match=msg):
        _extend(a)


def test_lens_must_pair_up():
    a = _args()
    with pytest.raises(ValueError, match="must be 1-D of one length"):
        cwlib.extend_attention(a["q"], a["k_new"], a["v_new"], a["k_pool"], a["v_pool"],
                               a["block_table"], LP, LS[:2], G, 0.125)


def test_decode_and_write_pages_check_too():
    a = _args()
    lp = [40, 0, 17]
    q = torch.zeros(3, HKV * G, D, dtype=torch.bfloat16)
    kn = torch.zeros(3, HKV, D, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="q has shape"):
        cwlib.decode_attention(q[:2], kn, kn, a["k_pool"], a["v_pool"], a["block_table"], lp, G, 0.1)
    with pytest.raises(ValueError, match="on the GPU"):
        cwlib.decode_attention(q, kn, kn, a["k_pool"], a["v_pool"], a["block_table"], lp, G, 0.1)
    with pytest.raises(ValueError, match="k_new has shape"):
        cwlib.kv_write_pages(a["k_new"][:-1], a["v_new"], a["k_pool"], a["v_pool"],
                             a["block_table"], LP, LS)
    with pytest.raises(ValueError, match="block_table must be a 2-D int32"):
        cwlib.kv_write_pages(a["k_new"], a["v_new"], a["k_pool"], a["v_pool"],
                             a["block_table"].long(), LP, LS)
    with pytest.raises(ValueError, match="on the GPU"):
        cwlib.kv_write_pages(a["k_new"], a["v_new"], a["k_pool"], a["v_pool"], a["block_table"],
                             LP, LS)
