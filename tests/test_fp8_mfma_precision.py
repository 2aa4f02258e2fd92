"""What an fp8 matrix product would cost in precision on fp8 pools.  An fp8
(e4m3fn) matrix product needs both operands in fp8, so besides the cached K or V
codes the other operand, Q (for Q K^T) or the softmax weights P (for P V), would
have to be rounded to e4m3fn, whose step is 2^-4 relative.
This emulates those roundings on the oracle's own inputs, the small fp8-pool
shapes of the GPU parity suite, in float64 (the causal softmax attention of the
oracle with one rounding inserted at a time), and measures the max-abs error
against the exact oracle next to the fp8-pool bound.

Models (per query row; K, V the exact dequantised values, so the page scales are
applied exactly in every model):
  bf16 path  scores exact; P = exp(s - rowmax) rounded to bf16; the row sum is
             the sum of the rounded weights (what the kernels compute)
  fp8 Q      q / 2^e rounded to e4m3fn, with 2^e the smallest power of two that
             brings max |q| within 448, then as the bf16 path
  fp8 P      cached-prefix weights as e4m3fn(256 P) / 256 (the suffix keys keep
             bf16 weights, since their V is bf16); sum of the rounded weights
These are favourable to fp8: the row max is exact (the kernels track a running
one), and the new tokens' bf16 K and V rows, which an fp8 product would also have
to round, stay exact.
"""
import zlib

import numpy as np
import pytest
import torch

import cw_workloads as cw
import oracle
from conftest import paged_inputs
from gpu_util import FP8_MAX_ABS

# the fp8-pool cases of the GPU parity suite: (prefix lens, suffix lens, Hkv, G, D, P)
FP8_CASES = {
    "fp8_small": ([50, 300], [30, 60], 2, 4, 128, 16),
    "fp8_p64_d64": ([129, 64], [1, 77], 1, 2, 64, 64),
    "gqa16_d128_fp8": ([200, 17], [24, 3], 1, 16, 128, 16),
    "fp8_p64_d128": ([129, 64, 300], [33, 90, 1], 2, 4, 128, 64),
    "fp8_p16_d64": ([50, 130, 17], [20, 45, 3], 2, 4, 64, 16),
}


def _bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).double().numpy()


def _e4m3(x):
    return oracle.e4m3fn_decode(oracle.e4m3fn_encode_rne(np.asarray(x, dtype=np.float64)))


def _row(model, q, k, v, n, lp, scale):
    """One query row against its n visible keys (lp of them cached) in `model`."""
    if model == "fp8_q":
        e = np.ceil(np.log2(np.abs(q).max() / 448.0)) if np.abs(q).max() > 0 else 0.0
        q = _e4m3(q / 2.0 ** e) * 2.0 ** e
    s = scale * (k[:n] @ q)
    p = np.exp(s - s.max())
    if model in ("bf16", "fp8_q"):
        p = _bf16(p)
    elif model == "fp8_p":
        c = min(lp, n)
        p = np.concatenate([_e4m3(256.0 * p[:c]) / 256.0, _bf16(p[c:])])
    return (p @ v[:n]) / p.sum()


def _emulate(inp, model):
    g = inp.gqa_group
    out = np.zeros(inp.q.shape, dtype=np.float64)
    q_all = oracle.bf16_bits_to_f64(inp.q)
    cu = inp.cu()
    for b in range(len(inp.suffix_lens)):
        lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
        k, v = oracle.gather_sequence_kv(inp, b)
        for i in range(ls):
            r = int(cu[b]) + i
            for h in range(inp.q.shape[1]):
                out[r, h] = _row(model, q_all[r, h], k[:, h // g], v[:, h // g], lp + i + 1, lp,
                                 inp.softmax_scale)
    return out


@pytest.fixture(scope="module")
def errors():
    res = {}
    for name, (lp, ls, hkv, g, d, p) in FP8_CASES.items():
        spec = cw.custom_spec(lp, ls, num_kv_heads=hkv, gqa_group=g, head_dim=d, page_size=p,
                              kv_dtype="fp8", seed=zlib.crc32(name.encode()) % 1000)
        inp = paged_inputs(cw.materialize(spec))
        ref, _ = oracle.extend_attention_blocked(inp)
        res[name] = {m: float(np.abs(_emulate(inp, m) - ref).max())
                     for m in ("exact", "bf16", "fp8_q", "fp8_p")}
    for name, e in res.items():
        print(f"[fp8 mfma] {name}: " + " ".join(f"{m} {x:.3e}" for m, x in e.items()))
    return res


def test_harness_without_rounding_is_the_oracle(errors):
    assert max(e["exact"] for e in errors.values()) < 1e-12


def test_bf16_path_model_is_far_inside_the_bound(errors):
    assert max(e["bf16"] for e in errors.values()) < 0.1 * FP8_MAX_ABS


def test_fp8_q_uses_more_than_half_the_bound(errors):
    worst = max(e["fp8_q"] for e in errors.values())
    assert 0.5 * FP8_MAX_ABS < worst < FP8_MAX_ABS, worst
    for e in errors.values():
        assert e["fp8_q"] > 10 * e["bf16"]


def test_fp8_p_on_the_prefix_fits_in_half_the_bound(errors):
    worst = max(e["fp8_p"] for e in errors.values())
    assert 0.2 * FP8_MAX_ABS < worst < 0.5 * FP8_MAX_ABS, worst
    for e in errors.values():
        assert e["fp8_p"] > 10 * e["bf16"]
