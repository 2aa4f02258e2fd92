"""Calls captured into a HIP graph (torch.cuda.CUDAGraph) and replayed.

A captured call carries its plan in the arguments of its copy kernels, so each
replay writes the plan it was captured with.  Between replays the test runs
eager calls of other shapes (more than the staging ring's eight slots, and
no-alloc calls that refill the static scratch array a captured no-alloc call
uses), clears the graph's outputs with eager fills (no memset inside the
graph), and checks every replay against the eager result of the same call, bit
for bit: the step (decodes and extends, bf16 and fp8 pools), the extend with
split-K partials, the no-alloc extend, the decode, and the page write with
swaps out and in (pinned host pools)."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import paper_2606_16824_amd as cwlib
from gpu_util import to_gpu

pytestmark = pytest.mark.gpu

CASES = {
    "step_bf16": ([300, 1000, 17, 500], [1, 70, 1, 129], "bf16"),
    "step_fp8": ([300, 1000, 17, 500], [1, 70, 1, 129], "fp8"),
    "extend": ([700, 90, 3000], [150, 64, 300], "bf16"),
    "noalloc": ([700, 90, 3000], [150, 64, 300], "bf16"),
    "decode": ([300, 1000, 2000, 5], [1, 1, 1, 1], "bf16"),
}


def _inputs(lp, ls, dt, seed):
    spec = cw.custom_spec(lp, ls, num_kv_heads=2, gqa_group=4, head_dim=128, page_size=16,
                          kv_dtype=dt, seed=seed)
    return spec, to_gpu(cw.materialize(spec))


def _call(name, spec, dw, out, lse, ws):
    s = spec
    args = (dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table)
    kw = dict(k_scale=dw.k_scale, v_scale=dw.v_scale, out=out, lse=lse)
    if name.startswith("step"):
        cwlib.step_attention(*args, s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale,
                             workspace=ws, **kw)
    elif name == "extend":
        cwlib.extend_attention(*args, s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale,
                               workspace=ws, **kw)
    elif name == "noalloc":
        cwlib.extend_attention_noalloc(*args, s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale, **kw)
    else:
        cwlib.decode_attention(*args, s.prefix_lens, s.gqa_group, s.softmax_scale, workspace=ws, **kw)


def _churn(n=10):
    """Eager calls of other shapes: each takes a staging slot, and the no-alloc
    ones overwrite the static scratch array."""
    spec, dw = _inputs([333, 50, 1200], [77, 1, 200], "bf16", 4711)
    out = torch.empty_like(dw.q)
    for i in range(n):
        cwlib.step_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                             spec.prefix_lens, spec.suffix_lens, spec.gqa_group, spec.softmax_scale, out=out)
        if i % 3 == 0:
            cwlib.extend_attention_noalloc(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                                           spec.prefix_lens, spec.suffix_lens, spec.gqa_group,
                                           spec.softmax_scale, out=out)
    torch.cuda.synchronize()


def _bits(t):
    return t.detach().cpu().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


@pytest.mark.parametrize("name", list(CASES))
def test_captured_call_replays_bit_identical(name):
    lp, ls, dt = CASES[name]
    print(f"\n[case] graph replay {name}: Lp={lp} Ls={ls} {dt}", flush=True)
    cwlib.init()
    spec, dw = _inputs(lp, ls, dt, 9100 + len(name))
    hq = dw.q.shape[1]
    nb = max(cwlib.step_workspace_bytes(spec.prefix_lens, spec.suffix_lens, 2, 4, 128, 16, dt),
             cwlib.extend_workspace_bytes(spec.prefix_lens, spec.suffix_lens, 2, 4, 128, 16),
             cwlib.decode_workspace_bytes(spec.prefix_lens, 2, 4, 128, 16, dt))
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    ref_out, ref_lse = torch.empty_like(dw.q), torch.empty(dw.q.shape[0], hq, device="cuda")
    _call(name, spec, dw, ref_out, ref_lse, ws)
    torch.cuda.synchronize()
    want_o, want_l = _bits(ref_out), _bits(ref_lse)
    assert np.isfinite(ref_lse.cpu().numpy()).all()

    out, lse = torch.empty_like(dw.q), torch.empty_like(ref_lse)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        _call(name, spec, dw, out, lse, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _call(name, spec, dw, out, lse, ws)
    torch.cuda.synchronize()
    for rep in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        _churn()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(_bits(out), want_o), (name, rep)
        assert np.array_equal(_bits(lse), want_l), (name, rep)
    print(f"[graph] {name}: 3 replays bit-identical to the eager call", flush=True)


def _capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("dt", ["bf16", "fp8"])
def test_captured_page_write_and_swaps_replay(dt):
    """cw_kv_write_pages into the pools, then cw_kv_swap_out of the written pages
    to a pinned host pool and cw_kv_swap_in of them to other pages, captured as
    one graph: every replay (after eager calls of other shapes, with the pools and
    the host pool cleared eagerly) leaves the same bytes as the eager calls."""
    print(f"\n[case] graph replay: page write and swaps, {dt}", flush=True)
    cwlib.init()
    spec, dw = _inputs([40, 0, 100], [30, 20, 70], dt, 9200)
    used = np.unique(dw.block_table.cpu().numpy()[:, :8])
    used = used[used < spec.num_pages]
    free = np.setdiff1d(np.arange(spec.num_pages), dw.block_table.cpu().numpy())[:len(used)]
    assert len(free) == len(used)
    host = np.arange(len(used), dtype=np.int32)
    kh = torch.empty((len(used),) + tuple(dw.k_pool.shape[1:]), dtype=dw.k_pool.dtype).pin_memory()
    vh = torch.empty_like(kh).pin_memory()
    ksh = vsh = None
    if dt == "fp8":
        ksh = torch.empty(len(used), dw.k_scale.shape[1], dtype=torch.float32).pin_memory()
        vsh = torch.empty_like(ksh).pin_memory()
    k0, v0 = dw.k_pool.clone(), dw.v_pool.clone()

    def work():
        cwlib.kv_write_pages(dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table, spec.prefix_lens,
                             spec.suffix_lens, k_scale=dw.k_scale, v_scale=dw.v_scale)
        cwlib.kv_swap_out(dw.k_pool, dw.v_pool, kh, vh, used, host, k_scale=dw.k_scale, v_scale=dw.v_scale,
                          k_scale_host=ksh, v_scale_host=vsh)
        cwlib.kv_swap_in(kh, vh, dw.k_pool, dw.v_pool, host, free, k_scale_host=ksh, v_scale_host=vsh,
                         k_scale=dw.k_scale, v_scale=dw.v_scale)

    raw = lambda t: t.detach().cpu().view(torch.uint8).numpy().copy()
    work()
    torch.cuda.synchronize()
    want = [raw(t) for t in (dw.k_pool, dw.v_pool, kh, vh)]
    g = _capture(work)
    for rep in range(3):
        dw.k_pool.copy_(k0)
        dw.v_pool.copy_(v0)
        kh.zero_()
        vh.zero_()
        _churn()
        g.replay()
        torch.cuda.synchronize()
        got = [raw(t) for t in (dw.k_pool, dw.v_pool, kh, vh)]
        for a, b, what in zip(got, want, ("k pool", "v pool", "k host", "v host")):
            assert np.array_equal(a, b), (dt, rep, what)
    print(f"[graph] page write and swaps {dt}: 3 replays byte-identical", flush=True)
