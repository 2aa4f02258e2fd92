"""Benchmark: prefix-cached paged extend attention on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload turn]

One step = one pass of the hot path over one batch: cw_kv_write_pages (the
new K/V into their pages) then cw_extend_attention (the new tokens over the
cached prefix and themselves).  The default workload is the single agent turn
(prefix 16384, suffix 1024, 32 query / 8 kv heads, head_dim 128, page 16,
bf16, pages randomly permuted in a 4096-page pool).  Inputs are synthetic,
seeded, and resident in HBM before timing starts.

Prints one JSON line: value = algorithmic extend TFLOP/s of the whole step
(4 * D * Hq * sum(Ls*Lp + Ls(Ls+1)/2) FLOPs per step), plus the roofline of
the extend kernel timed alone with HIP events, and the CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 2.4 GHz x 4096 FLOP/clk (dense bf16 MFMA)
PEAK_HBM_GBS = 8000.0

WORKLOAD_DESC = {
    "tiny": "tiny extend: prefix 256, suffix 64, 4q/1kv, D=64, P=16",
    "turn": "single agent turn: prefix 16384, suffix 1024, 32q/8kv (GQA 4), D=128, P=16, bf16, 4096-page permuted pool",
    "batch16": "16 agent turns sharing an 8192-token prefix, prefix lognormal(20k) 4k-64k, suffix U[200,4000], 32q/8kv, D=128, P=16, bf16",
    "long": "long-session extend: prefix 131072, suffix 8192, 64q/8kv (GQA 8), D=128, P=64, bf16",
    "mixed": "mixed step: 48 decodes + 16 extends, 32q/8kv, D=128, P=16, fp8-e4m3fn pool",
    "decode": "decode: the 48 decodes of the mixed step (prefix U[2k,32k]), 32q/8kv, D=128, P=16, fp8-e4m3fn pool",
    "decode_bf16": "decode: the 48 decodes of the mixed step, 32q/8kv, D=128, P=16, bf16 pool",
    "decode_long": "decode: 1 sequence, prefix 131072, 64q/8kv (GQA 8), D=128, P=64, bf16 pool",
    "chunked": "chunked prefill step: 32 chunks of U[128,512] tokens on prefixes U[8k,32k] + 32 decodes (prefix U[2k,32k]), 32q/8kv, D=128, P=16, bf16",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="turn", choices=list(WORKLOAD_DESC))
    ap.add_argument("--decode-steps", type=int, default=100,
                    help="steps of the decode measurement added to an extend run, after as many "
                         "warm-up steps as the main run (0 disables)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample (0 disables)")
    ap.add_argument("--no-policy", dest="policy", action="store_false",
                    help="skip the host KV-block policy comparison added to an extend run")
    ap.add_argument("--no-other-workloads", dest="others", action="store_false",
                    help="skip the other named workloads (batch16, long, mixed, decode_bf16, decode_long)")
    ap.add_argument("--other-steps", type=int, default=20,
                    help="timed steps per other workload (after 5 warm-up steps)")
    ap.add_argument("--no-swap", dest="swap", action="store_false",
                    help="skip the page swap measurement added to an extend run")
    ap.add_argument("--extend-kernel", type=int, default=0, choices=[0, 1, 2],
                    help="extend kernel for bf16 pools: 0 or 1 eight waves of 32 rows (default), "
                         "2 four waves of 64 rows")
    ap.add_argument("--deal-rounds", type=int, default=1, choices=[0, 1],
                    help="1 (default): a (sequence, kv head) that fills whole GPU rounds is dealt "
                         "across all XCDs round by round; 0: it stays on one XCD")
    ap.add_argument("--plan-direct", type=int, default=0, choices=[0, 1],
                    help="1: kernels read the plan from the pinned staging slot; 0 (default): "
                         "it is copied to the workspace first")
    ap.add_argument("--compact-decode", type=int, default=1, choices=[0, 1],
                    help="1 (default): decode plans are uploaded in compact form and rebuilt on "
                         "the device; 0: their work items are uploaded as they are")
    ap.add_argument("--arg-plans", type=int, default=1, choices=[0, 1],
                    help="1 (default): extend plans of up to 16 KB travel in the kernel arguments; "
                         "0: they are uploaded by a copy kernel")
    ap.add_argument("--suffix-weight", type=int, default=None,
                    help="split-K cost of a key tile past the cached prefix, percent of a prefix tile "
                         "(default: the library's)")
    ap.add_argument("--separate-calls", action="store_true",
                    help="time a step as cw_kv_write_pages + cw_extend_attention (or "
                         "cw_decode_attention) instead of cw_step_attention")
    ap.add_argument("--cold-steps", type=int, default=20,
                    help="extra steps, each after reading 1 GiB of another buffer so that the "
                         "memory-side cache holds none of its inputs (kernel time reported "
                         "separately; 0 disables)")
    ap.add_argument("--no-ceilings", dest="ceilings", action="store_false",
                    help="skip the measured MFMA and HBM ceilings")
    ap.add_argument("--power-seconds", type=float, default=3.0,
                    help="seconds of back-to-back steps (and of each MFMA loop) during which "
                         "amd-smi samples socket power and GFX clocks; 0 disables")
    ap.add_argument("--ceilings-only", action="store_true",
                    help="only measure the MFMA and HBM ceilings, print them as one JSON line "
                         "and exit")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (for "
                         "scaling the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


def calibrate_copy(mib: int):
    """A plain copy of known size, for reading HBM byte counters against."""
    import torch
    n = mib * (1 << 20)
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "copy", "bytes_read": n, "bytes_written": n, "launches": 3}))


EXTEND_KERNEL = 0  # --extend-kernel

KERNEL_SOURCES = {  # dominant kernel per pool dtype: (kernel, source, profile summary)
    "bf16": ("extend_lds_kernel", "paper_2606_16824_amd/csrc/kernels/extend_lds.hip", "extend_lds_{wl}.md"),
    "fp8": ("extend_lds_kernel", "paper_2606_16824_amd/csrc/kernels/extend_lds.hip", "extend_lds_{wl}.md"),
    "decode": ("decode_kernel", "paper_2606_16824_amd/csrc/kernels/decode.hip", "decode_kernel_{wl}.md"),
}


def measured_traffic(kind: str, workload: str):
    """HBM bytes per launch from the committed counter summary, or None when the
    summary is missing or was taken on a different version of the kernel source.
    `kind` is the pool dtype of an extend workload, or "decode"."""
    import hashlib
    import re
    kernel, src, prof = KERNEL_SOURCES[kind]
    path = os.path.join(ROOT, "profiles", prof.format(wl=workload))
    try:
        text = open(path).read()
        sha = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
    except OSError:
        return None
    m = re.search(r"traffic_bytes_per_launch=(\d+) kernel_source_sha256=([0-9a-f]+)", text)
    if not m or m.group(2) != sha:
        return None
    return int(m.group(1))


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or the platform's processor string."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def blas_vendor() -> str:
    """The BLAS numpy calls (runtime library as threadpoolctl sees it, and numpy's
    build configuration)."""
    parts = []
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                parts.append(f"{i.get('internal_api')} {i.get('version')} ({os.path.basename(i.get('filepath', ''))})")
    except Exception:
        pass
    try:
        cfg = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        parts.append(f"numpy built with {cfg.get('name')} {cfg.get('version')}")
    except Exception:
        pass
    return "; ".join(parts) or "unknown"


def cpu_baseline(w, target_s: float):
    """The oracle's blocked implementation in float32 (NumPy sgemm for S and P V, per
    (sequence, kv head) blocks of 64 tokens x G heads) on the first suffix tokens of
    sequence 0, as many as fit in about `target_s` seconds (the whole suffix when it
    is faster), with BLAS threads = the CPUs this process may run on."""
    import oracle
    from tests.conftest import paged_inputs

    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores, user_api="blas")
    except Exception:
        limiter = None
    inp = paged_inputs(w)
    s = w.spec
    lp, ls = int(s.prefix_lens[0]), int(s.suffix_lens[0])

    def run(n_tok):
        sub = oracle.PagedInputs(inp.q[:n_tok], inp.k_new[:n_tok], inp.v_new[:n_tok], inp.k_pool,
                                 inp.v_pool, inp.block_table[:1], np.array([lp]), np.array([n_tok]),
                                 inp.gqa_group, inp.softmax_scale, inp.kv_dtype, inp.k_scale,
                                 inp.v_scale)
        t0 = time.perf_counter()
        oracle.extend_attention_blocked(sub, block_tokens=64, dtype=np.float32)
        return time.perf_counter() - t0

    try:
        # the page gather is a fixed cost, so grow the sample by doubling until it
        # takes at least half the target (or covers the whole suffix)
        n = min(64, ls)
        dt = run(n)
        while dt < 0.5 * target_s and n < ls:
            n = min(ls, 2 * n)
            dt = run(n)
        # the whole suffix fits well inside the target: repeat it (up to the
        # target's half, at most 20 runs) and take the median run
        times = [dt]
        while n == ls and sum(times) < 0.5 * target_s and len(times) < 20:
            times.append(run(n))
        dt = float(np.median(times))
    finally:
        if limiter is not None:
            limiter.unregister()
    pairs = n * lp + n * (n + 1) // 2
    flops = 4.0 * s.head_dim * s.num_q_heads * pairs
    runs = f", median of {len(times)} runs" if len(times) > 1 else ""
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"first {n} of {ls} suffix tokens of sequence 0, all {s.num_q_heads} query heads "
                      f"(float32 blocked oracle: page gather, sgemm, mask, softmax, P V), {dt:.1f} s{runs}",
            "tok_s": n / dt, "cpu_model": cpu_model(), "blas": blas_vendor(),
            "wall_s": round(sum(times), 3), "runs": len(times)}


def _smi_json(args):
    """JSON from a ROCm SMI tool, or None when it is missing or fails."""
    import shutil
    import subprocess
    tool = shutil.which(args[0])
    if tool is None:
        return None
    try:
        r = subprocess.run([tool] + args[1:], capture_output=True, text=True, timeout=20)
        return json.loads(r.stdout)
    except (OSError, ValueError, subprocess.SubprocessError):
        return None


def _find(d, pred, out):
    """Collects (key, value) pairs anywhere in nested dicts / lists for which pred(key) holds."""
    if isinstance(d, dict):
        for k, v in d.items():
            if pred(str(k)):
                out.append((str(k), v))
            _find(v, pred, out)
    elif isinstance(d, list):
        for v in d:
            _find(v, pred, out)
    return out


def _num(v):
    if isinstance(v, dict):
        v = v.get("value")
    try:
        return float(v)
    except (TypeError, ValueError):
        return None


def parse_smi_metric(d):
    """(socket power W, median GFX clock MHz over the XCDs) from the JSON of
    `amd-smi metric -p -c --json`; either is None when the report lacks it."""
    pw = [_num(v) for _, v in _find(d, lambda k: k == "socket_power", [])]
    clk = [_num(v.get("clk")) for k, v in _find(d, lambda k: k.lower().startswith("gfx_"), [])
           if isinstance(v, dict)]
    clk = [c for c in clk if c]
    return (pw[0] if pw and pw[0] else None), (float(np.median(clk)) if clk else None)


def power_cap_w():
    """The board's power cap (W) as rocm-smi reports it, or None."""
    d = _smi_json(["rocm-smi", "--showmaxpower", "--json"])
    vals = [_num(v) for _, v in _find(d, lambda k: "Max Graphics Package Power" in k, [])]
    vals = [v for v in vals if v]
    return vals[0] if vals else None


def sample_power(enqueue, seconds: float, settle: float = 0.5):
    """Keeps the GPU busy with `enqueue()` (one batch of work per call, two batches in
    flight) for `seconds` while amd-smi samples socket power and the XCDs' GFX clocks
    of GPU 0 (the only GPU of the box); samples from the first `settle` seconds are
    dropped.  Returns medians over the samples, or None without amd-smi."""
    import threading
    import torch

    samples = []
    stop = threading.Event()
    t0 = time.perf_counter()

    def poll():
        while not stop.is_set():
            d = _smi_json(["amd-smi", "metric", "-g", "0", "-p", "-c", "--json"])
            if d is None:
                return
            if time.perf_counter() - t0 < settle:
                continue
            pw, clk = parse_smi_metric(d)
            if pw:
                samples.append((pw, clk))

    th = threading.Thread(target=poll, daemon=True)
    th.start()
    prev = None
    while time.perf_counter() - t0 < seconds:
        enqueue()
        ev = torch.cuda.Event()
        ev.record()
        if prev is not None:
            prev.synchronize()
        prev = ev
    torch.cuda.synchronize()
    stop.set()
    th.join(timeout=30)
    if not samples:
        return None
    pw = [a for a, _ in samples]
    clk = [b for _, b in samples if b]
    return {"socket_W_median": round(float(np.median(pw)), 1),
            "socket_W_max": round(float(np.max(pw)), 1),
            "gfx_MHz_median": round(float(np.median(clk)), 0) if clk else None,
            "samples": len(samples)}


def run_workload(name: str, steps: int, warmup: int, separate: bool = False, cold_steps: int = 0,
                 power_s: float = 0.0, one_launch: bool = False):
    """Times `steps` hot-path steps (page write + attention) of a named workload: one
    cw_step_attention per step (decodes on the decode kernel, extends on the extend
    kernel, the page write fused into the extend launch, or into the decode launch
    when there are no extends); with `separate`, cw_kv_write_pages followed by
    cw_extend_attention or cw_decode_attention; with `one_launch`, one
    cw_write_extend_attention over every sequence (decodes as one-token extends:
    the page write and all attention in one extend launch, plus the split-K merge)."""
    import torch
    import cw_workloads as cw
    import paper_2606_16824_amd as cwlib

    dev = torch.device("cuda:0")
    w = cw.make(name)
    s = w.spec
    decode = name.startswith("decode")
    print(f"[bench] workload {name}: {s.num_seqs} seqs, {s.total_new_tokens} new tokens, "
          f"{s.flops() / 1e12:.3f} TFLOP", file=sys.stderr, flush=True)
    mv = lambda t: None if t is None else t.to(dev).contiguous()
    q, kn, vn, kp, vp = mv(w.q), mv(w.k_new), mv(w.v_new), mv(w.k_pool), mv(w.v_pool)
    ks, vs, bt = mv(w.k_scale), mv(w.v_scale), mv(w.block_table)
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[0], q.shape[1], device=dev, dtype=torch.float32)
    if decode and separate:
        nb = cwlib.decode_workspace_bytes(s.prefix_lens, s.num_kv_heads, s.gqa_group, s.head_dim,
                                          s.page_size, s.kv_dtype)
    elif separate or one_launch:
        nb = cwlib.extend_workspace_bytes(s.prefix_lens, s.suffix_lens, s.num_kv_heads,
                                          s.gqa_group, s.head_dim, s.page_size)
    else:
        nb = cwlib.step_workspace_bytes(s.prefix_lens, s.suffix_lens, s.num_kv_heads,
                                        s.gqa_group, s.head_dim, s.page_size, s.kv_dtype)
    ws_att = torch.empty(nb, dtype=torch.uint8, device=dev)
    ws_wr = torch.empty(cwlib.write_pages_workspace_bytes(s.num_seqs), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        if one_launch:
            cwlib.write_extend_attention(q, kn, vn, kp, vp, bt, s.prefix_lens, s.suffix_lens,
                                         s.gqa_group, s.softmax_scale, k_scale=ks, v_scale=vs,
                                         out=out, lse=lse, workspace=ws_att)
            return
        if not separate:
            cwlib.step_attention(q, kn, vn, kp, vp, bt, s.prefix_lens, s.suffix_lens,
                                 s.gqa_group, s.softmax_scale, k_scale=ks, v_scale=vs,
                                 out=out, lse=lse, workspace=ws_att)
            return
        cwlib.kv_write_pages(kn, vn, kp, vp, bt, s.prefix_lens, s.suffix_lens, k_scale=ks,
                             v_scale=vs, workspace=ws_wr)
        if decode:
            cwlib.decode_attention(q, kn, vn, kp, vp, bt, s.prefix_lens, s.gqa_group,
                                   s.softmax_scale, k_scale=ks, v_scale=vs, out=out, lse=lse,
                                   workspace=ws_att)
        else:
            cwlib.extend_attention(q, kn, vn, kp, vp, bt, s.prefix_lens, s.suffix_lens,
                                   s.gqa_group, s.softmax_scale, k_scale=ks, v_scale=vs, out=out,
                                   lse=lse, workspace=ws_att)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    lib = cwlib.library()
    n_ev = max(steps, cold_steps)
    k_starts = [torch.cuda.Event(enable_timing=True) for _ in range(n_ev)]
    k_stops = [torch.cuda.Event(enable_timing=True) for _ in range(n_ev)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    for e in k_starts + k_stops:  # torch creates the HIP event on first record
        e.record(stream)
    torch.cuda.synchronize()
    # timed region: exactly `steps` steps, nothing recorded inside them
    t_start.record(stream)
    for i in range(steps):
        step()
    t_stop.record(stream)
    torch.cuda.synchronize()
    ms = t_start.elapsed_time(t_stop) / steps
    # then `steps` more steps in which the library records events around the main
    # attention kernel (the events themselves add a few us to a step)
    for i in range(steps):
        lib.cw_set_timing_events(k_starts[i].cuda_event, k_stops[i].cuda_event)
        step()
    torch.cuda.synchronize()
    lib.cw_set_timing_events(None, None)
    kern = np.array([a.elapsed_time(b) for a, b in zip(k_starts, k_stops)])
    # host cost of issuing one step (validation, planning, plan upload, launches)
    # with an idle queue, so that nothing waits on the GPU
    host = []
    for _ in range(20):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        step()
        host.append(time.perf_counter() - t0)
    torch.cuda.synchronize()
    kernel = "decode_kernel" if decode else KERNEL_SOURCES[s.kv_dtype][0]
    if not decode and s.kv_dtype == "bf16" and EXTEND_KERNEL == 2:
        kernel = "extend_w64_kernel"
    res = {"spec": s, "workload": w, "ms": ms, "kern_ms": float(kern.mean()),
           "kern_ms_median": float(np.median(kern)), "kern_ms_min": float(kern.min()),
           "host_us": float(np.median(host)) * 1e6, "kernel": kernel}
    if cold_steps > 0:
        # outside the kernel's events: before each step, 1 GiB of another buffer is
        # read so that the 256 MB memory-side cache (and every L2) holds none of the
        # step's inputs.  Reads leave clean lines: a flush by writing would leave
        # dirty lines whose write-back then competes with the measured kernel.
        flush = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        for i in range(cold_steps):
            flush.max()
            lib.cw_set_timing_events(k_starts[i].cuda_event, k_stops[i].cuda_event)
            step()
        torch.cuda.synchronize()
        lib.cw_set_timing_events(None, None)
        cold = np.array([k_starts[i].elapsed_time(k_stops[i]) for i in range(cold_steps)])
        res["cold_kern_ms_median"] = float(np.median(cold))
        res["cold_kern_ms_min"] = float(cold.min())
        del flush
    if power_s > 0:
        def batch():
            for _ in range(20):
                step()
        res["power"] = sample_power(batch, power_s)
    return res


OTHER_WORKLOADS = ("batch16", "long", "mixed", "chunked", "decode_bf16", "decode_long")


def run_others(names, steps: int, warmup: int = 5):
    """The other named workloads, each timed like the main one (one step = one
    cw_step_attention on inputs resident in HBM; kernel time by HIP events in a
    second pass), reported per workload."""
    import gc
    import torch
    import cw_workloads as cw

    out = {}
    for name in names:
        res = run_workload(name, steps, warmup)
        s, ms, kern = res["spec"], res["ms"], res["kern_ms"]
        if name.startswith("decode"):
            nbytes = cw.decode_bytes(s)
            out[name] = {"workload": WORKLOAD_DESC[name], "ms_per_step": round(ms, 5),
                         "kernel": res["kernel"], "kernel_ms": round(kern, 5),
                         "GB_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                         "kernel_GB_s": round(nbytes / (kern * 1e-3) / 1e9, 1),
                         "frac_hbm_peak": round(nbytes / (kern * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                         "algorithmic_bytes": nbytes, "traffic": measured_traffic("decode", name)}
        else:
            flops = s.flops()
            out[name] = {"workload": WORKLOAD_DESC[name], "ms_per_step": round(ms, 5),
                         "kernel": res["kernel"], "kernel_ms": round(kern, 5),
                         "TFLOP_s": round(flops / (ms * 1e-3) / 1e12, 2),
                         "kernel_TFLOP_s": round(flops / (kern * 1e-3) / 1e12, 2),
                         "frac_bf16_peak": round(flops / (kern * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                         "new_tok_s": round(s.total_new_tokens / (ms * 1e-3), 1),
                         "tflop_per_step": round(flops / 1e12, 5), "seed": s.seed,
                         "traffic": measured_traffic(s.kv_dtype, name) if EXTEND_KERNEL != 2 else None}
        out[name]["steps"] = steps
        if name == "chunked":
            # the same step as one extend launch (decodes as one-token extends)
            one = run_workload(name, steps, warmup, one_launch=True)
            out[name]["one_launch"] = {
                "calls": "cw_write_extend_attention (one extend launch, decodes as one-token extends)",
                "ms_per_step": round(one["ms"], 5), "kernel_ms": round(one["kern_ms"], 5)}
            del one
        print(f"[bench] {name}: step {ms:.4f} ms, kernel {kern:.4f} ms", file=sys.stderr, flush=True)
        del res
        gc.collect()
        torch.cuda.empty_cache()
    return out


def measure_ceilings(reps: int = 5, power_s: float = 0.0):
    """What the chip sustains on each roofline's unit of work with nothing else in
    the way: a matrix-core loop (bf16 MFMA, no memory traffic) with operand bits like
    real data (the ceiling attention is priced against) and with a few repeated bit
    patterns (less power per MFMA, so a higher clock), a streaming read and a streaming
    copy of 4 GiB (each launch median over `reps`).  For context also the vendor
    library's bf16 GEMM (torch.matmul, 8192^3, N(0,1) operands)."""
    import torch
    import paper_2606_16824_amd as cwlib

    def med(fn):
        fn()
        torch.cuda.synchronize()
        t = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            t.append(a.elapsed_time(b))
        return float(np.median(t))

    wgs, iters = 512, 40000  # two workgroups per CU, all resident at once: no tail
    sink = torch.empty(wgs * 8, dtype=torch.float32, device="cuda")
    flops = float(wgs) * 8 * iters * 131072
    mfma_ms = med(lambda: cwlib.ceiling_mfma_bf16(wgs, iters, sink, random=True))
    mfma_low_ms = med(lambda: cwlib.ceiling_mfma_bf16(wgs, iters, sink, random=False))
    n = 8192
    g = torch.Generator(device="cuda").manual_seed(7)
    a = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16)
    b = torch.randn(n, n, device="cuda", generator=g).to(torch.bfloat16)
    gemm_ms = med(lambda: torch.matmul(a, b))
    del a, b
    buf = torch.empty(4 << 30, dtype=torch.uint8, device="cuda").fill_(3)
    dst = torch.empty_like(buf)
    rsink = torch.empty(16384, dtype=torch.int32, device="cuda")
    read_ms = med(lambda: cwlib.ceiling_stream_read(buf, rsink))
    copy_ms = med(lambda: cwlib.ceiling_stream_copy(buf, dst))
    nb = buf.numel()
    del buf, dst
    power = None
    if power_s > 0:
        loop = lambda rnd: lambda: [cwlib.ceiling_mfma_bf16(wgs, iters, sink, random=rnd) for _ in range(4)]
        power = {"mfma_loop_random": sample_power(loop(True), power_s),
                 "mfma_loop_low_entropy": sample_power(loop(False), power_s)}
    return {"power": power,
            "mfma_bf16_TFLOP_s": round(flops / (mfma_ms * 1e-3) / 1e12, 1),
            "mfma_bf16_low_entropy_TFLOP_s": round(flops / (mfma_low_ms * 1e-3) / 1e12, 1),
            "vendor_gemm_bf16_TFLOP_s": round(2.0 * n ** 3 / (gemm_ms * 1e-3) / 1e12, 1),
            "hbm_read_GB_s": round(nb / (read_ms * 1e-3) / 1e9, 1),
            "hbm_copy_GB_s": round(2 * nb / (copy_ms * 1e-3) / 1e9, 1),
            "kernels": "mfma_loop_kernel (512 workgroups of 8 waves, 4 independent 32x32x16 bf16 "
                       "chains per wave; random operand bits, and low-entropy patterns), torch.matmul "
                       "bf16 8192^3 on N(0,1) data, stream_read_kernel / stream_copy_kernel (4 GiB, "
                       "16 B nontemporal loads, 4 in flight per lane, 16384 workgroups)"}


def run_swap(reps: int = 10):
    """Swap-out of the turn's cached prefix (1024 pages x 8 kv heads, K and V) to a
    pinned host block pool and swap-in to other pool pages, against a plain
    contiguous copy of the same bytes in each direction (the host link's ceiling)."""
    import torch
    import cw_workloads as cw
    import paper_2606_16824_amd as cwlib

    spec = cw.spec_for("turn")
    w = cw.materialize(spec)
    n = int(spec.prefix_lens[0]) // spec.page_size
    pages = w.block_table[0, :n].numpy().astype(np.int32)
    free = np.setdiff1d(np.arange(spec.num_pages), w.block_table[0].numpy())[:n].astype(np.int32)
    dk, dv = w.k_pool.cuda(), w.v_pool.cuda()
    hk = torch.empty((n,) + tuple(dk.shape[1:]), dtype=dk.dtype).pin_memory()
    hv = torch.empty_like(hk).pin_memory()
    host = np.arange(n, dtype=np.int32)
    nbytes = 2 * hk.numel() * hk.element_size()
    ws = torch.empty(cwlib.swap_workspace_bytes(n), dtype=torch.uint8, device="cuda")
    flat_d = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    flat_h = torch.empty(nbytes, dtype=torch.uint8).pin_memory()

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    out_ms = timed(lambda: cwlib.kv_swap_out(dk, dv, hk, hv, pages, host, workspace=ws))
    in_ms = timed(lambda: cwlib.kv_swap_in(hk, hv, dk, dv, host, free, workspace=ws))
    d2h_ms = timed(lambda: flat_h.copy_(flat_d, non_blocking=True))
    h2d_ms = timed(lambda: flat_d.copy_(flat_h, non_blocking=True))
    gbs = lambda ms: round(nbytes / (ms * 1e-3) / 1e9, 1)
    return {"workload": f"turn prefix: {n} pages x {spec.num_kv_heads} kv heads, K and V "
                        f"({nbytes / 2**20:.0f} MiB) to a pinned host block pool and back",
            "bound": "host link", "out_GB_s": gbs(out_ms), "in_GB_s": gbs(in_ms),
            "copy_d2h_GB_s": gbs(d2h_ms), "copy_h2d_GB_s": gbs(h2d_ms),
            "frac_out": round(d2h_ms / out_ms, 4), "frac_in": round(h2d_ms / in_ms, 4),
            "kernel": "swap_kernel"}


def main():
    args = parse()
    if args.calibrate_copy_mib:
        calibrate_copy(args.calibrate_copy_mib)
        return
    if args.ceilings_only:
        c = measure_ceilings(power_s=args.power_seconds)
        c["power_cap_W"] = power_cap_w()
        print(json.dumps({"ceilings": c}), flush=True)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    import torch
    import cw_workloads as cw
    import paper_2606_16824_amd as cwlib

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    global EXTEND_KERNEL
    EXTEND_KERNEL = args.extend_kernel
    cwlib.set_tuning(cwlib._lib.CW_TUNE_EXTEND_KERNEL, args.extend_kernel)
    cwlib.set_tuning(cwlib._lib.CW_TUNE_DEAL_ROUNDS, args.deal_rounds)
    cwlib.set_tuning(cwlib._lib.CW_TUNE_PLAN_DIRECT, args.plan_direct)
    cwlib.set_tuning(cwlib._lib.CW_TUNE_COMPACT_DECODE, args.compact_decode)
    cwlib.set_tuning(cwlib._lib.CW_TUNE_ARG_PLANS, args.arg_plans)
    if args.suffix_weight is not None:
        cwlib.set_tuning(cwlib._lib.CW_TUNE_SUFFIX_WEIGHT, args.suffix_weight)
    res = run_workload(args.workload, args.steps, args.warmup, separate=args.separate_calls,
                       cold_steps=args.cold_steps, power_s=args.power_seconds)
    ceil = measure_ceilings(power_s=args.power_seconds) if args.ceilings else None
    ceil_power = ceil.pop("power") if ceil is not None else None
    s, w = res["spec"], res["workload"]
    ms, kern_ms = res["ms"], res["kern_ms"]
    decode = s.suffix_lens.max() == 1 and args.workload.startswith("decode")
    if decode:
        nbytes = cw.decode_bytes(s)
        value = nbytes / (ms * 1e-3) / 1e9
        achieved = nbytes / (kern_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": measured_traffic("decode", args.workload),
                "kernel": res["kernel"], "kernel_ms": round(kern_ms, 5)}
        rate = lambda t: nbytes / (t * 1e-3) / 1e9
        ceil_key = "hbm_read_GB_s"
        unit = "GB/s"
    else:
        flops = s.flops()
        value = flops / (ms * 1e-3) / 1e12
        achieved = flops / (kern_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic(s.kv_dtype, args.workload) if EXTEND_KERNEL != 2 else None,
                "kernel": res["kernel"], "kernel_ms": round(kern_ms, 5)}
        rate = lambda t: flops / (t * 1e-3) / 1e12
        ceil_key = "mfma_bf16_TFLOP_s"
        unit = "TFLOP/s"
    roof["kernel_ms_median"] = round(res["kern_ms_median"], 5)
    roof["kernel_ms_min"] = round(res["kern_ms_min"], 5)
    if "cold_kern_ms_median" in res:
        roof["cold"] = {"steps": args.cold_steps, "kernel_ms_median": round(res["cold_kern_ms_median"], 5),
                        "kernel_ms_min": round(res["cold_kern_ms_min"], 5),
                        "achieved": round(rate(res["cold_kern_ms_median"]), 2),
                        "note": "1 GiB of another buffer read before each step, outside the kernel's events"}
    if ceil is not None:
        roof["measured_ceiling"] = ceil[ceil_key]
        roof["frac_of_measured_ceiling"] = round(roof["achieved"] / ceil[ceil_key], 4)
    print(f"[bench] step {ms:.4f} ms, main kernel {kern_ms:.4f} ms, {achieved:.1f} {unit} kernel",
          file=sys.stderr, flush=True)

    result = {
        "metric": "extend-attn TFLOP/s (% bf16 MFMA peak) + new tok/s; decode HBM GB/s % peak",
        "value": round(value, 2),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if s.kv_dtype == "bf16" else "bf16+fp8kv",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_DESC[args.workload], "new_tokens": s.total_new_tokens,
                   "calls": (("cw_kv_write_pages + cw_decode_attention" if decode else
                              "cw_kv_write_pages + cw_extend_attention") if args.separate_calls
                             else "cw_step_attention"),
                   "tflop_per_step": round(s.flops() / 1e12, 5), "seed": s.seed},
        "new_tok_s": round(s.total_new_tokens / (ms * 1e-3), 1),
        "host_us_per_step": round(res["host_us"], 1),
        "roofline": roof,
    }
    if ceil is not None:
        result["ceilings"] = ceil
    if args.power_seconds > 0:
        power = {"cap_W": power_cap_w(), args.workload: res.get("power")}
        if ceil_power is not None:
            power.update(ceil_power)
        power["source"] = ("amd-smi metric -p -c: socket power and the median of the XCDs' GFX "
                           "clocks, sampled while the work runs back to back; cap from rocm-smi")
        result["power"] = power
    if not decode and args.decode_steps > 0:
        # the decode side of the metric: the mixed step's 48 decodes, fp8 pool
        d = run_workload("decode", args.decode_steps, args.warmup, cold_steps=args.cold_steps,
                         power_s=args.power_seconds)
        if args.power_seconds > 0:
            result["power"]["decode"] = d.get("power")
        nbytes = cw.decode_bytes(d["spec"])
        result["decode"] = {
            "workload": WORKLOAD_DESC["decode"], "ms_per_step": round(d["ms"], 5),
            "GB_s": round(nbytes / (d["ms"] * 1e-3) / 1e9, 1),
            "kernel_GB_s": round(nbytes / (d["kern_ms"] * 1e-3) / 1e9, 1),
            "frac_hbm_peak": round(nbytes / (d["kern_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "algorithmic_bytes": nbytes, "traffic": measured_traffic("decode", "decode"),
            "kernel": d["kernel"], "kernel_ms": round(d["kern_ms"], 5),
            "kernel_ms_median": round(d["kern_ms_median"], 5),
            "host_us_per_step": round(d["host_us"], 1)}
        if "cold_kern_ms_median" in d:
            result["decode"]["cold_kernel_GB_s"] = round(
                nbytes / (d["cold_kern_ms_median"] * 1e-3) / 1e9, 1)
        if ceil is not None:
            result["decode"]["frac_of_measured_read_ceiling"] = round(
                nbytes / (d["kern_ms"] * 1e-3) / 1e9 / ceil["hbm_read_GB_s"], 4)
        print(f"[bench] decode step {d['ms']:.4f} ms, kernel {d['kern_ms']:.4f} ms", file=sys.stderr,
              flush=True)
    if args.others and args.workload == "turn":
        result["workloads"] = run_others(OTHER_WORKLOADS, args.other_steps)
    if not decode and args.policy:
        from paper_2606_16824_amd import policy_bench
        result["policy"] = policy_bench.run(host_fraction=1.0)
        result["policy_shared_prefix"] = policy_bench.run(shared_groups=4, shared_prefix_tokens=2000)
        print("[bench] policy simulation done", file=sys.stderr, flush=True)
    if not decode and args.swap:
        result["swap"] = run_swap()
        print(f"[bench] swap {result['swap']}", file=sys.stderr, flush=True)
    if args.cpu_seconds > 0:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
