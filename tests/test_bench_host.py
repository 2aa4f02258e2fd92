"""Host-side logic of bench.py: the amd-smi report parser, the committed traffic
lookup (tied to the kernel source hash) and the one-GPU guard."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# the shape of `amd-smi metric -g 0 -p -c --json` on MI355X (two of eight XCDs shown)
SMI = {"gpu_data": [{"gpu": 0,
                     "power": {"socket_power": {"value": 1283, "unit": "W"}, "gfx_voltage": "N/A"},
                     "clock": {"gfx_0": {"clk": {"value": 1970, "unit": "MHz"},
                                         "max_clk": {"value": 2400, "unit": "MHz"}},
                               "gfx_1": {"clk": {"value": 1990, "unit": "MHz"}},
                               "mem_0": {"clk": {"value": 2000, "unit": "MHz"}}}}]}


def test_smi_report_parsing():
    pw, clk = bench.parse_smi_metric(SMI)
    assert pw == 1283.0
    assert clk == 1980.0  # median over gfx_* only; the memory clock is not a GFX clock


def test_smi_report_without_fields():
    assert bench.parse_smi_metric({"gpu_data": [{"gpu": 0, "power": {"socket_power": "N/A"}}]}) == (None, None)
    assert bench.parse_smi_metric(None) == (None, None)


def test_committed_traffic_is_tied_to_the_kernel_sources():
    # every committed summary carries the bytes per launch and the hash of the kernel
    # source it was taken on; the bench reports the bytes only while that source is
    # unchanged, else null
    import hashlib
    import re
    for kind, wl in (("bf16", "turn"), ("bf16", "long"), ("bf16", "batch16"), ("fp8", "mixed"),
                     ("decode", "decode")):
        kernel, src, prof = bench.KERNEL_SOURCES[kind]
        text = open(os.path.join(ROOT, "profiles", prof.format(wl=wl))).read()
        m = re.search(r"traffic_bytes_per_launch=(\d+) kernel_source_sha256=([0-9a-f]{64})", text)
        assert m and int(m.group(1)) > 0, (kind, wl)
        sha = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
        want = int(m.group(1)) if m.group(2) == sha else None
        assert bench.measured_traffic(kind, wl) == want, (kind, wl)
    assert bench.measured_traffic("bf16", "no_such_workload") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]
