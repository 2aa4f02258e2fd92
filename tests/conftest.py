"""Shared pytest setup: the ``gpu`` marker and workload -> oracle-input glue."""
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def paged_inputs(w):
    """cw_workloads.Workload -> oracle.PagedInputs (raw bits, no arithmetic)."""
    from oracle import PagedInputs

    s = w.spec
    return PagedInputs(
        q=w.np_bits(w.q), k_new=w.np_bits(w.k_new), v_new=w.np_bits(w.v_new),
        k_pool=w.np_bits(w.k_pool), v_pool=w.np_bits(w.v_pool),
        block_table=w.block_table.numpy(), prefix_lens=s.prefix_lens.astype(np.int64),
        suffix_lens=s.suffix_lens.astype(np.int64), gqa_group=s.gqa_group,
        softmax_scale=s.softmax_scale, kv_dtype=s.kv_dtype,
        k_scale=None if w.k_scale is None else w.k_scale.numpy(),
        v_scale=None if w.v_scale is None else w.v_scale.numpy())


def pytest_collection_modifyitems(config, items):
    """GPU tests skip (never pass) where no GPU is visible."""
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="needs an MI355X GPU (run with -m gpu on the GPU box)")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


def pytest_terminal_summary(terminalreporter):
    """Error against tolerance of every GPU comparison of the run (largest first by
    share of the bound), so the headroom shows even in a quiet (-q) run."""
    try:
        from gpu_util import MARGINS
    except Exception:  # pragma: no cover
        return
    if not MARGINS:
        return
    tr = terminalreporter
    tr.section("parity margins (error / bound)")
    rows = sorted(MARGINS, key=lambda r: -(r[2] / r[3] if r[3] else 0.0))
    for what, n, mx, mxb, mean, meanb in rows:
        mean_s = f"mean {mean:.2e}/{meanb:.0e}" if meanb else f"mean {mean:.2e}"
        tr.write_line(f"{mx / mxb:6.1%} of max  max {mx:.2e}/{mxb:.0e}  {mean_s}  n={n}  {what}")
