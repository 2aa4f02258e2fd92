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
