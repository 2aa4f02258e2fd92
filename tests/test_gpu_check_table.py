"""cw_check_block_table counts exactly the out-of-range page ids among the
block-table entries a call would read, and nothing past a sequence's length."""
import numpy as np
import pytest
import torch

import cw_workloads as cw
import paper_2606_16824_amd as cwlib

pytestmark = pytest.mark.gpu


def _expected(bt, lp, ls, num_pages, page):
    out = []
    for b in range(len(lp)):
        n = -(-(int(lp[b]) + int(ls[b])) // page)
        row = bt[b, :n].astype(np.int64)
        out.append(int(((row < 0) | (row >= num_pages)).sum()))
    return np.array(out)


@pytest.mark.parametrize("page", [16, 64])
def test_counts_planted_bad_ids(page):
    rng = np.random.default_rng(7 + page)
    B, num_pages, stride = 37, 5000, 90
    lp = rng.integers(0, 60 * page, B).astype(np.int32)
    ls = rng.integers(0, 20 * page, B).astype(np.int32)
    lp[0], ls[0] = 0, 0  # an empty sequence reads nothing
    bt = np.full((B, stride), np.iinfo(np.int32).max, dtype=np.int32)  # never read
    for b in range(B):
        n = -(-(int(lp[b]) + int(ls[b])) // page)
        bt[b, :n] = rng.integers(0, num_pages, n)
        for _ in range(int(rng.integers(0, 4))):
            if n:
                bt[b, int(rng.integers(0, n))] = rng.choice([-1, num_pages, num_pages + 7,
                                                             np.iinfo(np.int32).min])
    want = _expected(bt, lp, ls, num_pages, page)
    print(f"\n[case] check_block_table P={page} B={B}: {int(want.sum())} planted", flush=True)
    got = cwlib.check_block_table(torch.from_numpy(bt).cuda(), lp, ls, num_pages, page)
    assert np.array_equal(got, want)
    assert want.sum() > 0


def test_many_sequences_grid_stride():
    B, page, num_pages = 70000, 16, 100
    lp = np.full(B, 17, dtype=np.int32)
    ls = np.ones(B, dtype=np.int32)
    bt = np.zeros((B, 2), dtype=np.int32)
    bt[::3, 1] = num_pages  # every third sequence reads one bad entry
    bt[1::3, 0] = -5
    print(f"\n[case] check_block_table B={B}", flush=True)
    got = cwlib.check_block_table(torch.from_numpy(bt).cuda(), lp, ls, num_pages, page)
    assert np.array_equal(got, _expected(bt, lp, ls, num_pages, page))


def test_valid_workloads_are_clean():
    for name in ("turn", "batch16", "long", "mixed"):
        s = cw.spec_for(name)
        bt = cw.build_block_table(s, np.random.default_rng(s.seed))
        print(f"\n[case] check_block_table {name}", flush=True)
        got = cwlib.check_block_table(torch.from_numpy(bt).cuda(), s.prefix_lens, s.suffix_lens,
                                      s.num_pages, s.page_size)
        assert got.shape == (s.num_seqs,) and not got.any()
