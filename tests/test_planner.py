"""Properties of the host work planner (runs on the CPU)."""
import numpy as np
import pytest

import paper_2606_16824_amd as cwlib

BN = 64
BM = 256  # packed query rows per work item (both pool dtypes)


def check_plan(lp, ls, hkv, g, d=128, p=16):
    items = cwlib.plan_items(lp, ls, hkv, g, d, p)
    bm = BM
    real = items[items[:, 0] >= 0]
    # every (seq, kv head, query tile) key range [0, kv_len) is covered exactly once
    cover = {}
    for seq, kvh, r0, kb, ke, part, rows, _ in real:
        assert 0 <= kb < ke and kb % BN == 0
        cover.setdefault((seq, kvh, r0), []).append((kb, ke, part, rows))
    for b in range(len(lp)):
        nrows = ls[b] * g
        for r0 in range(0, nrows, bm):
            rows = min(bm, nrows - r0)
            kv_len = lp[b] + (r0 + rows - 1) // g + 1
            for h in range(hkv):
                ch = sorted(cover.pop((b, h, r0)))
                assert ch[0][0] == 0 and ch[-1][1] == kv_len
                for (a0, a1, _, _), (b0, _, _, _) in zip(ch, ch[1:]):
                    assert a1 == b0
                assert all(c[3] == rows for c in ch)
                parts = [c[2] for c in ch]
                if len(ch) == 1:
                    assert parts == [-1]
                else:
                    assert parts == list(range(parts[0], parts[0] + len(ch)))
    assert not cover
    allp = real[:, 5][real[:, 5] >= 0]
    assert len(np.unique(allp)) == len(allp)
    return items


def test_turn_plan_fills_every_cu():
    # 256-row items, one resident per CU
    items = check_plan([16384], [1024], 8, 4)
    assert len(items) == 256
    # XCD-aware: workgroup i runs on XCD i % 8; all work of a kv head on one XCD
    for x in range(8):
        assert len(set(items[x::8, 1].tolist())) == 1


def test_split_boundaries_weight_suffix_tiles():
    """The turn's tiles split into two chunks of equal cost, a key tile past the
    prefix costing 1.25 prefix tiles: tile 15 (272 key tiles, 16 past the
    prefix) splits after 138 tiles (13800 of 27600), not at 136."""
    items = check_plan([16384], [1024], 8, 4)
    t15 = items[(items[:, 1] == 0) & (items[:, 2] == 15 * BM)]
    assert sorted(t15[:, 3:5].tolist()) == [[0, 138 * BN], [138 * BN, 17408]]
    cwlib.set_tuning(5, 100)
    try:
        items = check_plan([16384], [1024], 8, 4)
        t15 = items[(items[:, 1] == 0) & (items[:, 2] == 15 * BM)]
        assert sorted(t15[:, 3:5].tolist()) == [[0, 136 * BN], [136 * BN, 17408]]
    finally:
        cwlib.set_tuning(5, 125)


def test_long_plan_is_dealt_round_by_round():
    """Long: 8 kv heads x 256 tiles, unsplit.  Round r (workgroups 256r ..
    256r + 255, 32 per XCD) is all of kv head r, every XCD streaming it at once;
    XCD x gets the 32 consecutive tiles of block (x + r) % 8, in reverse order
    on odd rounds, so over the eight rounds every XCD does every block once."""
    items = check_plan([131072], [8192], 8, 8, p=64)
    assert len(items) == 2048 and np.all(items[:, 5] == -1)
    keys = np.zeros(8)
    for r in range(8):
        rnd = items[256 * r:256 * (r + 1)]
        assert set(rnd[:, 1].tolist()) == {r}
        for x in range(8):
            tiles = rnd[x::8, 2] // BM  # query tile index, in launch order on XCD x
            blk = (x + r) % 8
            want = np.arange(32 * blk, 32 * blk + 32)
            assert np.array_equal(tiles, want[::-1] if r % 2 else want)
            keys[x] += (rnd[x::8, 4] - rnd[x::8, 3]).sum()
    assert keys.max() == keys.min()  # every XCD streams the same number of keys


def test_long_plan_without_dealing_keeps_a_head_per_xcd():
    cwlib.set_tuning(3, 0)
    try:
        items = check_plan([131072], [8192], 8, 8, p=64)
    finally:
        cwlib.set_tuning(3, 1)
    assert len(items) == 2048
    for x in range(8):
        assert len(set(items[x::8, 1].tolist())) == 1


def test_dealt_rounds_then_bundles():
    """A bundle of 300 tiles deals one round (256 items) and leaves 44 items
    that, with a second sequence's bundles, go to the XCD queues after it."""
    items = check_plan([4000, 500], [300 * 64, 100], 1, 4)
    real = items[items[:, 0] >= 0]
    first = items[:256]
    assert np.all(first[:, 0] == 0) and np.all(first[:, 5] == -1)
    assert len(real) == 300 + 2


@pytest.mark.parametrize("lp,ls,hkv,g", [
    ([256], [64], 1, 4),
    ([0, 37, 200, 64], [70, 1, 129, 33], 2, 1),
    ([40, 10, 0], [0, 20, 0], 1, 4),
    ([5000, 30000, 12000], [1, 1, 1], 8, 4),
    ([100] * 40, [300] * 40, 4, 2),
])
def test_plan_coverage(lp, ls, hkv, g):
    check_plan(np.array(lp), np.array(ls), hkv, g)


def test_forced_chunking():
    cwlib.set_tuning(0, 3)
    try:
        items = check_plan(np.array([700]), np.array([150]), 2, 4)
        real = items[items[:, 0] >= 0]
        assert np.all(real[:, 4] - real[:, 3] <= 3 * BN)
    finally:
        cwlib.set_tuning(0, 0)
