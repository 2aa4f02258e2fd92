"""The library's CacheWise policy simulator (C++, host-only) against the oracle
(CPU): identical dispatch orders and counters on seeded agent-session traces for
every scheduling x eviction pair, and the validation of its C ABI."""
import ctypes as C
import itertools
import random

import numpy as np
import pytest

import cw_workloads as cw
from oracle import cachewise_policy as cp
from paper_2606_16824_amd import _lib as L
from paper_2606_16824_amd import policy


def _to_oracle(sessions):
    return [cp.SessionSpec(st, [cp.Turn(*t) for t in turns]) for st, turns in sessions]


FIELDS_EXACT = ("requests", "faults", "evicted_blocks", "recomputed_tokens", "prefilled_tokens",
                "heap_rebuilds")
FIELDS_TIME = ("makespan_s", "mean_session_s", "goodput_tok_s")


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("sched,evict", list(itertools.product(("fcfs", "prefix"),
                                                               ("lru", "predictive", "belady"))))
def test_simulator_matches_oracle(seed, sched, evict):
    tr = cw.agent_sessions(num_sessions=12, seed=2000 + seed, max_turns=12)
    kw = dict(capacity_blocks=tr.capacity_blocks, block_tokens=tr.block_tokens,
              prefill_s_per_token=tr.prefill_s_per_token, decode_s_per_token=tr.decode_s_per_token)
    got = policy.simulate(tr.sessions, tr.history, sched=sched, evict=evict, rebuild_every=3, **kw)
    want = cp.simulate(cp.Config(M=tr.capacity_blocks, block_tokens=tr.block_tokens,
                                 prefill_s_per_token=tr.prefill_s_per_token,
                                 decode_s_per_token=tr.decode_s_per_token, sched=sched, evict=evict,
                                 n_rebuild=3), _to_oracle(tr.sessions), tr.history)
    assert got["dispatch"] == want.dispatch
    for f in FIELDS_EXACT:
        assert got[f] == getattr(want, f), f
    for f in FIELDS_TIME:
        assert got[f] == pytest.approx(getattr(want, f), rel=1e-12), f
    assert got["evicted_blocks"] > 0  # the traces are sized to need eviction


def test_predictor_matches_oracle():
    rng = np.random.default_rng(3)
    hist = [rng.lognormal(1.0, 1.2, size=500).tolist(), [2.0, 8.0], []]
    for y in (0, 1):
        for e in (0.0, 0.7, 3.0, 9.0, 50.0):
            assert policy.predict(hist, y, e) == pytest.approx(cp.predict_remaining(hist[y], e), rel=1e-12)
    assert policy.predict(hist, 2, 4.0) == 4.0  # no history: elapsed


def _raw(cfg=None, trace=None, result=True):
    return L.SIGNATURES and policy.library().cw_policy_simulate(
        None if cfg is None else C.byref(cfg), None if trace is None else C.byref(trace),
        C.byref(policy._Result()) if result else None, None, 0)


def test_validation():
    sessions = [(0.0, [(10, 2, 0, 1.0), (5, 1, 0, 0.0)])]
    tr, keep = policy._trace(sessions, [[1.0]])
    good = policy._Config(8, 4, 0.0, 0.0, 1, 1, 3)
    assert _raw(good, tr) == L.CW_OK
    assert _raw(None, tr) == L.CW_ERR_NULL
    assert _raw(good, None) == L.CW_ERR_NULL
    assert _raw(good, tr, result=False) == L.CW_ERR_NULL
    for bad in (policy._Config(0, 4, 0, 0, 1, 1, 3), policy._Config(8, 0, 0, 0, 1, 1, 3),
                policy._Config(8, 4, -1.0, 0, 1, 1, 3), policy._Config(8, 4, 0, 0, 2, 1, 3),
                policy._Config(8, 4, 0, 0, 1, 3, 3), policy._Config(8, 4, 0, 0, 1, 1, 0)):
        assert _raw(bad, tr) == L.CW_ERR_UNSUPPORTED
    # a turn needing more blocks than the node holds
    assert _raw(policy._Config(4, 4, 0, 0, 1, 1, 3), tr) == L.CW_ERR_BAD_LENS
    for bad_sessions, hist in (([(0.0, [(-1, 2, 0, 1.0)])], [[1.0]]),      # negative tokens
                               ([(0.0, [(1, 2, 5, 1.0), (1, 1, 0, 0.0)])], [[1.0]]),  # tool id
                               ([(-2.0, [(1, 2, 0, 1.0)])], [[1.0]]),      # negative start
                               ([(0.0, [(1, 2, 0, -1.0), (1, 0, 0, 0.0)])], [[1.0]]),  # tool time
                               ([(0.0, [(1, 2, 0, 1.0)])], [[-1.0]])):      # history sample
        t2, k2 = policy._trace(bad_sessions, hist)
        assert _raw(good, t2) == L.CW_ERR_BAD_LENS
    assert policy.library().cw_last_error_message()


# ---- the block manager with shared prefix groups

def _to_oracle_groups(sessions, groups):
    return [cp.SessionSpec(st, [cp.Turn(*t) for t in turns], group=groups[i])
            for i, (st, turns) in enumerate(sessions)]


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("sched,evict", list(itertools.product(("fcfs", "prefix"),
                                                               ("lru", "predictive", "belady"))))
def test_simulator_with_shared_prefixes_matches_oracle(seed, sched, evict):
    tr = cw.agent_sessions(num_sessions=10, seed=2100 + seed, max_turns=8, shared_groups=2,
                           shared_prefix_tokens=1024)
    kw = dict(capacity_blocks=tr.capacity_blocks, block_tokens=tr.block_tokens,
              prefill_s_per_token=tr.prefill_s_per_token, decode_s_per_token=tr.decode_s_per_token)
    got = policy.simulate(tr.sessions, tr.history, sched=sched, evict=evict, rebuild_every=3,
                          groups=tr.groups, shared_tokens=tr.shared_tokens, log=True, **kw)
    want, wlog = cp.simulate_blocks(
        cp.Config(M=tr.capacity_blocks, block_tokens=tr.block_tokens,
                  prefill_s_per_token=tr.prefill_s_per_token, decode_s_per_token=tr.decode_s_per_token,
                  sched=sched, evict=evict, n_rebuild=3),
        _to_oracle_groups(tr.sessions, tr.groups), tr.history, shared_tokens=tr.shared_tokens)
    assert got["dispatch"] == want.dispatch
    for f in FIELDS_EXACT:
        assert got[f] == getattr(want, f), f
    for f in FIELDS_TIME:
        assert got[f] == pytest.approx(getattr(want, f), rel=1e-12), f
    assert [(s, c, n, len(t)) for s, c, n, t in got["log"]] == \
        [(d.session, d.cached_tokens, d.new_tokens, d.blocks) for d in wlog]
    assert any(c > 0 for _, c, _, _ in got["log"])
    for _, _, _, t in got["log"]:
        assert len(set(t)) == len(t) and min(t) >= 0 and max(t) < tr.capacity_blocks


def test_simulator_worked_sharing_examples():
    # the oracle's hand-worked cases, through the library
    got = policy.simulate([(0.0, [(10, 2, 0, 0.0)]), (100.0, [(9, 3, 0, 0.0)])], [[1.0]],
                          capacity_blocks=10, block_tokens=4, prefill_s_per_token=1.0, sched="fcfs",
                          evict="lru", groups=[0, 0], shared_tokens=[8], log=True)
    assert [(s, c, n, len(t)) for s, c, n, t in got["log"]] == [(0, 0, 10, 3), (1, 8, 1, 3)]
    assert got["log"][0][3][:2] == got["log"][1][3][:2]  # the shared blocks are the same blocks
    got = policy.simulate([(0.0, [(10, 2, 0, 50.0), (4, 0, 0, 0.0)]), (20.0, [(9, 3, 0, 0.0)]),
                           (30.0, [(8, 0, 0, 0.0)])], [[1.0]], capacity_blocks=5, block_tokens=4,
                          prefill_s_per_token=1.0, sched="fcfs", evict="lru", groups=[0, 0, -1],
                          shared_tokens=[8], log=True)
    assert got["dispatch"] == [0, 1, 2, 0]
    assert [(c, n, len(t)) for _, c, n, t in got["log"]] == [(0, 10, 3), (8, 1, 3), (0, 8, 2), (8, 8, 4)]
    assert (got["evicted_blocks"], got["faults"], got["recomputed_tokens"], got["prefilled_tokens"]) == (3, 1, 4, 27)


def test_block_manager_references_sharing_and_eviction_order():
    bm = policy.BlockManager(capacity_blocks=6, block_tokens=4)
    bm.add_session(0, group=0, shared_tokens=8)
    bm.add_session(1, group=0, shared_tokens=8)
    bm.add_session(2)
    t0, cached, ev = bm.admit(0, 0, 10, 2)  # 3 blocks: 2 shared + 1 private
    assert len(t0) == 3 and cached == 0 and ev == 0
    assert bm.stats() == {"free_blocks": 3, "referenced_blocks": 3}
    t1, cached, ev = bm.admit(1, 0, 9, 3)   # both requests run at once: the shared blocks have 2 refs
    assert list(t1[:2]) == list(t0[:2]) and cached == 8 and len(t1) == 3 and t1[2] != t0[2]
    assert bm.stats() == {"free_blocks": 2, "referenced_blocks": 4}
    with pytest.raises(RuntimeError):
        bm.admit(2, 0, 12, 0)  # 3 blocks, only 2 free and nothing unreferenced
    bm.release(0, 5.0)
    assert bm.stats()["referenced_blocks"] == 3  # session 1 still holds the shared blocks
    t2, cached, ev = bm.admit(2, 0, 12, 0)      # evicts session 0's private block only
    assert cached == 0 and ev == 1 and t0[2] in list(t2)
    bm.release(1, 1.0)
    bm.release(2, 9.0)
    # session 3 needs 5 blocks with none free: session 2's blocks go first (value
    # 9), then session 1's private block (value 1), then the tail shared block
    # (the smallest sharer value, 1, and after the sharers' private blocks)
    bm.add_session(3)
    t3, _, ev = bm.admit(3, 0, 20, 0)
    assert ev == 5 and set(t3) == set(t2) | {t1[2], t1[1]}
    assert bm.stats() == {"free_blocks": 0, "referenced_blocks": 5}
    bm.release(3, 7.0)
    t0b, cached, _ = bm.admit(0, 12, 4, 0)      # only the head shared block is still resident
    assert cached == 4 and t0b[0] == t0[0]
    with pytest.raises(RuntimeError):
        bm.release(2, 0.0)  # no request running
    bm.close()


def test_block_manager_rebuild_reorders_eviction():
    bm = policy.BlockManager(capacity_blocks=4, block_tokens=4)
    for s in range(3):
        bm.add_session(s)
    a, _, _ = bm.admit(0, 0, 8, 0)
    bm.release(0, 1.0)
    b, _, _ = bm.admit(1, 0, 8, 0)
    bm.release(1, 2.0)  # larger value: evicted first
    bm.rebuild({0: 3.0, 1: 2.0})  # now session 0's blocks go first
    c, _, ev = bm.admit(2, 0, 8, 0)
    assert ev == 2 and set(c) == set(a)


def test_block_manager_limits_are_errors_not_crashes():
    """Sizes past the documented limits come back as status codes, and a
    rejected call changes nothing."""
    lib = L.load()
    h = C.c_void_p()
    assert lib.cw_bm_create((1 << 26) + 1, 16, C.byref(h)) == L.CW_ERR_UNSUPPORTED and not h.value
    assert lib.cw_bm_create(0, 16, C.byref(h)) == L.CW_ERR_UNSUPPORTED
    assert lib.cw_bm_create(64, 0, C.byref(h)) == L.CW_ERR_UNSUPPORTED
    assert lib.cw_bm_create(64, 16, None) == L.CW_ERR_NULL
    assert lib.cw_bm_create(64, 16, C.byref(h)) == L.CW_OK
    try:
        assert lib.cw_bm_add_session(h, 1 << 24, -1, 0) == L.CW_ERR_UNSUPPORTED
        assert lib.cw_bm_add_session(h, 3, 1 << 24, 0) == L.CW_ERR_UNSUPPORTED
        assert lib.cw_bm_add_session(h, -1, -1, 0) == L.CW_ERR_BAD_LENS
        blocks, cached, ev = C.c_int32(), C.c_int64(), C.c_int64()
        table = np.zeros(8, np.int32)
        # session 3 was not registered by the rejected calls
        assert lib.cw_bm_admit(h, 3, 0, 10, 0, table.ctypes.data, 8, C.byref(blocks), C.byref(cached),
                               C.byref(ev)) == L.CW_ERR_BAD_LENS
        assert lib.cw_bm_add_session(h, 3, -1, 0) == L.CW_OK
        assert lib.cw_bm_add_session(h, 3, -1, 0) == L.CW_ERR_BAD_LENS  # twice
        for args in ((1 << 40) + 1, 0, 0), (0, (1 << 40) + 1, 0), (0, 0, -1):
            assert lib.cw_bm_admit(h, 3, *args, table.ctypes.data, 8, C.byref(blocks), C.byref(cached),
                                   C.byref(ev)) == L.CW_ERR_BAD_LENS
        assert lib.cw_bm_admit(h, 3, 0, 10, 0, table.ctypes.data, -1, C.byref(blocks), C.byref(cached),
                               C.byref(ev)) == L.CW_ERR_BAD_LENS
        free, ref = C.c_int64(), C.c_int64()
        assert lib.cw_bm_stats(h, C.byref(free), C.byref(ref)) == L.CW_OK
        assert (free.value, ref.value) == (64, 0)
        # a request larger than the node
        assert lib.cw_bm_admit(h, 3, 0, 65 * 16, 0, table.ctypes.data, 8, C.byref(blocks), C.byref(cached),
                               C.byref(ev)) == L.CW_ERR_WORKSPACE
        assert lib.cw_bm_admit(h, 3, 0, 40, 0, table.ctypes.data, 8, C.byref(blocks), C.byref(cached),
                               C.byref(ev)) == L.CW_OK
        assert blocks.value == 3 and list(table[:3]) == [0, 1, 2]
        assert lib.cw_bm_release(h, 3, float("nan")) == L.CW_ERR_BAD_LENS
        assert lib.cw_bm_release(h, 3, 1.0) == L.CW_OK
        assert lib.cw_bm_release(h, 3, 1.0) == L.CW_ERR_BAD_LENS  # nothing running
    finally:
        lib.cw_bm_destroy(h)


def test_simulator_capacity_limit():
    tr = cw.agent_sessions(num_sessions=2, seed=2000, max_turns=2)
    with pytest.raises(RuntimeError):
        policy.simulate(tr.sessions, tr.history, capacity_blocks=(1 << 26) + 1, block_tokens=16)
