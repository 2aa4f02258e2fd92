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
