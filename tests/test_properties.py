"""Randomised properties (hypothesis, CPU only).

- The extend planner: for any lengths, head counts and tunings, every
  (sequence, kv head, query tile) key range is covered exactly once, partial
  slots are unique and consecutive per tile, and idle items carry no work.
- The decode plan: rebuilt from its compact form (what the upload kernel does
  on the device), it is exactly the planner's work list and merge groups.
- The policy: the library's simulator and block manager give exactly the
  oracle's block-level model (dispatch order, counters, block counts and cached
  tokens of every dispatch) on small random traces with random shared-prefix
  groups, for every scheduling x eviction pair, with and without offload to a
  host pool (sizes from none to more than every evicted block)."""
import os

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import paper_2606_16824_amd as cwlib
from oracle import cachewise_policy as cp
from paper_2606_16824_amd import policy
from test_planner import check_plan

# CW_PROPERTY_EXAMPLES raises the number of examples for a longer search
SETTINGS = settings(max_examples=int(os.environ.get("CW_PROPERTY_EXAMPLES", "120")), deadline=None,
                    suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])


@st.composite
def plan_case(draw):
    b = draw(st.integers(1, 12))
    lp = draw(st.lists(st.integers(0, 3000), min_size=b, max_size=b))
    ls = draw(st.lists(st.integers(0, 700), min_size=b, max_size=b))
    hkv = draw(st.sampled_from([1, 2, 3, 8]))
    g = draw(st.sampled_from([1, 2, 4, 8, 16]))
    chunk = draw(st.sampled_from([0, 0, 0, 1, 3, 7]))
    weight = draw(st.sampled_from([1, 100, 125, 250, 10000]))
    deal = draw(st.sampled_from([0, 1]))
    target = draw(st.sampled_from([0, 0, 16, 1000]))
    return lp, ls, hkv, g, chunk, weight, deal, target


@SETTINGS
@given(plan_case())
def test_planner_covers_every_key_range_once(case):
    lp, ls, hkv, g, chunk, weight, deal, target = case
    cwlib.set_tuning(0, chunk)
    cwlib.set_tuning(1, target)
    cwlib.set_tuning(3, deal)
    cwlib.set_tuning(5, weight)
    try:
        items = check_plan(np.array(lp), np.array(ls), hkv, g)
    finally:
        cwlib.set_tuning(0, 0)
        cwlib.set_tuning(1, 0)
        cwlib.set_tuning(3, 1)
        cwlib.set_tuning(5, 125)
    idle = items[items[:, 0] < 0]
    assert np.all(idle[:, 4] == idle[:, 3])  # no keys
    if len(items):
        assert items[-1, 0] >= 0  # no trailing idle items


@st.composite
def decode_case(draw):
    b = draw(st.integers(1, 40))
    lp = draw(st.lists(st.sampled_from([0, 1, 15, 16, 17, 63, 64, 65, 255, 256, 257, 1000, 4095, 4096,
                                        4097, 20000, 65536, 131071]), min_size=b, max_size=b))
    hkv = draw(st.sampled_from([1, 2, 8]))
    g = draw(st.sampled_from([1, 4, 8, 16]))
    d = draw(st.sampled_from([64, 128]))
    p = draw(st.sampled_from([16, 64]))
    dt = draw(st.sampled_from(["bf16", "fp8"]))
    chunk = draw(st.sampled_from([0, 0, 1, 2, 5, 64]))
    target = draw(st.sampled_from([0, 0, 16, 1000, 100000]))
    return lp, hkv, g, d, p, dt, chunk, target


@SETTINGS
@given(decode_case())
def test_decode_plan_rebuilt_from_compact_form_is_the_plan(case):
    """The upload kernel's rebuild of a decode plan from its compact form (the
    same function, run on the host) gives exactly the planner's items and merge
    groups, for any lengths, head counts, tile shapes and tunings."""
    lp, hkv, g, d, p, dt, chunk, target = case
    cwlib.set_tuning(0, chunk)
    cwlib.set_tuning(1, target)
    try:
        items, groups = cwlib.decode_plan(lp, hkv, g, d, p, dt, rebuilt=False)
        r_items, r_groups = cwlib.decode_plan(lp, hkv, g, d, p, dt, rebuilt=True)
    finally:
        cwlib.set_tuning(0, 0)
        cwlib.set_tuning(1, 0)
    assert np.array_equal(items, r_items)
    assert np.array_equal(groups, r_groups)
    # and the plan covers every (sequence, kv head) key range [0, Lp + 1) once
    for b in range(len(lp)):
        for h in range(hkv):
            rows = items[(items[:, 0] == b) & (items[:, 1] == h)]
            spans = sorted((int(x[3]), int(x[4])) for x in rows)
            assert spans[0][0] == 0 and spans[-1][1] == lp[b] + 1
            assert all(spans[i][1] == spans[i + 1][0] for i in range(len(spans) - 1))


B = 4  # block tokens of the random traces


@st.composite
def trace(draw):
    n = draw(st.integers(1, 5))
    n_tools = draw(st.integers(1, 2))
    n_groups = draw(st.integers(0, 2))
    shared = [draw(st.integers(0, 12)) for _ in range(n_groups)]
    sessions, groups = [], []
    for _ in range(n):
        g = draw(st.integers(-1, n_groups - 1))
        k = draw(st.integers(1, 4))
        turns = []
        for j in range(k):
            lo = shared[g] if (g >= 0 and j == 0) else 1
            tin = draw(st.integers(lo, lo + 30))
            tout = draw(st.integers(0, 8))
            tool = draw(st.integers(0, n_tools - 1))
            dur = draw(st.sampled_from([0.0, 0.5, 2.0, 7.0, 19.0, 40.0]))
            turns.append((tin, tout, tool, dur))
        start = draw(st.sampled_from([0.0, 0.0, 1.0, 5.0, 12.5]))
        sessions.append((start, turns))
        groups.append(g)
    history = [sorted(draw(st.lists(st.sampled_from([0.5, 1.0, 3.0, 10.0, 30.0]), min_size=1,
                                    max_size=4))) for _ in range(n_tools)]
    need = max(-(-sum(ti + to for ti, to, _, _ in turns) // B) for _, turns in sessions)
    cap = max(1, need) + draw(st.integers(0, 12))
    sched = draw(st.sampled_from(["fcfs", "prefix"]))
    evict = draw(st.sampled_from(["lru", "predictive", "belady"]))
    rebuild = draw(st.integers(1, 4))
    host = draw(st.sampled_from([0, 0, 1, 2, 5, 40]))
    swap_s = draw(st.sampled_from([0.0, 0.03]))
    return sessions, groups, shared, history, cap, sched, evict, rebuild, host, swap_s


@SETTINGS
@given(trace())
def test_simulator_matches_the_block_level_oracle(case):
    sessions, groups, shared, history, cap, sched, evict, rebuild, host, swap_s = case
    kw = dict(capacity_blocks=cap, block_tokens=B, prefill_s_per_token=0.01, decode_s_per_token=0.05)
    got = policy.simulate(sessions, history, sched=sched, evict=evict, rebuild_every=rebuild,
                          groups=groups if shared else None, shared_tokens=shared if shared else None,
                          log=True, host_blocks=host, swap_s_per_block=swap_s, **kw)
    want, wlog = cp.simulate_blocks(
        cp.Config(M=cap, block_tokens=B, prefill_s_per_token=0.01, decode_s_per_token=0.05,
                  sched=sched, evict=evict, n_rebuild=rebuild, host_blocks=host,
                  swap_s_per_block=swap_s),
        [cp.SessionSpec(st_, [cp.Turn(*t) for t in turns], group=groups[i] if shared else -1)
         for i, (st_, turns) in enumerate(sessions)],
        history, shared_tokens=shared)
    assert got["dispatch"] == want.dispatch
    for f in ("requests", "faults", "evicted_blocks", "recomputed_tokens", "prefilled_tokens",
              "heap_rebuilds", "swapped_out_blocks", "swapped_in_blocks"):
        assert got[f] == getattr(want, f), f
    for f in ("makespan_s", "mean_session_s"):
        assert got[f] == pytest.approx(getattr(want, f), rel=1e-12), f
    assert [(s, c, n, len(t)) for s, c, n, t in got["log"]] == \
        [(d.session, d.cached_tokens, d.new_tokens, d.blocks) for d in wlog]
    assert got["log_swaps"] == [(d.swapped_in, d.swapped_out) for d in wlog]
    for _, _, _, t in got["log"]:
        assert len(set(t)) == len(t) and all(0 <= x < cap for x in t)
