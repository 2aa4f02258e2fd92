"""Pins of the CacheWise policy oracle (CPU): the predictor's closed forms,
Belady's rule against an exhaustive search and LRU against a textbook cache on
classic paging traces, a hand-worked prefix-aware dispatch, and the equality of
predictive eviction with a perfect predictor and Belady's rule."""
import itertools
import random
from collections import OrderedDict

import numpy as np
import pytest

from oracle import cachewise_policy as cp


def test_predictor_closed_forms():
    h = [1.0, 2.0, 3.0, 4.0]
    assert cp.predict_remaining(h, 0.0) == 2.5
    assert cp.predict_remaining(h, 2.5) == pytest.approx(1.0)   # (0.5 + 1.5) / 2
    assert cp.predict_remaining(h, 5.0) == 5.0                  # no sample left: elapsed
    # memoryless exponential: the expected remaining time does not depend on elapsed
    x = np.random.default_rng(0).exponential(10.0, size=200_000).tolist()
    for e in (0.0, 5.0, 20.0):
        assert cp.predict_remaining(x, e) == pytest.approx(10.0, rel=0.03)
    # uniform on [0, 10]: E[remaining | elapsed e] = (10 - e) / 2
    u = np.linspace(0.0, 10.0, 100_001).tolist()
    for e in (0.0, 4.0, 9.0):
        assert cp.predict_remaining(u, e) == pytest.approx((10.0 - e) / 2, rel=1e-3)


def _paging_sessions(seq):
    """Classic paging as sessions of one block each: access number n of page p
    arrives at time n + 1 and is served in zero time."""
    times = {}
    for n, p in enumerate(seq):
        times.setdefault(p, []).append(float(n + 1))
    sessions = []
    for p in sorted(times):
        ts = times[p]
        turns = [cp.Turn(1, 0, 0, ts[m + 1] - ts[m] if m + 1 < len(ts) else 0.0) for m in range(len(ts))]
        sessions.append(cp.SessionSpec(ts[0], turns))
    return sessions, sorted(times)


def _min_misses(seq, cap):
    best = [None]

    def go(i, cache, misses):
        if best[0] is not None and misses >= best[0]:
            return
        if i == len(seq):
            best[0] = misses
            return
        p = seq[i]
        if p in cache:
            go(i + 1, cache, misses)
        elif len(cache) < cap:
            go(i + 1, cache | {p}, misses + 1)
        else:
            for v in cache:
                go(i + 1, (cache - {v}) | {p}, misses + 1)
    go(0, frozenset(), 0)
    return best[0]


def _lru_misses(seq, cap):
    c, m = OrderedDict(), 0
    for p in seq:
        if p in c:
            c.move_to_end(p)
        else:
            m += 1
            if len(c) == cap:
                c.popitem(last=False)
            c[p] = True
    return m


@pytest.mark.parametrize("seed", range(40))
def test_belady_is_optimal_and_lru_is_lru_on_paging_traces(seed):
    rng = random.Random(seed)
    pages = rng.randint(3, 4)
    cap = rng.randint(2, pages - 1)
    seq = [rng.randrange(pages) for _ in range(rng.randint(4, 11))]
    sessions, ids = _paging_sessions(seq)
    hist = [[1.0]]
    compulsory = len(ids)
    for evict, want in (("belady", _min_misses(seq, cap)), ("lru", _lru_misses(seq, cap))):
        r = cp.simulate(cp.Config(M=cap, block_tokens=1000, sched="fcfs", evict=evict), sessions, hist)
        assert r.faults + compulsory == want, (seq, cap, evict)
        # dispatch order is the access order
        assert [ids[i] for i in r.dispatch] == seq


def test_prefix_aware_dispatch_hand_worked():
    # session 3 occupies the engine from 9.9 to 11.9; sessions 0, 1, 2 queue meanwhile
    # with a_i = 4, 1, 3 new blocks (block = 1 token): prefix-aware serves 1, 2, 0,
    # FCFS serves them in arrival order 0, 2, 1
    S = cp.SessionSpec
    T = cp.Turn
    sessions = [
        S(0.0, [T(5, 0, 0, 10.0), T(4, 0)]),    # resident 5 after turn 1, then needs 4 more (at t=10.0)
        S(0.1, [T(2, 0, 0, 10.1), T(1, 0)]),    # resident 2, needs 1 more (at t=10.2)
        S(10.1, [T(3, 0)]),                     # first turn: 3 blocks
        S(9.9, [T(2000, 0)]),                   # long: 2000 tokens at 1 ms each
    ]
    hist = [[1.0]]
    base = dict(M=10_000, block_tokens=1, prefill_s_per_token=1e-3)
    r = cp.simulate(cp.Config(sched="prefix", evict="lru", **base), sessions, hist)
    assert r.dispatch == [0, 1, 3, 1, 2, 0]
    r = cp.simulate(cp.Config(sched="fcfs", evict="lru", **base), sessions, hist)
    assert r.dispatch == [0, 1, 3, 0, 2, 1]


def _random_sessions(rng, n_sessions, n_tools, fixed_tool_s=None):
    sessions = []
    for s in range(n_sessions):
        turns = []
        for _ in range(rng.randint(1, 6)):
            y = rng.randrange(n_tools)
            dur = fixed_tool_s[y] if fixed_tool_s else rng.uniform(0.0, 30.0)
            turns.append(cp.Turn(rng.randint(1, 400), rng.randint(0, 60), y, dur))
        sessions.append(cp.SessionSpec(rng.uniform(0.0, 20.0), turns))
    return sessions


@pytest.mark.parametrize("seed", range(12))
def test_predictive_with_a_perfect_predictor_is_belady(seed):
    # every call of tool type y takes exactly x_y and the history is [x_y]: the
    # predictor returns the true remaining time, and with a rebuild at every
    # dispatch the predictive policy makes Belady's choices
    rng = random.Random(100 + seed)
    x = [rng.uniform(0.5, 40.0) for _ in range(3)]
    sessions = _random_sessions(rng, rng.randint(3, 8), 3, fixed_tool_s=x)
    cfg = dict(M=rng.randint(30, 60), block_tokens=16, prefill_s_per_token=2e-3, decode_s_per_token=2e-2)
    need = max(-(-sum(t.in_tokens + t.out_tokens for t in s.turns) // 16) for s in sessions)
    cfg["M"] = max(cfg["M"], need)
    a = cp.simulate(cp.Config(sched="prefix", evict="predictive", n_rebuild=1, **cfg), sessions, [[v] for v in x])
    b = cp.simulate(cp.Config(sched="prefix", evict="belady", **cfg), sessions, [[v] for v in x])
    assert a.dispatch == b.dispatch
    assert (a.evicted_blocks, a.faults, a.recomputed_tokens) == (b.evicted_blocks, b.faults, b.recomputed_tokens)
    assert a.makespan_s == b.makespan_s


def test_unbounded_capacity_never_evicts():
    rng = random.Random(7)
    sessions = _random_sessions(rng, 6, 2)
    for sched, evict in itertools.product(("fcfs", "prefix"), ("lru", "predictive", "belady")):
        r = cp.simulate(cp.Config(M=10**9, block_tokens=16, prefill_s_per_token=1e-3, sched=sched,
                                  evict=evict), sessions, [[1.0, 2.0], [3.0]])
        assert r.evicted_blocks == 0 and r.faults == 0 and r.recomputed_tokens == 0
        assert r.prefilled_tokens == sum(t.in_tokens for s in sessions for t in s.turns)
        assert r.requests == sum(len(s.turns) for s in sessions)


# ---- block-level model with shared prefix blocks (simulate_blocks)

def _to_oracle_sessions(sessions, groups=None):
    return [cp.SessionSpec(st, [cp.Turn(*t) for t in turns], group=-1 if groups is None else groups[i])
            for i, (st, turns) in enumerate(sessions)]


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("sched,evict", list(itertools.product(("fcfs", "prefix"),
                                                               ("lru", "predictive", "belady"))))
def test_block_model_without_groups_is_the_session_model(seed, sched, evict):
    import cw_workloads as cw
    tr = cw.agent_sessions(num_sessions=12, seed=2000 + seed, max_turns=12)
    cfg = cp.Config(M=tr.capacity_blocks, block_tokens=tr.block_tokens,
                    prefill_s_per_token=tr.prefill_s_per_token, decode_s_per_token=tr.decode_s_per_token,
                    sched=sched, evict=evict, n_rebuild=3)
    a = cp.simulate(cfg, _to_oracle_sessions(tr.sessions), tr.history)
    b, log = cp.simulate_blocks(cfg, _to_oracle_sessions(tr.sessions), tr.history)
    assert a.dispatch == b.dispatch and [d.session for d in log] == a.dispatch
    for f in ("requests", "faults", "evicted_blocks", "recomputed_tokens", "prefilled_tokens",
              "heap_rebuilds", "makespan_s", "mean_session_s"):
        assert getattr(a, f) == getattr(b, f), f
    assert sum(d.new_tokens for d in log) == a.prefilled_tokens


def test_shared_prefix_hit_worked_example():
    # B = 4, shared prefix of 8 tokens (2 blocks).  S0 prefills its 10-token prompt
    # (no hit) into 3 blocks; S1 arrives later, finds both shared blocks resident
    # and prefills 1 of its 9 prompt tokens.
    cfg = cp.Config(M=10, block_tokens=4, prefill_s_per_token=1.0, sched="fcfs", evict="lru")
    ss = [cp.SessionSpec(0.0, [cp.Turn(10, 2)], group=0), cp.SessionSpec(100.0, [cp.Turn(9, 3)], group=0)]
    r, log = cp.simulate_blocks(cfg, ss, [[1.0]], shared_tokens=[8])
    assert [(d.session, d.cached_tokens, d.new_tokens, d.blocks) for d in log] == [(0, 0, 10, 3), (1, 8, 1, 3)]
    assert (r.requests, r.evicted_blocks, r.prefilled_tokens, r.recomputed_tokens) == (2, 0, 11, 0)


def test_shared_blocks_outlive_their_sharers_private_tails_worked_example():
    # M = 5 blocks of 4 tokens, LRU.  S0 (group 0) and S1 (group 0) share 2 blocks and
    # hold one private block each; S2 arrives at t = 30 needing 2 blocks with 1 free:
    # the least recently used candidate is S0's private block (last use 10; the shared
    # blocks count as used at 21 by S1).  S0's second turn at t = 60 finds its shared
    # blocks but not its private one (a fault, 4 context tokens recomputed) and needs 2
    # blocks with none free: S1's private block (21) goes, then S2's tail (38).
    cfg = cp.Config(M=5, block_tokens=4, prefill_s_per_token=1.0, sched="fcfs", evict="lru")
    ss = [cp.SessionSpec(0.0, [cp.Turn(10, 2, 0, 50.0), cp.Turn(4, 0)], group=0),
          cp.SessionSpec(20.0, [cp.Turn(9, 3)], group=0),
          cp.SessionSpec(30.0, [cp.Turn(8, 0)])]
    r, log = cp.simulate_blocks(cfg, ss, [[1.0]], shared_tokens=[8])
    assert r.dispatch == [0, 1, 2, 0]
    assert [(d.cached_tokens, d.new_tokens, d.blocks) for d in log] == [(0, 10, 3), (8, 1, 3), (0, 8, 2), (8, 8, 4)]
    assert (r.evicted_blocks, r.faults, r.recomputed_tokens, r.prefilled_tokens) == (3, 1, 4, 27)


def test_shared_blocks_of_finished_sharers_are_evicted_first_worked_example():
    # Predictive eviction, rebuilt every dispatch.  S0 (group 0) fills the 2 shared
    # blocks and finishes; S1 needs all 4 blocks: the shared blocks' only attached
    # sharer is done (priority +inf), so they go; S2 of group 0 then misses them.
    cfg = cp.Config(M=4, block_tokens=4, prefill_s_per_token=1.0, sched="fcfs", evict="predictive",
                    n_rebuild=1)
    ss = [cp.SessionSpec(0.0, [cp.Turn(8, 0)], group=0), cp.SessionSpec(10.0, [cp.Turn(12, 4)]),
          cp.SessionSpec(20.0, [cp.Turn(8, 4)], group=0)]
    r, log = cp.simulate_blocks(cfg, ss, [[5.0]], shared_tokens=[8])
    assert [d.cached_tokens for d in log] == [0, 0, 0]
    assert (r.requests, r.evicted_blocks, r.prefilled_tokens, r.heap_rebuilds) == (3, 5, 28, 3)


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("sched,evict", list(itertools.product(("fcfs", "prefix"),
                                                               ("lru", "predictive", "belady"))))
def test_block_model_with_groups_accounting(seed, sched, evict):
    import cw_workloads as cw
    tr = cw.agent_sessions(num_sessions=10, seed=2100 + seed, max_turns=8, shared_groups=2,
                           shared_prefix_tokens=1024)
    cfg = cp.Config(M=tr.capacity_blocks, block_tokens=tr.block_tokens, prefill_s_per_token=1e-5,
                    decode_s_per_token=1e-3, sched=sched, evict=evict, n_rebuild=3)
    r, log = cp.simulate_blocks(cfg, _to_oracle_sessions(tr.sessions, tr.groups), tr.history,
                                shared_tokens=tr.shared_tokens)
    assert sum(d.new_tokens for d in log) == r.prefilled_tokens
    # every session's later turns and every group's first requests after the first can hit
    assert any(d.cached_tokens > 0 for d in log)
    # the same sessions without the groups prefill at least as much
    r0, _ = cp.simulate_blocks(cfg, _to_oracle_sessions(tr.sessions), tr.history)
    assert r0.prefilled_tokens >= r.prefilled_tokens


# ---- offload (evicted blocks to a host pool, swapped back when the session resumes)

def test_offload_worked_example():
    """M = 4 blocks of 4 tokens, prefill 1 s/token, swaps 1 s/block, FCFS + LRU.
    A (t=0): 8 tokens, tool 10 s, then 4.  B (t=1): 8 tokens, tool 20 s, then 4.
    A runs 0-8, B 8-16.  A's second turn (t=18) needs a third block: B's tail goes
    to the host (1 swap out), A prefills its 4 new tokens: ends 18 + 4 + 1 = 23.
    B's second turn (t=36) needs 3 blocks with 1 resident: A's two tail blocks go
    out (2 swaps), B's host block comes back (1 swap in), B prefills 4 tokens:
    ends 36 + 4 + 3 = 43.  Without the host pool B recomputes its dropped 4 tokens
    instead: ends 36 + 8 = 44."""
    sess = [cp.SessionSpec(0.0, [cp.Turn(8, 0, 0, 10.0), cp.Turn(4, 0)]),
            cp.SessionSpec(1.0, [cp.Turn(8, 0, 0, 20.0), cp.Turn(4, 0)])]
    kw = dict(M=4, block_tokens=4, prefill_s_per_token=1.0, sched="fcfs", evict="lru",
              swap_s_per_block=1.0)
    r, log = cp.simulate_blocks(cp.Config(host_blocks=8, **kw), sess, [[1.0]])
    assert r.dispatch == [0, 1, 0, 1]
    assert [(d.cached_tokens, d.new_tokens, d.blocks, d.swapped_in, d.swapped_out) for d in log] == \
        [(0, 8, 2, 0, 0), (0, 8, 2, 0, 0), (8, 4, 3, 0, 1), (8, 4, 3, 1, 2)]
    assert (r.evicted_blocks, r.swapped_out_blocks, r.swapped_in_blocks, r.recomputed_tokens,
            r.prefilled_tokens, r.makespan_s) == (3, 3, 1, 0, 24, 43.0)
    r0, log0 = cp.simulate_blocks(cp.Config(host_blocks=0, **kw), sess, [[1.0]])
    assert [(d.cached_tokens, d.new_tokens) for d in log0] == [(0, 8), (0, 8), (8, 4), (4, 8)]
    assert (r0.evicted_blocks, r0.swapped_out_blocks, r0.swapped_in_blocks, r0.recomputed_tokens,
            r0.prefilled_tokens, r0.makespan_s) == (3, 0, 0, 4, 28, 44.0)


def test_offload_full_host_pool_drops_the_tail_worked_example():
    """A host pool of 1 block: an evicted block goes out while the pool has room;
    the next finds it full and is dropped together with the host-held block behind
    it, which frees the pool again; the copy of that block is then not made (nor
    charged).  A (t=0): 12 tokens (3 blocks), tool 50 s, then 4.  B (t=1, runs
    12-24): 12 tokens in a 4-block node: A's tail (position 2) goes out, A's
    position 1 is dropped and takes position 2 with it (no swap out remains).
    A's second turn (t=62) keeps position 0 (4 tokens found) and needs 3 more
    blocks: B's position 2 goes out, position 1 is dropped (freeing the pool and
    cancelling that copy), position 0 goes out (1 swap out); A recomputes 8
    context tokens."""
    sess = [cp.SessionSpec(0.0, [cp.Turn(12, 0, 0, 50.0), cp.Turn(4, 0)]),
            cp.SessionSpec(1.0, [cp.Turn(12, 0)])]
    cfg = cp.Config(M=4, block_tokens=4, prefill_s_per_token=1.0, sched="fcfs", evict="lru",
                    host_blocks=1, swap_s_per_block=1.0)
    r, log = cp.simulate_blocks(cfg, sess, [[1.0]])
    assert r.dispatch == [0, 1, 0]
    assert [(d.cached_tokens, d.new_tokens, d.swapped_in, d.swapped_out) for d in log] == \
        [(0, 12, 0, 0), (0, 12, 0, 0), (4, 12, 0, 1)]
    assert (r.evicted_blocks, r.swapped_out_blocks, r.swapped_in_blocks, r.recomputed_tokens) == (5, 1, 0, 8)
    assert r.makespan_s == 62.0 + 12 + 1


@pytest.mark.parametrize("seed", range(3))
def test_free_unbounded_offload_is_a_node_that_never_evicts(seed):
    """FCFS with an unbounded host pool and free swaps gives the dispatch order,
    times and prefill of FCFS on a node large enough never to evict: with FCFS
    the order depends only on times, and no request recomputes or pays a swap."""
    import cw_workloads as cw
    tr = cw.agent_sessions(num_sessions=10, seed=2200 + seed, max_turns=8, shared_groups=2,
                           shared_prefix_tokens=512)
    sess = _to_oracle_sessions(tr.sessions, tr.groups)
    kw = dict(block_tokens=tr.block_tokens, prefill_s_per_token=1e-4, decode_s_per_token=1e-3,
              sched="fcfs", evict="lru")
    off, _ = cp.simulate_blocks(cp.Config(M=tr.capacity_blocks, host_blocks=10 ** 9, **kw), sess,
                                tr.history, shared_tokens=tr.shared_tokens)
    big, _ = cp.simulate_blocks(cp.Config(M=10 ** 9, **kw), sess, tr.history, shared_tokens=tr.shared_tokens)
    assert off.evicted_blocks > 0 and big.evicted_blocks == 0
    assert off.dispatch == big.dispatch
    assert off.recomputed_tokens == 0 and off.prefilled_tokens == big.prefilled_tokens
    assert off.makespan_s == pytest.approx(big.makespan_s, rel=1e-12)
    assert 0 < off.swapped_in_blocks <= off.swapped_out_blocks == off.evicted_blocks


@pytest.mark.parametrize("seed", range(2))
@pytest.mark.parametrize("sched,evict", list(itertools.product(("fcfs", "prefix"),
                                                               ("lru", "predictive", "belady"))))
def test_offload_accounting(seed, sched, evict):
    """With groups: a host pool of 0 is the model without offload; with a bounded
    pool every block swapped in was swapped out before, and the log's counts add
    up to the totals; an unbounded pool never recomputes."""
    import cw_workloads as cw
    tr = cw.agent_sessions(num_sessions=10, seed=2300 + seed, max_turns=8, shared_groups=2,
                           shared_prefix_tokens=1024)
    sess = _to_oracle_sessions(tr.sessions, tr.groups)
    kw = dict(M=tr.capacity_blocks, block_tokens=tr.block_tokens, prefill_s_per_token=1e-5,
              decode_s_per_token=1e-3, sched=sched, evict=evict, n_rebuild=3, swap_s_per_block=1e-3)
    base, blog = cp.simulate_blocks(cp.Config(**kw), sess, tr.history, shared_tokens=tr.shared_tokens)
    zero, zlog = cp.simulate_blocks(cp.Config(host_blocks=0, **kw), sess, tr.history,
                                    shared_tokens=tr.shared_tokens)
    assert zero == base and zlog == blog
    for host in (40, 10 ** 9):
        r, log = cp.simulate_blocks(cp.Config(host_blocks=host, **kw), sess, tr.history,
                                    shared_tokens=tr.shared_tokens)
        assert r.swapped_in_blocks <= r.swapped_out_blocks <= r.evicted_blocks
        assert sum(d.swapped_in for d in log) == r.swapped_in_blocks
        assert sum(d.swapped_out for d in log) == r.swapped_out_blocks
        assert sum(d.new_tokens for d in log) == r.prefilled_tokens
        if host == 10 ** 9:
            # every evicted block goes out, but those no one uses again
            # (predictive and Belady know them: value +inf)
            assert r.recomputed_tokens == 0
            if evict == "lru":
                assert r.swapped_out_blocks == r.evicted_blocks
            else:
                assert r.swapped_out_blocks < r.evicted_blocks


def test_offload_skips_blocks_no_one_uses_again():
    """A (t=0) runs one 8-token turn (2 blocks) and finishes at t=8; B (t=1) needs
    3 blocks of a 4-block node after it and evicts one of A's.  Predictive and
    Belady give a finished session's blocks the value +inf: the block is dropped,
    not copied; LRU cannot tell and copies it."""
    sess = [cp.SessionSpec(0.0, [cp.Turn(8, 0)]), cp.SessionSpec(1.0, [cp.Turn(12, 0)])]
    for evict, out in (("lru", 1), ("predictive", 0), ("belady", 0)):
        cfg = cp.Config(M=4, block_tokens=4, prefill_s_per_token=1.0, sched="fcfs", evict=evict,
                        host_blocks=8, swap_s_per_block=1.0)
        r, log = cp.simulate_blocks(cfg, sess, [[1.0]])
        assert (r.evicted_blocks, r.swapped_out_blocks, r.swapped_in_blocks) == (1, out, 0), evict
        assert r.makespan_s == 8.0 + 12 + out, evict
