"""CacheWise KV-block policy, simulated plainly -- oracle (test infrastructure).

Written from the paper's model and design: Sec. 4 (a node holds M KV blocks;
session S_i's context needs d_i blocks, k_i of which are resident, so a new
request allocates a_i = d_i - k_i blocks, evicting other sessions' blocks
when the working set would exceed M; the ideal victim is the session whose
next reuse time tau is largest), Sec. 5.1 (dispatch the queued request with
the fewest a_i), Sec. 5.2 (evict in decreasing order of the predicted
E[tau | tau > elapsed], estimated from historical tool durations), Sec. 5.3
(one priority per session, set when its blocks become unreferenced and
recomputed for all unreferenced sessions every N_rebuild engine iterations).
The baselines are FCFS dispatch and LRU eviction; Belady's rule uses the true
tau.  The readings the paper leaves open (one request at a time, eviction
from the tail of a context, service time linear in prefilled and generated
tokens, the predictor's fallback) are the ones the library states.

Plain Python with one pass over sessions per decision, no data structures
beyond lists: slow and easy to check.
"""
import math
from dataclasses import dataclass, field
from typing import List, Sequence

INF = math.inf


@dataclass
class Turn:
    in_tokens: int
    out_tokens: int
    tool: int = 0          # type of the tool call after this turn
    tool_s: float = 0.0    # its true duration


@dataclass
class SessionSpec:
    start: float
    turns: List[Turn]
    group: int = -1        # shared-prefix group (-1: none)


@dataclass
class Config:
    M: int                     # capacity in blocks
    block_tokens: int
    prefill_s_per_token: float = 0.0
    decode_s_per_token: float = 0.0
    sched: str = "prefix"      # "fcfs" | "prefix"
    evict: str = "predictive"  # "lru" | "predictive" | "belady"
    n_rebuild: int = 3
    host_blocks: int = 0       # offload: blocks of the host pool evicted blocks go to (0: none)
    swap_s_per_block: float = 0.0  # engine time of one block's transfer either way


@dataclass
class Result:
    makespan_s: float = 0.0
    mean_session_s: float = 0.0
    goodput_tok_s: float = 0.0
    requests: int = 0
    faults: int = 0
    evicted_blocks: int = 0
    recomputed_tokens: int = 0
    prefilled_tokens: int = 0
    heap_rebuilds: int = 0
    swapped_out_blocks: int = 0
    swapped_in_blocks: int = 0
    dispatch: List[int] = field(default_factory=list)


def predict_remaining(history: Sequence[float], elapsed: float) -> float:
    """E[tau - elapsed | tau > elapsed] from samples; `elapsed` if no sample exceeds it."""
    rest = [x - elapsed for x in history if x > elapsed]
    return sum(rest) / len(rest) if rest else elapsed


def _blocks(tokens: int, block_tokens: int) -> int:
    return -(-tokens // block_tokens)


def simulate(cfg: Config, sessions: Sequence[SessionSpec], history: Sequence[Sequence[float]]) -> Result:
    B = cfg.block_tokens
    n = len(sessions)
    nxt = [0] * n                 # next turn of each session
    ctx = [0] * n                 # context tokens
    k = [0] * n                   # resident leading blocks (k_i)
    state = ["wait"] * n          # wait | queued | running | done
    arrival = [s.start for s in sessions]
    last_use = [0.0] * n
    tool_start = [0.0] * n
    tool = [0] * n
    prio = [0.0] * n
    done_at = [0.0] * n
    for i, s in enumerate(sessions):
        if not s.turns:
            state[i], done_at[i], prio[i] = "done", s.start, INF
    r = Result()
    t = 0.0
    running, run_end = -1, 0.0

    def need(i):  # d_i of session i's pending turn
        tr = sessions[i].turns[nxt[i]]
        return _blocks(ctx[i] + tr.in_tokens + tr.out_tokens, B)

    def tau_true(j):
        if state[j] == "done":
            return INF
        if state[j] == "queued":
            return 0.0
        return max(0.0, arrival[j] - t)

    while True:
        for i in range(n):
            if state[i] == "wait" and arrival[i] <= t:
                state[i] = "queued"
        if running < 0:
            queued = [i for i in range(n) if state[i] == "queued"]
            if queued:
                if cfg.sched == "prefix":   # fewest new blocks a_i, then earliest arrival
                    i = min(queued, key=lambda q: (need(q) - k[q], arrival[q], q))
                else:                       # first come, first served
                    i = min(queued, key=lambda q: (arrival[q], q))
                # engine iteration: the eviction heap is rebuilt every N_rebuild of them
                r.requests += 1
                if cfg.evict == "predictive" and r.requests % cfg.n_rebuild == 0:
                    for j in range(n):
                        if state[j] == "done":
                            prio[j] = INF
                        elif state[j] == "queued":
                            prio[j] = 0.0
                        elif state[j] == "wait":
                            prio[j] = predict_remaining(history[tool[j]], t - tool_start[j])
                    r.heap_rebuilds += 1
                tr = sessions[i].turns[nxt[i]]
                d = need(i)
                a = d - k[i]
                if k[i] < _blocks(ctx[i], B):
                    r.faults += 1
                free = cfg.M - sum(k)
                while free < a:
                    cands = [j for j in range(n) if j != i and k[j] > 0]
                    if cfg.evict == "lru":
                        v = min(cands, key=lambda j: (last_use[j], j))
                    elif cfg.evict == "predictive":
                        v = min(cands, key=lambda j: (-prio[j], j))
                    else:
                        v = min(cands, key=lambda j: (-tau_true(j), j))
                    take = min(k[v], a - free)   # from the tail of its context
                    k[v] -= take
                    free += take
                    r.evicted_blocks += take
                recompute = max(0, ctx[i] - k[i] * B)
                r.recomputed_tokens += recompute
                r.prefilled_tokens += recompute + tr.in_tokens
                k[i] = d
                state[i] = "running"
                running = i
                run_end = t + (cfg.prefill_s_per_token * (recompute + tr.in_tokens)
                               + cfg.decode_s_per_token * tr.out_tokens)
                r.dispatch.append(i)
                continue
        nexts = [arrival[i] for i in range(n) if state[i] == "wait"]
        if running >= 0:
            nexts.append(run_end)
        if not nexts:
            break
        t = max(t, min(nexts))
        if running >= 0 and run_end <= t:
            i = running
            tr = sessions[i].turns[nxt[i]]
            ctx[i] += tr.in_tokens + tr.out_tokens
            last_use[i] = t
            nxt[i] += 1
            if nxt[i] == len(sessions[i].turns):
                state[i], done_at[i], prio[i] = "done", t, INF
            else:
                state[i] = "wait"
                tool[i], tool_start[i] = tr.tool, t
                arrival[i] = t + tr.tool_s
                prio[i] = predict_remaining(history[tr.tool], 0.0)
            running = -1
    r.makespan_s = max(done_at) if n else 0.0
    spans = [done_at[i] - sessions[i].start for i in range(n) if sessions[i].turns]
    r.mean_session_s = sum(spans) / len(spans) if spans else 0.0
    total = sum(tr.in_tokens + tr.out_tokens for s in sessions for tr in s.turns)
    r.goodput_tok_s = total / r.makespan_s if r.makespan_s > 0 else 0.0
    return r


# ---------------------------------------------------------------------------
# The same model at block granularity, with prefix blocks shared across sessions.
#
# Readings (the paper's engine keeps prefix blocks cached by content and shares
# them; its formal model leaves these open):
#  * group g shares the first shared_tokens[g] tokens of each member's context;
#    the whole blocks among them (G_g = shared_tokens // B) are one copy, the
#    rest of a member's context is private.  A member's first turn's input
#    starts with the shared tokens.
#  * a request's resident run k is the leading run of its blocks that are
#    resident (shared blocks count even before the session's first request);
#    the tokens whose K/V it finds resident are min(k B, max(context, G B)):
#    its own context, or the shared prefix before its first request.  It
#    prefills the rest of context + input; `recomputed` counts the tokens of its
#    own context among them.
#  * eviction takes one block at a time, the largest key first.  A private
#    block of session s at position p has key (v_s, -s, p) with v_s the
#    policy's value (predictive: priority; LRU: -last use; Belady: true time
#    to next use).  A shared block's v is the value of the sharer that needs it
#    soonest (smallest priority or time to next use, latest last use) over the
#    sessions attached to the group, its s the largest id among the sharers with
#    that value.  So every sharer's private blocks (positions after it) leave
#    first: resident blocks stay a leading run of every context.  The
#    dispatching session's resident run is never a candidate.
# Offload (the paper's Sec. 6.4 configuration: evicted blocks go to CPU memory
# and are swapped back when the session resumes), with host_blocks > 0:
#  * an evicted block goes to the host pool while it has a free block (a swap
#    out); the host-held blocks of a context follow its resident run.  When the
#    pool is full the block is dropped instead, and with it the owner's host-held
#    blocks (past it, so no longer part of a leading run); a dropped shared block
#    also drops the sharers' host-held private blocks.  A block whose value is
#    +inf (predictive: its session has finished; Belady: never used again) is
#    dropped the same way rather than copied.  A copy to the host pool
#    that a drop in the same admission discards is not made (its data would
#    never be read) and is not counted.
#  * a request first swaps its host-held blocks back in (shared ones, then its
#    private ones once the shared run is complete), after the evictions that make
#    room for them; they count as found (no prefill).  Every swap, out or in,
#    costs swap_s_per_block of engine time.
# With no groups this is exactly simulate() above (pinned by a test), and with a
# host pool of 0 blocks exactly the model without offload.
# ---------------------------------------------------------------------------

@dataclass
class Dispatch:
    session: int
    cached_tokens: int     # prompt tokens whose K/V are resident (attention prefix)
    new_tokens: int        # tokens prefilled (context + input - cached)
    blocks: int            # blocks of the request (context + input + output)
    swapped_in: int = 0    # of them, blocks brought back from the host pool
    swapped_out: int = 0   # blocks of other sessions moved to the host pool to make room


def simulate_blocks(cfg: Config, sessions: Sequence[SessionSpec], history: Sequence[Sequence[float]],
                    shared_tokens: Sequence[int] = ()) -> tuple:
    """Returns (Result, [Dispatch])."""
    B = cfg.block_tokens
    n = len(sessions)
    G = [shared_tokens[s.group] // B if s.group >= 0 else 0 for s in sessions]
    nxt = [0] * n
    ctx = [0] * n
    state = ["wait"] * n
    arrival = [s.start for s in sessions]
    last_use = [0.0] * n
    tool_start = [0.0] * n
    tool = [0] * n
    prio = [0.0] * n
    done_at = [0.0] * n
    attached = [False] * n
    res_private = [0] * n               # resident private blocks (positions G .. G + r - 1)
    res_shared = [0] * len(shared_tokens)  # resident shared blocks of each group (leading)
    host_private = [0] * n              # host-held private blocks, following the resident ones
    host_shared = [0] * len(shared_tokens)
    for i, s in enumerate(sessions):
        if not s.turns:
            state[i], done_at[i], prio[i] = "done", s.start, INF
    r = Result()
    log = []
    t = 0.0
    running, run_end = -1, 0.0

    def resident_run(i):
        g = sessions[i].group
        if g < 0:
            return res_private[i]
        if res_shared[g] < G[i]:
            return res_shared[g]
        return G[i] + res_private[i]

    def need(i):
        tr = sessions[i].turns[nxt[i]]
        return _blocks(ctx[i] + tr.in_tokens + tr.out_tokens, B)

    def tau_true(j):
        if state[j] == "done":
            return INF
        if state[j] == "queued":
            return 0.0
        return max(0.0, arrival[j] - t)

    def value(j):
        if cfg.evict == "lru":
            return -last_use[j]
        if cfg.evict == "predictive":
            return prio[j]
        return tau_true(j)

    def victim(i):
        """Largest key among the tail blocks of other sessions' private runs and of
        the groups' shared runs: ('p', session, value) or ('g', group, value)."""
        best, best_key = None, None
        for j in range(n):
            if j != i and res_private[j] > 0:
                key = (value(j), -j, G[j] + res_private[j] - 1)
                if best_key is None or key > best_key:
                    best, best_key = ("p", j, key[0]), key
        for g in range(len(shared_tokens)):
            if res_shared[g] == 0:
                continue
            if sessions[i].group == g and res_shared[g] <= resident_run(i):
                continue  # every resident shared block is in the dispatching run
            sharers = [j for j in range(n) if sessions[j].group == g and attached[j]]
            v = min(value(j) for j in sharers)
            jsel = max(j for j in sharers if value(j) == v)
            key = (v, -jsel, res_shared[g] - 1)
            if best_key is None or key > best_key:
                best, best_key = ("g", g, v), key
        return best

    while True:
        for i in range(n):
            if state[i] == "wait" and arrival[i] <= t:
                state[i] = "queued"
        if running < 0:
            queued = [i for i in range(n) if state[i] == "queued"]
            if queued:
                if cfg.sched == "prefix":
                    i = min(queued, key=lambda q: (need(q) - resident_run(q), arrival[q], q))
                else:
                    i = min(queued, key=lambda q: (arrival[q], q))
                r.requests += 1
                if cfg.evict == "predictive" and r.requests % cfg.n_rebuild == 0:
                    for j in range(n):
                        if state[j] == "done":
                            prio[j] = INF
                        elif state[j] == "queued":
                            prio[j] = 0.0
                        elif state[j] == "wait":
                            prio[j] = predict_remaining(history[tool[j]], t - tool_start[j])
                    r.heap_rebuilds += 1
                tr = sessions[i].turns[nxt[i]]
                d = need(i)
                k = resident_run(i)
                if k < _blocks(ctx[i], B):
                    r.faults += 1
                a = d - k
                free = cfg.M - sum(res_private) - sum(res_shared)
                swapped_out = 0
                # copies to the host pool made by this admission and still held
                new_private = [0] * n
                new_shared = [0] * len(shared_tokens)
                while free < a:
                    kind, x, v = victim(i)
                    # a block no one will use again (value +inf) is not worth a copy
                    to_host = v != INF and sum(host_private) + sum(host_shared) < cfg.host_blocks
                    if kind == "p":
                        res_private[x] -= 1
                        if to_host:
                            host_private[x] += 1
                            new_private[x] += 1
                        else:
                            host_private[x] = 0
                            swapped_out -= new_private[x]
                            new_private[x] = 0
                    else:
                        res_shared[x] -= 1
                        # the key order keeps every sharer's private blocks out first
                        assert all(res_private[j] == 0 for j in range(n) if sessions[j].group == x)
                        if to_host:
                            host_shared[x] += 1
                            new_shared[x] += 1
                        else:
                            host_shared[x] = 0
                            swapped_out -= new_shared[x]
                            new_shared[x] = 0
                            for j in range(n):
                                if sessions[j].group == x:
                                    host_private[j] = 0
                                    swapped_out -= new_private[j]
                                    new_private[j] = 0
                    swapped_out += 1 if to_host else 0
                    free += 1
                    r.evicted_blocks += 1
                # swap the host-held run back in, in position order
                swapped_in = 0
                g = sessions[i].group
                if g >= 0 and res_shared[g] < G[i]:
                    take = host_shared[g]
                    host_shared[g] -= take
                    res_shared[g] += take
                    swapped_in += take
                if g < 0 or res_shared[g] >= G[i]:
                    take = host_private[i]
                    host_private[i] = 0
                    res_private[i] += take
                    swapped_in += take
                r.swapped_out_blocks += swapped_out
                r.swapped_in_blocks += swapped_in
                k = resident_run(i)
                known = max(ctx[i], G[i] * B)
                hit = min(k * B, known)
                recompute = max(0, ctx[i] - hit)
                r.recomputed_tokens += recompute
                r.prefilled_tokens += ctx[i] + tr.in_tokens - hit
                log.append(Dispatch(i, hit, ctx[i] + tr.in_tokens - hit, d, swapped_in, swapped_out))
                g = sessions[i].group
                if g >= 0:
                    res_shared[g] = max(res_shared[g], min(d, G[i]))
                res_private[i] = max(0, d - G[i])
                attached[i] = True
                state[i] = "running"
                running = i
                run_end = t + (cfg.prefill_s_per_token * (ctx[i] + tr.in_tokens - hit)
                               + cfg.decode_s_per_token * tr.out_tokens
                               + cfg.swap_s_per_block * (swapped_in + swapped_out))
                r.dispatch.append(i)
                continue
        nexts = [arrival[i] for i in range(n) if state[i] == "wait"]
        if running >= 0:
            nexts.append(run_end)
        if not nexts:
            break
        t = max(t, min(nexts))
        if running >= 0 and run_end <= t:
            i = running
            tr = sessions[i].turns[nxt[i]]
            ctx[i] += tr.in_tokens + tr.out_tokens
            last_use[i] = t
            nxt[i] += 1
            if nxt[i] == len(sessions[i].turns):
                state[i], done_at[i], prio[i] = "done", t, INF
            else:
                state[i] = "wait"
                tool[i], tool_start[i] = tr.tool, t
                arrival[i] = t + tr.tool_s
                prio[i] = predict_remaining(history[tr.tool], 0.0)
            running = -1
    r.makespan_s = max(done_at) if n else 0.0
    spans = [done_at[i] - sessions[i].start for i in range(n) if sessions[i].turns]
    r.mean_session_s = sum(spans) / len(spans) if spans else 0.0
    total = sum(tr.in_tokens + tr.out_tokens for s in sessions for tr in s.turns)
    r.goodput_tok_s = total / r.makespan_s if r.makespan_s > 0 else 0.0
    return r, log
