"""Python binding of the CacheWise host policy simulator (include/cw_policy.h).

Argument marshalling only: the simulation runs in the library's C++ code.

Sessions are given as a list of (start_s, turns) with turns a list of
(in_tokens, out_tokens, tool_type, tool_s); `history[y]` is the list of past
durations of tool type y that the predictor conditions on; `groups[s]` (or
None) the shared-prefix group of session s and `shared_tokens[g]` the tokens
group g shares.  BlockManager wraps the stateful KV block manager.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import _check, library

SCHED = {"fcfs": 0, "prefix": 1}
EVICT = {"lru": 0, "predictive": 1, "belady": 2}


class _Config(C.Structure):
    _fields_ = [("capacity_blocks", C.c_int32), ("block_tokens", C.c_int32),
                ("prefill_s_per_token", C.c_double), ("decode_s_per_token", C.c_double),
                ("sched", C.c_int32), ("evict", C.c_int32), ("rebuild_every", C.c_int32),
                ("host_blocks", C.c_int32), ("swap_s_per_block", C.c_double)]


class _Trace(C.Structure):
    _fields_ = [("num_sessions", C.c_int32), ("turn_off", C.c_void_p), ("session_start", C.c_void_p),
                ("in_tokens", C.c_void_p), ("out_tokens", C.c_void_p), ("tool", C.c_void_p),
                ("tool_s", C.c_void_p), ("num_tools", C.c_int32), ("hist_off", C.c_void_p),
                ("hist_s", C.c_void_p), ("num_groups", C.c_int32), ("session_group", C.c_void_p),
                ("group_shared_tokens", C.c_void_p)]


class _Log(C.Structure):
    _fields_ = [("capacity", C.c_int64), ("session", C.c_void_p), ("cached_tokens", C.c_void_p),
                ("new_tokens", C.c_void_p), ("table_off", C.c_void_p), ("tables", C.c_void_p),
                ("table_capacity", C.c_int64), ("written", C.c_int64), ("swapped_in", C.c_void_p),
                ("swapped_out", C.c_void_p)]


class _Swaps(C.Structure):
    _fields_ = [("out_device", C.c_void_p), ("out_host", C.c_void_p), ("in_host", C.c_void_p),
                ("in_device", C.c_void_p), ("capacity", C.c_int32), ("n_out", C.c_int32),
                ("n_in", C.c_int32)]


class _Result(C.Structure):
    _fields_ = [("makespan_s", C.c_double), ("mean_session_s", C.c_double),
                ("goodput_tok_s", C.c_double), ("requests", C.c_int64), ("faults", C.c_int64),
                ("evicted_blocks", C.c_int64), ("recomputed_tokens", C.c_int64),
                ("prefilled_tokens", C.c_int64), ("heap_rebuilds", C.c_int64),
                ("swapped_out_blocks", C.c_int64), ("swapped_in_blocks", C.c_int64)]


def _trace(sessions: Sequence[Tuple[float, Sequence[Tuple[int, int, int, float]]]],
           history: Sequence[Sequence[float]], groups=None, shared_tokens=None):
    turns = [t for _, ts in sessions for t in ts]
    arr = {
        "turn_off": np.cumsum([0] + [len(ts) for _, ts in sessions]).astype(np.int32),
        "session_start": np.asarray([s for s, _ in sessions], dtype=np.float64),
        "in_tokens": np.asarray([t[0] for t in turns], dtype=np.int32),
        "out_tokens": np.asarray([t[1] for t in turns], dtype=np.int32),
        "tool": np.asarray([t[2] for t in turns], dtype=np.int32),
        "tool_s": np.asarray([t[3] for t in turns], dtype=np.float64),
        "hist_off": np.cumsum([0] + [len(h) for h in history]).astype(np.int32),
        "hist_s": np.asarray([x for h in history for x in h], dtype=np.float64),
        "session_group": np.asarray(groups if groups is not None else [], dtype=np.int32),
        "group_shared_tokens": np.asarray(shared_tokens if shared_tokens is not None else [], dtype=np.int32),
    }
    ptr = lambda a: a.ctypes.data if a.size else None
    n_groups = len(arr["group_shared_tokens"]) if groups is not None else 0
    tr = _Trace(len(sessions), ptr(arr["turn_off"]), ptr(arr["session_start"]), ptr(arr["in_tokens"]),
                ptr(arr["out_tokens"]), ptr(arr["tool"]), ptr(arr["tool_s"]), len(history),
                ptr(arr["hist_off"]), ptr(arr["hist_s"]), n_groups,
                ptr(arr["session_group"]) if n_groups else None,
                ptr(arr["group_shared_tokens"]) if n_groups else None)
    return tr, arr  # keep the arrays alive with the struct


def simulate(sessions, history, *, capacity_blocks: int, block_tokens: int,
             prefill_s_per_token: float = 0.0, decode_s_per_token: float = 0.0,
             sched: str = "prefix", evict: str = "predictive", rebuild_every: int = 3,
             groups=None, shared_tokens=None, log: bool = False, host_blocks: int = 0,
             swap_s_per_block: float = 0.0) -> Dict:
    """Runs the simulation; with `log`, out["log"] lists per dispatch (session,
    cached_tokens, new_tokens, block table) and out["log_swaps"] its (blocks
    swapped in, blocks swapped out).  host_blocks > 0 turns on offload."""
    tr, keep = _trace(sessions, history, groups, shared_tokens)
    cfg = _Config(capacity_blocks, block_tokens, prefill_s_per_token, decode_s_per_token,
                  SCHED[sched], EVICT[evict], rebuild_every, host_blocks, swap_s_per_block)
    res = _Result()
    n_turns = int(keep["turn_off"][-1])
    if not log:
        order = np.zeros(max(n_turns, 1), dtype=np.int32)
        _check(library().cw_policy_simulate(C.byref(cfg), C.byref(tr), C.byref(res), order.ctypes.data,
                                            n_turns))
        out = {name: getattr(res, name) for name, _ in _Result._fields_}
        out["dispatch"] = order[:min(res.requests, n_turns)].tolist()
        return out
    cap = max(n_turns, 1)
    tcap = int(sum(-(-sum(t[0] + t[1] for t in ts[:j + 1]) // block_tokens)
                   for _, ts in sessions for j in range(len(ts)))) + 1
    a = {"session": np.zeros(cap, np.int32), "cached_tokens": np.zeros(cap, np.int32),
         "new_tokens": np.zeros(cap, np.int32), "table_off": np.zeros(cap + 1, np.int64),
         "tables": np.zeros(max(tcap, 1), np.int32), "swapped_in": np.zeros(cap, np.int32),
         "swapped_out": np.zeros(cap, np.int32)}
    lg = _Log(cap, a["session"].ctypes.data, a["cached_tokens"].ctypes.data, a["new_tokens"].ctypes.data,
              a["table_off"].ctypes.data, a["tables"].ctypes.data, len(a["tables"]), 0,
              a["swapped_in"].ctypes.data, a["swapped_out"].ctypes.data)
    _check(library().cw_policy_simulate_log(C.byref(cfg), C.byref(tr), C.byref(res), C.byref(lg)))
    out = {name: getattr(res, name) for name, _ in _Result._fields_}
    n = lg.written
    out["dispatch"] = a["session"][:n].tolist()
    out["log"] = [(int(a["session"][i]), int(a["cached_tokens"][i]), int(a["new_tokens"][i]),
                   a["tables"][a["table_off"][i]:a["table_off"][i + 1]].tolist()) for i in range(n)]
    out["log_swaps"] = [(int(a["swapped_in"][i]), int(a["swapped_out"][i])) for i in range(n)]
    return out


class BlockManager:
    """The KV block manager (cw_bm_*): register sessions, admit and release
    their requests, rebuild the eviction heap.  With host_blocks > 0 evicted
    blocks go to a host pool of that many blocks (offload) and requests are
    admitted with admit_swaps, which also returns the page copies to make."""

    def __init__(self, capacity_blocks: int, block_tokens: int, host_blocks: int = 0):
        self._h = C.c_void_p()
        if host_blocks:
            _check(library().cw_bm_create_with_host_pool(capacity_blocks, block_tokens, host_blocks,
                                                         C.byref(self._h)))
        else:
            _check(library().cw_bm_create(capacity_blocks, block_tokens, C.byref(self._h)))
        self.capacity_blocks, self.block_tokens = capacity_blocks, block_tokens
        self.host_blocks = host_blocks

    def close(self):
        if self._h:
            library().cw_bm_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def add_session(self, session: int, group: int = -1, shared_tokens: int = 0):
        _check(library().cw_bm_add_session(self._h, session, group, shared_tokens))

    def admit(self, session: int, context_tokens: int, input_tokens: int, output_tokens: int):
        """Returns (block table, cached prompt tokens, evicted blocks)."""
        need = -(-(context_tokens + input_tokens + output_tokens) // self.block_tokens)
        table = np.zeros(max(need, 1), dtype=np.int32)
        blocks, cached, evicted = C.c_int32(), C.c_int64(), C.c_int64()
        _check(library().cw_bm_admit(self._h, session, context_tokens, input_tokens, output_tokens,
                                     table.ctypes.data, len(table), C.byref(blocks), C.byref(cached),
                                     C.byref(evicted)))
        return table[:blocks.value].copy(), cached.value, evicted.value

    def admit_swaps(self, session: int, context_tokens: int, input_tokens: int, output_tokens: int):
        """Returns (block table, cached prompt tokens, evicted blocks, swap-outs
        [(device block, host block)], swap-ins [(host block, device block)]);
        make the swap-outs' copies, then the swap-ins', before the step."""
        need = -(-(context_tokens + input_tokens + output_tokens) // self.block_tokens)
        table = np.zeros(max(need, 1), dtype=np.int32)
        lists = [np.zeros(max(need, 1), dtype=np.int32) for _ in range(4)]
        sw = _Swaps(*(x.ctypes.data for x in lists), len(lists[0]), 0, 0)
        blocks, cached, evicted = C.c_int32(), C.c_int64(), C.c_int64()
        _check(library().cw_bm_admit_swaps(self._h, session, context_tokens, input_tokens, output_tokens,
                                           table.ctypes.data, len(table), C.byref(blocks), C.byref(cached),
                                           C.byref(evicted), C.byref(sw)))
        od, oh, ih, idv = lists
        outs = list(zip(od[:sw.n_out].tolist(), oh[:sw.n_out].tolist()))
        ins = list(zip(ih[:sw.n_in].tolist(), idv[:sw.n_in].tolist()))
        return table[:blocks.value].copy(), cached.value, evicted.value, outs, ins

    def release(self, session: int, value: float):
        _check(library().cw_bm_release(self._h, session, float(value)))

    def rebuild(self, values: Dict[int, float]):
        s = np.asarray(list(values.keys()), dtype=np.int32)
        v = np.asarray(list(values.values()), dtype=np.float64)
        _check(library().cw_bm_rebuild(self._h, s.ctypes.data if s.size else None,
                                       v.ctypes.data if v.size else None, len(s)))

    def stats(self):
        f, r = C.c_int64(), C.c_int64()
        _check(library().cw_bm_stats(self._h, C.byref(f), C.byref(r)))
        return {"free_blocks": f.value, "referenced_blocks": r.value}

    def host_stats(self):
        f, h = C.c_int64(), C.c_int64()
        _check(library().cw_bm_host_stats(self._h, C.byref(f), C.byref(h)))
        return {"free_host_blocks": f.value, "held_host_blocks": h.value}


def predict(history: Sequence[Sequence[float]], tool: int, elapsed_s: float) -> float:
    tr, keep = _trace([], history)
    v = C.c_double()
    _check(library().cw_policy_predict(C.byref(tr), tool, elapsed_s, C.byref(v)))
    return v.value
