"""Python binding of the CacheWise host policy simulator (include/cw_policy.h).

Argument marshalling only: the simulation runs in the library's C++ code.

Sessions are given as a list of (start_s, turns) with turns a list of
(in_tokens, out_tokens, tool_type, tool_s); `history[y]` is the list of past
durations of tool type y that the predictor conditions on.
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
                ("sched", C.c_int32), ("evict", C.c_int32), ("rebuild_every", C.c_int32)]


class _Trace(C.Structure):
    _fields_ = [("num_sessions", C.c_int32), ("turn_off", C.c_void_p), ("session_start", C.c_void_p),
                ("in_tokens", C.c_void_p), ("out_tokens", C.c_void_p), ("tool", C.c_void_p),
                ("tool_s", C.c_void_p), ("num_tools", C.c_int32), ("hist_off", C.c_void_p),
                ("hist_s", C.c_void_p)]


class _Result(C.Structure):
    _fields_ = [("makespan_s", C.c_double), ("mean_session_s", C.c_double),
                ("goodput_tok_s", C.c_double), ("requests", C.c_int64), ("faults", C.c_int64),
                ("evicted_blocks", C.c_int64), ("recomputed_tokens", C.c_int64),
                ("prefilled_tokens", C.c_int64), ("heap_rebuilds", C.c_int64)]


def _trace(sessions: Sequence[Tuple[float, Sequence[Tuple[int, int, int, float]]]],
           history: Sequence[Sequence[float]]):
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
    }
    ptr = lambda a: a.ctypes.data if a.size else None
    tr = _Trace(len(sessions), ptr(arr["turn_off"]), ptr(arr["session_start"]), ptr(arr["in_tokens"]),
                ptr(arr["out_tokens"]), ptr(arr["tool"]), ptr(arr["tool_s"]), len(history),
                ptr(arr["hist_off"]), ptr(arr["hist_s"]))
    return tr, arr  # keep the arrays alive with the struct


def simulate(sessions, history, *, capacity_blocks: int, block_tokens: int,
             prefill_s_per_token: float = 0.0, decode_s_per_token: float = 0.0,
             sched: str = "prefix", evict: str = "predictive", rebuild_every: int = 3) -> Dict:
    tr, keep = _trace(sessions, history)
    cfg = _Config(capacity_blocks, block_tokens, prefill_s_per_token, decode_s_per_token,
                  SCHED[sched], EVICT[evict], rebuild_every)
    res = _Result()
    n_turns = int(keep["turn_off"][-1])
    order = np.zeros(max(n_turns, 1), dtype=np.int32)
    _check(library().cw_policy_simulate(C.byref(cfg), C.byref(tr), C.byref(res), order.ctypes.data,
                                        n_turns))
    out = {name: getattr(res, name) for name, _ in _Result._fields_}
    out["dispatch"] = order[:min(res.requests, n_turns)].tolist()
    return out


def predict(history: Sequence[Sequence[float]], tool: int, elapsed_s: float) -> float:
    tr, keep = _trace([], history)
    v = C.c_double()
    _check(library().cw_policy_predict(C.byref(tr), tool, elapsed_s, C.byref(v)))
    return v.value
