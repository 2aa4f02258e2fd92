"""Compares the KV-block policies on seeded agent sessions (host-only).

    python -m paper_2606_16824_amd.policy_bench [--sessions 32] [--turns 24] [--seed 2000]

Prints one JSON object: per (scheduler, eviction) pair the simulator's
counters and times, and its own run time (the scheduling overhead).
"""
from __future__ import annotations

import argparse
import json
import time

from . import policy

PAIRS = (("fcfs", "lru"), ("prefix", "lru"), ("prefix", "predictive"), ("prefix", "belady"),
         ("fcfs", "predictive"))


def run(num_sessions: int = 32, max_turns: int = 24, seed: int = 2000,
        capacity_fraction: float = 0.4, shared_groups: int = 0, shared_prefix_tokens: int = 0) -> dict:
    import cw_workloads as cw  # the seeded input generator (repository root)

    tr = cw.agent_sessions(num_sessions=num_sessions, seed=seed, max_turns=max_turns,
                           capacity_fraction=capacity_fraction, shared_groups=shared_groups,
                           shared_prefix_tokens=shared_prefix_tokens)
    turns = sum(len(t) for _, t in tr.sessions)
    out = {"workload": f"{num_sessions} synthetic agent sessions ({turns} turns, seed {seed}), "
                       f"{tr.capacity_blocks} blocks of {tr.block_tokens} tokens "
                       f"({capacity_fraction:.0%} of the final working set)"
                       + (f", {shared_groups} groups sharing a {shared_prefix_tokens}-token prefix"
                          if shared_groups else ""),
           "policies": {}}
    for sched, evict in PAIRS:
        t0 = time.perf_counter()
        r = policy.simulate(tr.sessions, tr.history, capacity_blocks=tr.capacity_blocks,
                            block_tokens=tr.block_tokens, prefill_s_per_token=tr.prefill_s_per_token,
                            decode_s_per_token=tr.decode_s_per_token, sched=sched, evict=evict,
                            rebuild_every=3, groups=tr.groups, shared_tokens=tr.shared_tokens)
        dt = time.perf_counter() - t0
        out["policies"][f"{sched}+{evict}"] = {
            "mean_session_s": round(r["mean_session_s"], 3), "makespan_s": round(r["makespan_s"], 3),
            "goodput_tok_s": round(r["goodput_tok_s"], 1), "evicted_blocks": r["evicted_blocks"],
            "recomputed_tokens": r["recomputed_tokens"], "prefilled_tokens": r["prefilled_tokens"],
            "faults": r["faults"],
            "sim_us_per_request": round(dt / max(1, r["requests"]) * 1e6, 2)}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--sessions", type=int, default=32)
    ap.add_argument("--turns", type=int, default=24)
    ap.add_argument("--seed", type=int, default=2000)
    ap.add_argument("--capacity-fraction", type=float, default=0.4)
    ap.add_argument("--shared-groups", type=int, default=0)
    ap.add_argument("--shared-prefix-tokens", type=int, default=0)
    a = ap.parse_args()
    print(json.dumps(run(a.sessions, a.turns, a.seed, a.capacity_fraction, a.shared_groups,
                         a.shared_prefix_tokens), indent=1))


if __name__ == "__main__":
    main()
