"""Compares the KV-block policies on seeded agent sessions (host-only).

    python -m paper_2606_16824_amd.policy_bench [--sessions 32] [--turns 24] [--seed 2000]
        [--host-fraction 1.0]

Prints one JSON object: per (scheduler, eviction) pair the simulator's
counters and times, and its own run time (the scheduling overhead); with a
host pool (--host-fraction of the device blocks), the same pairs with offload
(CacheWise Sec. 6.4), a swap costing one KV block of an 8B-class model (32
layers x 8 kv heads x 128 dims x K and V in bf16: 128 KiB per token) over the
host link at the rate the page-swap kernel reaches (54 GB/s).
"""
from __future__ import annotations

import argparse
import json
import time

from . import policy

PAIRS = (("fcfs", "lru"), ("prefix", "lru"), ("prefix", "predictive"), ("prefix", "belady"),
         ("fcfs", "predictive"))
KV_BYTES_PER_TOKEN = 32 * 8 * 128 * 2 * 2
SWAP_BYTES_PER_S = 54e9


def run(num_sessions: int = 32, max_turns: int = 24, seed: int = 2000,
        capacity_fraction: float = 0.4, shared_groups: int = 0, shared_prefix_tokens: int = 0,
        host_fraction: float = 0.0) -> dict:
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
    host_blocks = int(host_fraction * tr.capacity_blocks)
    swap_s = tr.block_tokens * KV_BYTES_PER_TOKEN / SWAP_BYTES_PER_S
    if host_blocks:
        out["offload"] = {"host_blocks": host_blocks, "swap_us_per_block": round(swap_s * 1e6, 2),
                          "recompute_us_per_block": round(tr.block_tokens * tr.prefill_s_per_token * 1e6, 2),
                          "policies": {}}
    for sched, evict in PAIRS:
        for host in ((0, host_blocks) if host_blocks else (0,)):
            t0 = time.perf_counter()
            r = policy.simulate(tr.sessions, tr.history, capacity_blocks=tr.capacity_blocks,
                                block_tokens=tr.block_tokens, prefill_s_per_token=tr.prefill_s_per_token,
                                decode_s_per_token=tr.decode_s_per_token, sched=sched, evict=evict,
                                rebuild_every=3, groups=tr.groups, shared_tokens=tr.shared_tokens,
                                host_blocks=host, swap_s_per_block=swap_s if host else 0.0)
            dt = time.perf_counter() - t0
            row = {
                "mean_session_s": round(r["mean_session_s"], 3), "makespan_s": round(r["makespan_s"], 3),
                "goodput_tok_s": round(r["goodput_tok_s"], 1), "evicted_blocks": r["evicted_blocks"],
                "recomputed_tokens": r["recomputed_tokens"], "prefilled_tokens": r["prefilled_tokens"],
                "faults": r["faults"],
                "sim_us_per_request": round(dt / max(1, r["requests"]) * 1e6, 2)}
            if host:
                row["swapped_out_blocks"] = r["swapped_out_blocks"]
                row["swapped_in_blocks"] = r["swapped_in_blocks"]
                out["offload"]["policies"][f"{sched}+{evict}"] = row
            else:
                out["policies"][f"{sched}+{evict}"] = row
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--sessions", type=int, default=32)
    ap.add_argument("--turns", type=int, default=24)
    ap.add_argument("--seed", type=int, default=2000)
    ap.add_argument("--capacity-fraction", type=float, default=0.4)
    ap.add_argument("--shared-groups", type=int, default=0)
    ap.add_argument("--shared-prefix-tokens", type=int, default=0)
    ap.add_argument("--host-fraction", type=float, default=0.0,
                    help="host pool size as a fraction of the device blocks (0: no offload)")
    a = ap.parse_args()
    print(json.dumps(run(a.sessions, a.turns, a.seed, a.capacity_fraction, a.shared_groups,
                         a.shared_prefix_tokens, a.host_fraction), indent=1))


if __name__ == "__main__":
    main()
