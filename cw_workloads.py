"""Seeded synthetic workloads for prefix-cached paged extend attention.

This module only draws inputs: sequence lengths, the page pool, the block
table, queries and new keys/values.  It contains none of the attention
arithmetic, and it is shared by the GPU path's tests/benchmark and by the
CPU oracle's tests (neither side imports the other).

The paper (CacheWise, Sec. 2 and Sec. 3) describes coding-agent sessions whose
every turn reuses and extends a long cached prefix held in fixed-size KV
blocks; it ships no dataset here, so the five workloads below stand in for its
traces with the shapes and length mixes named in the design notes:

  tiny     1 seq, prefix 256, suffix 64, 4q/1kv heads, D=64,  P=16, 64-page pool
  turn     1 seq, prefix 16384, suffix 1024, 32q/8kv, D=128, P=16, 4096-page pool
  batch16  16 seqs sharing an 8192-token prefix, prefix ~ lognormal(median 20k,
           sigma 0.6, clipped 4k..64k, at least 8192), suffix ~ U[200,4000]
  long     1 seq, prefix 131072, suffix 8192, 64q/8kv, D=128, P=64, 4096 pages
  mixed    64 seqs, seeded shuffle of 48 decodes (suffix 1, prefix U[2k,32k])
           and 16 extends (suffix U[256,2048], prefix U[8k,32k]), fp8-e4m3fn
           pool with per-(page, kv-head) scales U(0.01, 0.1)

Seeds: workload ``i`` of the list above uses seed ``1000 + i``.  Lengths come
from ``default_rng(seed)``; the page permutation, q, k_new, v_new, pool K,
pool V and the fp8 scales each come from their own child stream of
``SeedSequence(seed)`` (spawned in that order), and bulk tensors are drawn in
fixed row chunks from grandchild streams, so several threads give the same
bits as one.

Bulk values are N(0,1) float32 rounded to bf16 (round-to-nearest-even, done by
torch's dtype cast).  Pool slots that hold no prefix token (the tail of the
last prefix page, suffix pages, unused pages) hold a NaN sentinel so that any
read of them poisons the output: bf16 0x7FC0, fp8 0x7F.  For the fp8 pool the
codes are torch's float8_e4m3fn cast of clamp(x / s, -448, 448).
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np
import torch

BF16_NAN_BITS = 0x7FC0
FP8_NAN_CODE = 0x7F
BT_UNUSED = np.iinfo(np.int32).max  # block-table entries past a sequence

CONFIG_NAMES = ("tiny", "turn", "batch16", "long", "mixed")
# decode-only workloads (every suffix length 1): the 48 decodes of the mixed step
# with its fp8 pool, the same lengths with a bf16 pool, and one 131072-token decode
DECODE_NAMES = ("decode", "decode_bf16", "decode_long")
# chunked prefill as a serving engine schedules it (the paper serves with prefill
# chunks of at most 512 tokens, co-scheduled with decodes)
EXTRA_NAMES = ("chunked",)


@dataclasses.dataclass
class WorkloadSpec:
    """Shapes and lengths of one attention call (no tensor data)."""

    name: str
    prefix_lens: np.ndarray  # int32 [B]
    suffix_lens: np.ndarray  # int32 [B]
    num_kv_heads: int
    gqa_group: int
    head_dim: int
    page_size: int
    num_pages: int
    kv_dtype: str = "bf16"  # "bf16" or "fp8"
    shared_prefix_tokens: int = 0  # leading tokens whose pages all sequences share
    seed: int = 0

    @property
    def num_seqs(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def num_q_heads(self) -> int:
        return self.num_kv_heads * self.gqa_group

    @property
    def total_new_tokens(self) -> int:
        return int(self.suffix_lens.sum())

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def pages_needed(self) -> np.ndarray:
        p = self.page_size
        return (self.prefix_lens.astype(np.int64) + self.suffix_lens + p - 1) // p

    def attention_pairs(self) -> int:
        """Unmasked (query, key) pairs per query head."""
        lp = self.prefix_lens.astype(np.int64)
        ls = self.suffix_lens.astype(np.int64)
        return int((ls * lp + ls * (ls + 1) // 2).sum())

    def flops(self) -> float:
        """Algorithmic FLOPs: 2*D for Q.K^T plus 2*D for P.V per unmasked pair."""
        return 4.0 * self.head_dim * self.num_q_heads * self.attention_pairs()


@dataclasses.dataclass
class Workload:
    """A spec plus its CPU tensors (bf16 as torch.bfloat16, fp8 as uint8 codes)."""

    spec: WorkloadSpec
    q: torch.Tensor  # bf16 [T, Hq, D]
    k_new: torch.Tensor  # bf16 [T, Hkv, D]
    v_new: torch.Tensor  # bf16 [T, Hkv, D]
    k_pool: torch.Tensor  # bf16 or uint8 [NP, Hkv, P, D]
    v_pool: torch.Tensor
    k_scale: Optional[torch.Tensor]  # fp32 [NP, Hkv] (fp8 only)
    v_scale: Optional[torch.Tensor]
    block_table: torch.Tensor  # int32 [B, bt_stride]

    @property
    def prefix_lens(self) -> np.ndarray:
        return self.spec.prefix_lens

    @property
    def suffix_lens(self) -> np.ndarray:
        return self.spec.suffix_lens

    def np_bits(self, t: torch.Tensor) -> np.ndarray:
        """Raw storage bits of a bf16 tensor as uint16, of a fp8 pool as uint8."""
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()


# ----------------------------------------------------------------------------
# lengths


def _pool_size(pages_required: int) -> int:
    """1.25 x the pages a workload needs, rounded up to a multiple of 64."""
    n = int(math.ceil(1.25 * pages_required))
    return ((n + 63) // 64) * 64


def spec_for(name: str, seed: Optional[int] = None) -> WorkloadSpec:
    """Draw the lengths of one of the named workloads."""
    if name in DECODE_NAMES:
        return _decode_spec(name, seed)
    if name == "chunked":
        return _chunked_spec(seed)
    idx = CONFIG_NAMES.index(name)
    seed = 1000 + idx if seed is None else seed
    rng = np.random.default_rng(seed)
    i32 = lambda v: np.asarray(v, dtype=np.int32)
    if name == "tiny":
        return WorkloadSpec(name, i32([256]), i32([64]), 1, 4, 64, 16, 64, seed=seed)
    if name == "turn":
        return WorkloadSpec(name, i32([16384]), i32([1024]), 8, 4, 128, 16, 4096, seed=seed)
    if name == "long":
        return WorkloadSpec(name, i32([131072]), i32([8192]), 8, 8, 128, 64, 4096, seed=seed)
    if name == "batch16":
        b, shared, p = 16, 8192, 16
        lp = np.rint(rng.lognormal(math.log(20000.0), 0.6, size=b))
        lp = np.maximum(np.clip(lp, 4096, 65536), shared).astype(np.int32)
        ls = rng.integers(200, 4000 + 1, size=b).astype(np.int32)
        spec = WorkloadSpec(name, lp, ls, 8, 4, 128, p, 0, shared_prefix_tokens=shared, seed=seed)
        need = shared // p + int((spec.pages_needed() - shared // p).sum())
        spec.num_pages = _pool_size(need)
        return spec
    if name == "mixed":
        kinds = np.array([0] * 48 + [1] * 16)
        rng.shuffle(kinds)
        lp = np.where(kinds == 0, rng.integers(2048, 32768 + 1, size=64),
                      rng.integers(8192, 32768 + 1, size=64)).astype(np.int32)
        ls = np.where(kinds == 0, 1, rng.integers(256, 2048 + 1, size=64)).astype(np.int32)
        spec = WorkloadSpec(name, lp, ls, 8, 4, 128, 16, 0, kv_dtype="fp8", seed=seed)
        spec.num_pages = _pool_size(int(spec.pages_needed().sum()))
        return spec
    raise ValueError(name)


def _chunked_spec(seed: Optional[int]) -> WorkloadSpec:
    """One step of chunked prefill: 32 sequences each extending a cached prefix
    U[8192, 32768] by a chunk of U[128, 512] tokens, and 32 decodes (prefix
    U[2048, 32768]), in a seeded order; 32q/8kv, D = 128, P = 16, bf16 pool."""
    seed = 1008 if seed is None else seed
    rng = np.random.default_rng(seed)
    kinds = np.array([0] * 32 + [1] * 32)
    rng.shuffle(kinds)
    lp = np.where(kinds == 0, rng.integers(2048, 32768 + 1, size=64),
                  rng.integers(8192, 32768 + 1, size=64)).astype(np.int32)
    ls = np.where(kinds == 0, 1, rng.integers(128, 512 + 1, size=64)).astype(np.int32)
    spec = WorkloadSpec("chunked", lp, ls, 8, 4, 128, 16, 0, seed=seed)
    spec.num_pages = _pool_size(int(spec.pages_needed().sum()))
    return spec


def _decode_spec(name: str, seed: Optional[int]) -> WorkloadSpec:
    if name == "decode_long":
        seed = 1007 if seed is None else seed
        return WorkloadSpec(name, np.asarray([131072], np.int32), np.asarray([1], np.int32), 8, 8,
                            128, 64, 4096, seed=seed)
    mixed = spec_for("mixed")
    dec = decode_subset(mixed)
    lp = mixed.prefix_lens[dec].astype(np.int32)
    seed = (1005 if name == "decode" else 1006) if seed is None else seed
    spec = WorkloadSpec(name, lp, np.ones_like(lp), 8, 4, 128, 16, 0,
                        kv_dtype="fp8" if name == "decode" else "bf16", seed=seed)
    spec.num_pages = _pool_size(int(spec.pages_needed().sum()))
    return spec


def decode_bytes(spec: WorkloadSpec) -> int:
    """Algorithmic HBM bytes of one decode call: every cached K/V element once, the
    fp8 scales and block-table entries of the prefix pages, q/out and the new K/V."""
    lp = spec.prefix_lens.astype(np.int64)
    pages = (lp + spec.page_size - 1) // spec.page_size
    elem = 1 if spec.kv_dtype == "fp8" else 2
    hkv, d = spec.num_kv_heads, spec.head_dim
    kv = 2 * lp * hkv * d * elem
    scales = 2 * pages * hkv * 4 if spec.kv_dtype == "fp8" else 0
    per_seq = kv + scales + pages * 4 + 2 * spec.num_q_heads * d * 2 + 2 * hkv * d * 2
    return int(per_seq.sum())


def custom_spec(prefix_lens, suffix_lens, *, num_kv_heads=1, gqa_group=1, head_dim=64,
                page_size=16, kv_dtype="bf16", shared_prefix_tokens=0, seed=0,
                num_pages=None, name="custom") -> WorkloadSpec:
    """A spec with explicit lengths (edge cases, parity sweeps)."""
    lp = np.asarray(prefix_lens, dtype=np.int32).reshape(-1)
    ls = np.asarray(suffix_lens, dtype=np.int32).reshape(-1)
    spec = WorkloadSpec(name, lp, ls, num_kv_heads, gqa_group, head_dim, page_size, 0,
                        kv_dtype=kv_dtype, shared_prefix_tokens=shared_prefix_tokens, seed=seed)
    sp = shared_prefix_tokens // page_size
    need = sp + int(np.maximum(spec.pages_needed() - sp, 0).sum())
    spec.num_pages = int(num_pages) if num_pages is not None else _pool_size(max(need, 1))
    return spec


def decode_subset(spec: WorkloadSpec) -> np.ndarray:
    """Indices of the sequences with a one-token suffix."""
    return np.nonzero(spec.suffix_lens == 1)[0]


# ----------------------------------------------------------------------------
# tensors


def _normal_bf16(seed_seq: np.random.SeedSequence, shape, chunk_rows: int = 1 << 14,
                 threads: int = 8) -> torch.Tensor:
    """N(0,1) fp32 rounded to bf16, drawn in fixed row chunks from child streams."""
    rows = int(shape[0])
    inner = int(np.prod(shape[1:])) if len(shape) > 1 else 1
    out = torch.empty((rows, inner), dtype=torch.bfloat16)
    n_chunks = max(1, (rows + chunk_rows - 1) // chunk_rows)
    children = seed_seq.spawn(n_chunks)

    def work(c):
        r0, r1 = c * chunk_rows, min(rows, (c + 1) * chunk_rows)
        g = np.random.default_rng(children[c])
        x = g.standard_normal((r1 - r0, inner), dtype=np.float32)
        out[r0:r1] = torch.from_numpy(x).to(torch.bfloat16)

    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(work, range(n_chunks)))
    return out.view(*shape)


def _normal_fp8_codes(seed_seq, shape, scales: torch.Tensor, chunk_rows: int = 1 << 12,
                      threads: int = 8) -> torch.Tensor:
    """fp8-e4m3fn codes of N(0,1)/scale (scale per leading row and head), clamped."""
    rows, heads = int(shape[0]), int(shape[1])
    inner = int(np.prod(shape[2:]))
    out = torch.empty((rows, heads, inner), dtype=torch.uint8)
    n_chunks = max(1, (rows + chunk_rows - 1) // chunk_rows)
    children = seed_seq.spawn(n_chunks)

    def work(c):
        r0, r1 = c * chunk_rows, min(rows, (c + 1) * chunk_rows)
        g = np.random.default_rng(children[c])
        x = torch.from_numpy(g.standard_normal((r1 - r0, heads, inner), dtype=np.float32))
        x = (x / scales[r0:r1, :, None]).clamp_(-448.0, 448.0)
        out[r0:r1] = x.to(torch.float8_e4m3fn).view(torch.uint8)

    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(work, range(n_chunks)))
    return out.view(*shape)


def build_block_table(spec: WorkloadSpec, rng: np.random.Generator) -> np.ndarray:
    """Logical pages take ids from a seeded permutation of the pool, shared prefix first."""
    p = spec.page_size
    need = spec.pages_needed()
    stride = int(max(1, need.max()))
    bt = np.full((spec.num_seqs, stride), BT_UNUSED, dtype=np.int32)
    perm = rng.permutation(spec.num_pages).astype(np.int32)
    n_shared = spec.shared_prefix_tokens // p
    if spec.shared_prefix_tokens % p:
        raise ValueError("shared prefix must be page aligned")
    if np.any(spec.prefix_lens < spec.shared_prefix_tokens):
        raise ValueError("every prefix must contain the shared prefix")
    cursor = n_shared
    for b in range(spec.num_seqs):
        bt[b, :n_shared] = perm[:n_shared]
        k = int(need[b]) - n_shared
        bt[b, n_shared:n_shared + k] = perm[cursor:cursor + k]
        cursor += k
    if cursor > spec.num_pages:
        raise ValueError(f"pool of {spec.num_pages} pages is too small ({cursor} needed)")
    return bt


def prefix_page_slots(spec: WorkloadSpec, bt: np.ndarray):
    """(physical page, number of prefix slots it holds) in logical order, each page once."""
    p = spec.page_size
    n_shared = spec.shared_prefix_tokens // p
    pages, valid = [], []
    for j in range(n_shared):
        pages.append(int(bt[0, j])); valid.append(p)
    for b in range(spec.num_seqs):
        lp = int(spec.prefix_lens[b])
        for j in range(n_shared, (lp + p - 1) // p):
            pages.append(int(bt[b, j])); valid.append(min(p, lp - j * p))
    return np.asarray(pages, dtype=np.int64), np.asarray(valid, dtype=np.int64)


def materialize(spec: WorkloadSpec, threads: int = 8) -> Workload:
    """Draw every tensor of ``spec`` on the CPU."""
    ss = np.random.SeedSequence(spec.seed)
    c_perm, c_q, c_kn, c_vn, c_kp, c_vp, c_sc = ss.spawn(7)
    bt = build_block_table(spec, np.random.default_rng(c_perm))
    t, hq, hkv, d, p = spec.total_new_tokens, spec.num_q_heads, spec.num_kv_heads, spec.head_dim, spec.page_size
    q = _normal_bf16(c_q, (t, hq, d), threads=threads)
    k_new = _normal_bf16(c_kn, (t, hkv, d), threads=threads)
    v_new = _normal_bf16(c_vn, (t, hkv, d), threads=threads)
    pages, valid = prefix_page_slots(spec, bt)
    n_used = int(pages.shape[0])
    pool_shape = (spec.num_pages, hkv, p, d)
    k_scale = v_scale = None
    if spec.kv_dtype == "bf16":
        k_pool = torch.full(pool_shape, 0, dtype=torch.int16)
        k_pool.fill_(BF16_NAN_BITS)
        k_pool = k_pool.view(torch.bfloat16)
        v_pool = k_pool.clone()
        if n_used:
            kv = _normal_bf16(c_kp, (n_used, hkv, p, d), threads=threads)
            vv = _normal_bf16(c_vp, (n_used, hkv, p, d), threads=threads)
    elif spec.kv_dtype == "fp8":
        g = np.random.default_rng(c_sc)
        k_scale = torch.from_numpy(g.uniform(0.01, 0.1, size=(spec.num_pages, hkv)).astype(np.float32))
        v_scale = torch.from_numpy(g.uniform(0.01, 0.1, size=(spec.num_pages, hkv)).astype(np.float32))
        k_pool = torch.full(pool_shape, FP8_NAN_CODE, dtype=torch.uint8)
        v_pool = k_pool.clone()
        if n_used:
            idx = torch.from_numpy(pages)
            kv = _normal_fp8_codes(c_kp, (n_used, hkv, p, d), k_scale[idx], threads=threads)
            vv = _normal_fp8_codes(c_vp, (n_used, hkv, p, d), v_scale[idx], threads=threads)
    else:
        raise ValueError(spec.kv_dtype)
    if n_used:
        full = np.nonzero(valid == p)[0]
        part = np.nonzero(valid < p)[0]
        for src, dst in ((kv, k_pool), (vv, v_pool)):
            dst[torch.from_numpy(pages[full])] = src[torch.from_numpy(full)]
            # slots past the prefix in a partly filled page keep the sentinel
            for u in part:
                dst[int(pages[u]), :, :int(valid[u])] = src[int(u), :, :int(valid[u])]
    return Workload(spec, q, k_new, v_new, k_pool, v_pool, k_scale, v_scale,
                    torch.from_numpy(bt))


def make(name: str, seed: Optional[int] = None, threads: int = 8) -> Workload:
    return materialize(spec_for(name, seed), threads=threads)


# ----------------------------------------------------------------------------
# agent sessions for the KV-block policy (stand-ins for the paper's traces)

# tool types: (median seconds, lognormal sigma), spanning the orders of magnitude
# of tool execution times the paper reports (sub-second one-liners to builds)
AGENT_TOOLS = ((0.1, 0.8), (1.0, 0.7), (3.0, 1.0), (10.0, 1.2), (22.0, 0.9))


@dataclasses.dataclass
class AgentTrace:
    """Closed-loop agent sessions: sessions[s] = (start_s, [(in_tokens, out_tokens,
    tool_type, tool_s), ...]); history[y] = past durations of tool type y; a node of
    capacity_blocks blocks of block_tokens tokens and a linear service-time model."""

    sessions: list
    history: list
    capacity_blocks: int
    block_tokens: int
    prefill_s_per_token: float
    decode_s_per_token: float
    groups: Optional[list] = None         # shared-prefix group of each session (None: no sharing)
    shared_tokens: Optional[list] = None  # shared prefix tokens of each group


def agent_sessions(num_sessions: int = 32, seed: int = 2000, max_turns: int = 24,
                   block_tokens: int = 16, capacity_fraction: float = 0.4,
                   history_samples: int = 400, shared_groups: int = 0,
                   shared_prefix_tokens: int = 0) -> AgentTrace:
    """Seeded synthetic sessions: a 2-6k-token opening prompt, then turns whose
    inputs are tool outputs (lognormal, median 300 tokens) and outputs of 20-300
    tokens, each followed by a tool call of one of AGENT_TOOLS; starts U[0, 30) s.
    The node holds `capacity_fraction` of the sessions' final KV blocks (at least
    the largest session's), so they compete for memory.  With `shared_groups`,
    session s belongs to group s % shared_groups, whose members' opening prompts
    begin with the same `shared_prefix_tokens` tokens (a system prompt and tool
    schema): trace.groups[s], trace.shared_tokens[g]."""
    ss = np.random.SeedSequence(seed)
    c_sess, c_hist = ss.spawn(2)
    g = np.random.default_rng(c_sess)
    sessions = []
    final_blocks = []
    for _ in range(num_sessions):
        n_turns = int(g.integers(max(1, max_turns // 2), max_turns + 1))
        turns = []
        ctx = 0
        for j in range(n_turns):
            tin = int(g.integers(2000, 6001)) if j == 0 else int(min(4000, g.lognormal(np.log(300.0), 0.8)))
            tout = int(g.integers(20, 301))
            y = int(g.integers(0, len(AGENT_TOOLS)))
            med, sig = AGENT_TOOLS[y]
            turns.append((tin, tout, y, float(g.lognormal(np.log(med), sig))))
            ctx += tin + tout
        sessions.append((float(g.uniform(0.0, 30.0)), turns))
        final_blocks.append(-(-ctx // block_tokens))
    gh = np.random.default_rng(c_hist)
    history = [gh.lognormal(np.log(med), sig, size=history_samples).tolist() for med, sig in AGENT_TOOLS]
    cap = max(max(final_blocks), int(capacity_fraction * sum(final_blocks)))
    tr = AgentTrace(sessions, history, cap, block_tokens, 5e-5, 1e-2)
    if shared_groups > 0:
        assert shared_prefix_tokens <= 2000, "opening prompts start at 2000 tokens"
        tr.groups = [s % shared_groups for s in range(num_sessions)]
        tr.shared_tokens = [shared_prefix_tokens] * shared_groups
    return tr
