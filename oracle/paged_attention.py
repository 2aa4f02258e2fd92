"""Paged prefix + causal suffix attention, by its plain definition (float64).

Test infrastructure (see the package docstring): not used by the library.

Steps, for sequence b with cached prefix length Lp and suffix length Ls, GQA
group G, page size P (the paper's premise: Sec. 2, fixed-size KV blocks reused
by requests that extend a prefix; Sec. 6.1, GQA models):

1. cu[b] = sum of the suffix lengths before b; suffix row i of b is q[cu[b]+i].
2. Gather K_b, V_b of length Lp+Ls: key j < Lp comes from physical page
   block_table[b][j // P], slot j % P (fp8 codes decoded and multiplied by the
   page's per-(page, kv-head) scale); key Lp+i comes from k_new/v_new[cu[b]+i].
3. For query head h (kv head h // G) and row i: n = Lp+i+1 visible keys,
   s = scale * K_b[:n] q, m = max s, p = exp(s - m), l = sum p,
   o = p V_b[:n] / l, lse = m + ln l.

write_pages stores new row i of b at page block_table[b][(Lp+i) // P], slot
(Lp+i) % P: a bit copy for bf16; for fp8 the code nearest to
clamp(x / scale, -448, 448) (IEEE fp32 quotient, ties to even).
"""
from __future__ import annotations

import dataclasses
from typing import Iterable, Optional, Sequence, Tuple

import numpy as np

from .codecs import E4M3FN_MAX, bf16_bits_to_f64, e4m3fn_decode, e4m3fn_encode_rne


@dataclasses.dataclass
class PagedInputs:
    """Raw inputs of one extend call, as host arrays.

    bf16 tensors are uint16 bit patterns; an fp8 pool is uint8 codes.
    """

    q: np.ndarray  # uint16 [T, Hq, D]
    k_new: np.ndarray  # uint16 [T, Hkv, D]
    v_new: np.ndarray  # uint16 [T, Hkv, D]
    k_pool: np.ndarray  # uint16 or uint8 [NP, Hkv, P, D]
    v_pool: np.ndarray
    block_table: np.ndarray  # int32 [B, stride]
    prefix_lens: np.ndarray  # int [B]
    suffix_lens: np.ndarray  # int [B]
    gqa_group: int
    softmax_scale: float
    kv_dtype: str = "bf16"
    k_scale: Optional[np.ndarray] = None  # float32 [NP, Hkv]
    v_scale: Optional[np.ndarray] = None

    @property
    def page_size(self) -> int:
        return int(self.k_pool.shape[2])

    @property
    def num_kv_heads(self) -> int:
        return int(self.k_new.shape[1])

    @property
    def head_dim(self) -> int:
        return int(self.q.shape[2])

    def cu(self) -> np.ndarray:
        c = np.zeros(len(self.suffix_lens) + 1, dtype=np.int64)
        c[1:] = np.cumsum(np.asarray(self.suffix_lens, dtype=np.int64))
        return c


def _pool_rows(pool: np.ndarray, scale: Optional[np.ndarray], pages: np.ndarray,
               slots: np.ndarray, kv_dtype: str) -> np.ndarray:
    """Values of pool[pages[j], :, slots[j], :] as float64 [n, Hkv, D]."""
    raw = pool[pages, :, slots, :]
    if kv_dtype == "bf16":
        return bf16_bits_to_f64(raw)
    if kv_dtype == "fp8":
        return e4m3fn_decode(raw) * scale[pages].astype(np.float64)[:, :, None]
    raise ValueError(kv_dtype)


def gather_sequence_kv(inp: PagedInputs, b: int) -> Tuple[np.ndarray, np.ndarray]:
    """Contiguous K_b, V_b (float64 [Lp+Ls, Hkv, D]) of sequence b (step 2)."""
    lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
    p = inp.page_size
    j = np.arange(lp, dtype=np.int64)
    pages = inp.block_table[b, j // p].astype(np.int64)
    slots = j % p
    c0 = int(inp.cu()[b])
    k = np.concatenate([_pool_rows(inp.k_pool, inp.k_scale, pages, slots, inp.kv_dtype),
                        bf16_bits_to_f64(inp.k_new[c0:c0 + ls])], axis=0)
    v = np.concatenate([_pool_rows(inp.v_pool, inp.v_scale, pages, slots, inp.kv_dtype),
                        bf16_bits_to_f64(inp.v_new[c0:c0 + ls])], axis=0)
    return k, v


def _one_row(k: np.ndarray, v: np.ndarray, q: np.ndarray, n: int, scale: float):
    """Step 3 for one query vector against the first n keys (k, v: [N, D])."""
    s = scale * (k[:n] @ q)
    m = s.max()
    p = np.exp(s - m)
    l = p.sum()
    return (p @ v[:n]) / l, m + np.log(l)


def extend_attention_rowwise(inp: PagedInputs):
    """Implementation (i): one query row at a time.  Returns (out, lse) float64."""
    t_total, hq, d = inp.q.shape
    g = inp.gqa_group
    out = np.zeros((t_total, hq, d), dtype=np.float64)
    lse = np.zeros((t_total, hq), dtype=np.float64)
    cu = inp.cu()
    q = bf16_bits_to_f64(inp.q)
    for b in range(len(inp.suffix_lens)):
        lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
        if ls == 0:
            continue
        k, v = gather_sequence_kv(inp, b)
        for h in range(hq):
            kvh = h // g
            for i in range(ls):
                r = int(cu[b]) + i
                out[r, h], lse[r, h] = _one_row(k[:, kvh], v[:, kvh], q[r, h], lp + i + 1,
                                                inp.softmax_scale)
    return out, lse


def extend_attention_rows(inp: PagedInputs, rows: Iterable[Tuple[int, int]]):
    """Selected outputs only: rows are (packed token index, query head) pairs.

    Returns (out float64 [n, D], lse float64 [n]) in the order given.
    """
    rows = list(rows)
    cu = inp.cu()
    seq_of = np.searchsorted(cu, np.asarray([r for r, _ in rows], dtype=np.int64), side="right") - 1
    out = np.zeros((len(rows), inp.head_dim), dtype=np.float64)
    lse = np.zeros(len(rows), dtype=np.float64)
    order = np.argsort(seq_of, kind="stable")
    cached_b, k, v = -1, None, None
    for idx in order:
        tok, h = rows[idx]
        b = int(seq_of[idx])
        if b != cached_b:
            k, v = gather_sequence_kv(inp, b)
            cached_b = b
        i = tok - int(cu[b])
        kvh = h // inp.gqa_group
        qv = bf16_bits_to_f64(inp.q[tok, h])
        out[idx], lse[idx] = _one_row(k[:, kvh], v[:, kvh], qv, int(inp.prefix_lens[b]) + i + 1,
                                      inp.softmax_scale)
    return out, lse


def _blocked_rows(inp: PagedInputs, b: int, k: np.ndarray, v: np.ndarray, t0: int, t1: int):
    """Suffix tokens [t0, t1) of sequence b, every query head, by implementation
    (ii): per kv head, S = Q K^T over the visible keys with one matrix product
    (row = token * G + group member), keys past each row's causal limit set to
    -inf, row softmax, then P V.  k, v: the sequence's gathered keys/values; the
    arithmetic runs in their dtype (float64, or float32 for the timed CPU
    baseline).  Returns (out [t1-t0, Hq, D], lse [t1-t0, Hq]) in that dtype."""
    _, hq, d = inp.q.shape
    g = inp.gqa_group
    lp = int(inp.prefix_lens[b])
    c0 = int(inp.cu()[b])
    dt = k.dtype
    out = np.zeros((t1 - t0, hq, d), dtype=dt)
    lse = np.zeros((t1 - t0, hq), dtype=dt)
    n_max = lp + t1
    limit = lp + np.repeat(np.arange(t0, t1), g) + 1  # visible keys per row
    for kvh in range(inp.num_kv_heads):
        kh, vh = k[:, kvh], v[:, kvh]
        qb = bf16_bits_to_f64(inp.q[c0 + t0:c0 + t1, kvh * g:(kvh + 1) * g]).astype(dt)
        qb = qb.reshape((t1 - t0) * g, d)
        s = dt.type(inp.softmax_scale) * (qb @ kh[:n_max].T)
        s[np.arange(n_max)[None, :] >= limit[:, None]] = -np.inf
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        l = p.sum(axis=1, keepdims=True)
        o = (p @ vh[:n_max]) / l
        out[:, kvh * g:(kvh + 1) * g] = o.reshape(t1 - t0, g, d)
        lse[:, kvh * g:(kvh + 1) * g] = (m + np.log(l)).reshape(t1 - t0, g)
    return out, lse


def extend_attention_blocked(inp: PagedInputs, block_tokens: int = 64, dtype=np.float64):
    """Implementation (ii): per (sequence, kv head), blocks of query tokens x G heads.

    S = Q K^T over all visible keys with a matrix product, keys past each
    row's causal limit set to -inf, row softmax, then P V.  `dtype` float32
    runs the same steps in single precision (the CPU baseline the benchmark
    times); the parity checks use the float64 default.
    """
    t_total, hq, d = inp.q.shape
    out = np.zeros((t_total, hq, d), dtype=dtype)
    lse = np.zeros((t_total, hq), dtype=dtype)
    cu = inp.cu()
    for b in range(len(inp.suffix_lens)):
        ls = int(inp.suffix_lens[b])
        if ls == 0:
            continue
        k, v = gather_sequence_kv(inp, b)
        if dtype != np.float64:
            k, v = k.astype(dtype), v.astype(dtype)
        c0 = int(cu[b])
        for t0 in range(0, ls, block_tokens):
            t1 = min(ls, t0 + block_tokens)
            out[c0 + t0:c0 + t1], lse[c0 + t0:c0 + t1] = _blocked_rows(inp, b, k, v, t0, t1)
    return out, lse


def extend_attention_token_blocks(inp: PagedInputs, blocks: Sequence[Tuple[int, int, int]]):
    """Implementation (ii) on chosen blocks only: `blocks` lists (sequence b,
    first suffix token t0, end t1).  Returns a list of (out float64
    [t1-t0, Hq, D], lse float64 [t1-t0, Hq]) in the order given; each
    sequence's keys are gathered once."""
    res = [None] * len(blocks)
    by_seq = {}
    for i, (b, t0, t1) in enumerate(blocks):
        by_seq.setdefault(int(b), []).append(i)
    for b, idx in by_seq.items():
        k, v = gather_sequence_kv(inp, b)
        for i in idx:
            _, t0, t1 = blocks[i]
            res[i] = _blocked_rows(inp, b, k, v, int(t0), int(t1))
    return res


def decode_attention(q: np.ndarray, k_new: np.ndarray, v_new: np.ndarray, k_pool: np.ndarray,
                     v_pool: np.ndarray, block_table: np.ndarray, prefix_lens: np.ndarray,
                     gqa_group: int, softmax_scale: float, kv_dtype: str = "bf16",
                     k_scale=None, v_scale=None):
    """One new token per sequence: extend attention with every suffix length 1."""
    b = len(prefix_lens)
    inp = PagedInputs(q, k_new, v_new, k_pool, v_pool, block_table, np.asarray(prefix_lens),
                      np.ones(b, dtype=np.int64), gqa_group, softmax_scale, kv_dtype,
                      k_scale, v_scale)
    return extend_attention_rowwise(inp)


def write_pages(inp: PagedInputs) -> Tuple[np.ndarray, np.ndarray]:
    """Pools after storing every new K/V row in its slot; other bytes unchanged."""
    k_pool = inp.k_pool.copy()
    v_pool = inp.v_pool.copy()
    p = inp.page_size
    cu = inp.cu()
    for b in range(len(inp.suffix_lens)):
        lp, ls = int(inp.prefix_lens[b]), int(inp.suffix_lens[b])
        for i in range(ls):
            pos = lp + i
            pg = int(inp.block_table[b, pos // p])
            sl = pos % p
            r = int(cu[b]) + i
            if inp.kv_dtype == "bf16":
                k_pool[pg, :, sl, :] = inp.k_new[r]
                v_pool[pg, :, sl, :] = inp.v_new[r]
            else:
                for src, dst, sc in ((inp.k_new, k_pool, inp.k_scale), (inp.v_new, v_pool, inp.v_scale)):
                    x = bf16_bits_to_f64(src[r]).astype(np.float32)  # exact
                    quot = x / sc[pg].astype(np.float32)[:, None]  # IEEE fp32 division
                    quot = np.clip(quot, -E4M3FN_MAX, E4M3FN_MAX)
                    dst[pg, :, sl, :] = e4m3fn_encode_rne(quot.astype(np.float64))
    return k_pool, v_pool
