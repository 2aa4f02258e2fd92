"""Page swap between the device page pool and a host block pool -- oracle.

The paper's offloading configuration (CacheWise, Sec. 6.4, KV cache movement)
moves evicted KV blocks from GPU memory to CPU DRAM and back when their
session resumes.  What moves is a list of whole pages: entry i of a swap-out
copies pool page pages[i] (every kv head of it, K and V, and for fp8 pools
its per-(page, kv head) scales) to host block host_blocks[i]; a swap-in copies
host block host_blocks[i] to pool page pages[i].  Bytes are copied unchanged.

Arrays are numpy: pools [num_pages, Hkv, P, D] of any element type (raw bf16
bits or fp8 codes), scales [num_pages, Hkv] float32 or None; host pools
[num_host_blocks, Hkv, P, D] and [num_host_blocks, Hkv].  Each function
returns new arrays and leaves its inputs alone.  Destinations must be
distinct (two entries writing one block would make the result order
dependent); sources may repeat.
"""
from typing import Optional, Sequence, Tuple

import numpy as np


def _check(src_ids: Sequence[int], dst_ids: Sequence[int], n_src: int, n_dst: int):
    if len(src_ids) != len(dst_ids):
        raise ValueError("the two block lists differ in length")
    for s, d in zip(src_ids, dst_ids):
        if not (0 <= s < n_src and 0 <= d < n_dst):
            raise ValueError(f"block id out of range: {s} -> {d}")
    if len(set(int(d) for d in dst_ids)) != len(dst_ids):
        raise ValueError("a destination block appears twice")


def _copy_blocks(src: np.ndarray, dst: np.ndarray, src_ids, dst_ids) -> np.ndarray:
    out = dst.copy()
    for s, d in zip(src_ids, dst_ids):  # one whole block per entry, in list order
        out[int(d)] = src[int(s)]
    return out


def swap_out(k_pool: np.ndarray, v_pool: np.ndarray, k_scale: Optional[np.ndarray],
             v_scale: Optional[np.ndarray], pages: Sequence[int], host_k: np.ndarray,
             host_v: np.ndarray, host_ks: Optional[np.ndarray], host_vs: Optional[np.ndarray],
             host_blocks: Sequence[int]) -> Tuple:
    """Pool page pages[i] -> host block host_blocks[i]; returns the new host arrays."""
    _check(pages, host_blocks, k_pool.shape[0], host_k.shape[0])
    hk = _copy_blocks(k_pool, host_k, pages, host_blocks)
    hv = _copy_blocks(v_pool, host_v, pages, host_blocks)
    hks = None if k_scale is None else _copy_blocks(k_scale, host_ks, pages, host_blocks)
    hvs = None if v_scale is None else _copy_blocks(v_scale, host_vs, pages, host_blocks)
    return hk, hv, hks, hvs


def swap_in(host_k: np.ndarray, host_v: np.ndarray, host_ks: Optional[np.ndarray],
            host_vs: Optional[np.ndarray], host_blocks: Sequence[int], k_pool: np.ndarray,
            v_pool: np.ndarray, k_scale: Optional[np.ndarray], v_scale: Optional[np.ndarray],
            pages: Sequence[int]) -> Tuple:
    """Host block host_blocks[i] -> pool page pages[i]; returns the new pool arrays."""
    _check(host_blocks, pages, host_k.shape[0], k_pool.shape[0])
    k = _copy_blocks(host_k, k_pool, host_blocks, pages)
    v = _copy_blocks(host_v, v_pool, host_blocks, pages)
    ks = None if k_scale is None else _copy_blocks(host_ks, k_scale, host_blocks, pages)
    vs = None if v_scale is None else _copy_blocks(host_vs, v_scale, host_blocks, pages)
    return k, v, ks, vs
