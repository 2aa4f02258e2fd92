"""Prefix-cached paged extend attention on MI355X: Python binding of libcw.so.

Thin argument marshalling over the C ABI of include/cw.h: every function
passes device pointers (``tensor.data_ptr()``), host length arrays and torch's
current HIP stream to the library, which runs the HIP kernels.  There is no
fallback: without the built library every call raises.

    extend_attention(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens,
                     suffix_lens, gqa_group, softmax_scale, k_scale=None,
                     v_scale=None, out=None, lse=None, workspace=None)
    decode_attention(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens,
                     gqa_group, softmax_scale, ...)
    kv_write_pages(k_new, v_new, k_pool, v_pool, block_table, prefix_lens,
                   suffix_lens, k_scale=None, v_scale=None, workspace=None)

Page size and head dim are read from the pool shape [num_pages, Hkv, P, D];
an fp8 pool is a uint8 (or float8_e4m3fn) tensor of e4m3fn codes.

The C side sees only pointers, so the binding checks every tensor's dtype and
shape against the call's lengths before passing a pointer (ValueError on a
mismatch): block_table 2-D int32 with a row per sequence; q and out bf16
[T, Hkv*G, D]; k_new, v_new bf16 [T, Hkv, D]; lse fp32 [T, Hkv*G]; v_pool like
k_pool; fp8 scales fp32 [num_pages, Hkv] (and absent for bf16 pools); every
tensor on one GPU and contiguous.
"""
from __future__ import annotations

import ctypes as C
from typing import Optional

import numpy as np
import torch

from . import _lib as L

__all__ = ["CWError", "init", "pinned_allocations", "arg_plan_calls", "extend_attention", "extend_attention_noalloc", "write_extend_attention", "decode_attention", "kv_write_pages",
           "extend_workspace_bytes", "decode_workspace_bytes", "write_pages_workspace_bytes",
           "set_tuning", "plan_items", "decode_plan", "library", "kv_swap_out", "kv_swap_in", "swap_workspace_bytes",
           "step_attention", "step_workspace_bytes", "check_block_table", "ceiling_mfma_bf16", "ceiling_stream_read",
           "ceiling_stream_copy"]


class CWError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


def library():
    return L.load()


def _check(status: int):
    if status != L.CW_OK:
        lib = library()
        raise CWError(status, lib.cw_last_error_message().decode(errors="replace"))


def _lens(x) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
    return a


def _ptr(a: Optional[np.ndarray]):
    return None if a is None or a.size == 0 else a.ctypes.data


def _dptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _want(t, name, dtypes, shape):
    """Marshalling check: `t` has one of `dtypes` and exactly `shape`."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {' or '.join(map(str, dtypes))}")
    if tuple(t.shape) != tuple(int(x) for x in shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(int(x) for x in shape)}")


_BF16 = (torch.bfloat16,)
_FP8 = (torch.uint8, torch.float8_e4m3fn)


def _check_pools(k_pool, v_pool, k_scale, v_scale):
    """Pool, scale and their dtypes; returns (num_pages, Hkv, P, D)."""
    if not isinstance(k_pool, torch.Tensor) or k_pool.dim() != 4:
        raise ValueError("k_pool must be a 4-D tensor [num_pages, Hkv, P, D]")
    _kv_dtype(k_pool)
    _want(v_pool, "v_pool", (k_pool.dtype,), k_pool.shape)
    num_pages, hkv, page, d = k_pool.shape
    if k_pool.dtype == torch.bfloat16:
        if k_scale is not None or v_scale is not None:
            raise ValueError("k_scale / v_scale are for fp8 pools only")
    else:
        if k_scale is None or v_scale is None:
            raise ValueError("an fp8 pool needs k_scale and v_scale")
        _want(k_scale, "k_scale", (torch.float32,), (num_pages, hkv))
        _want(v_scale, "v_scale", (torch.float32,), (num_pages, hkv))
    return num_pages, hkv, page, d


def _check_call(q, k_new, v_new, k_pool, v_pool, block_table, num_seqs, total, gqa_group,
                k_scale=None, v_scale=None, out=None, lse=None):
    """dtype and shape of every tensor of an attention call against its lengths
    (`total` packed rows, `num_seqs` sequences); returns the pool dimensions."""
    num_pages, hkv, page, d = _check_pools(k_pool, v_pool, k_scale, v_scale)
    if not isinstance(block_table, torch.Tensor) or block_table.dim() != 2 \
            or block_table.dtype != torch.int32:
        raise ValueError("block_table must be a 2-D int32 tensor [num_seqs, bt_stride]")
    if block_table.shape[0] < num_seqs:
        raise ValueError(f"block_table has {block_table.shape[0]} rows for {num_seqs} sequences")
    if int(gqa_group) < 1:
        raise ValueError(f"gqa_group = {gqa_group} must be >= 1")
    hq = hkv * int(gqa_group)
    if q is not None:
        _want(q, "q", _BF16, (total, hq, d))
    if out is not None:
        _want(out, "out", _BF16, (total, hq, d))
    _want(k_new, "k_new", _BF16, (total, hkv, d))
    _want(v_new, "v_new", _BF16, (total, hkv, d))
    if lse is not None:
        _want(lse, "lse", (torch.float32,), (total, hq))
    devs = {t.device for t in (q, out, k_new, v_new, k_pool, v_pool, k_scale, v_scale, block_table, lse)
            if t is not None}
    if len(devs) > 1:
        raise ValueError(f"tensors are on different devices: {sorted(map(str, devs))}")
    return num_pages, hkv, page, d


def _lens_pair(prefix_lens, suffix_lens):
    lp, ls = _lens(prefix_lens), _lens(suffix_lens)
    if lp.ndim != 1 or lp.shape != ls.shape:
        raise ValueError(f"prefix_lens {lp.shape} and suffix_lens {ls.shape} must be 1-D of one length")
    return lp, ls


def init():
    """cw_init on the current device (the one-time pinned staging set-up)."""
    _check(library().cw_init())


def pinned_allocations() -> int:
    """Pinned host allocations the library has made in this process."""
    return int(library().cw_pinned_allocations())


def arg_plan_calls() -> int:
    """Calls whose plan travelled in the kernel arguments, in this process."""
    return int(library().cw_arg_plan_calls())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _kv_dtype(pool: torch.Tensor) -> int:
    if pool.dtype == torch.bfloat16:
        return L.CW_KV_BF16
    if pool.dtype in (torch.uint8, torch.float8_e4m3fn):
        return L.CW_KV_FP8_E4M3FN
    raise ValueError(f"unsupported pool dtype {pool.dtype}")


def _workspace(nbytes: int, device, workspace: Optional[torch.Tensor]):
    if workspace is None:
        return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    return workspace


def write_pages_workspace_bytes(num_seqs: int) -> int:
    return int(library().cw_write_pages_workspace_bytes(num_seqs))


def _dtype_code(kv_dtype) -> int:
    if kv_dtype in ("bf16", L.CW_KV_BF16):
        return L.CW_KV_BF16
    if kv_dtype in ("fp8", "fp8_e4m3fn", L.CW_KV_FP8_E4M3FN):
        return L.CW_KV_FP8_E4M3FN
    raise ValueError(f"unsupported kv dtype {kv_dtype!r}")


def extend_workspace_bytes(prefix_lens, suffix_lens, num_kv_heads, gqa_group, head_dim,
                           page_size) -> int:
    lp, ls = _lens(prefix_lens), _lens(suffix_lens)
    return int(library().cw_extend_workspace_bytes(_ptr(lp), _ptr(ls), len(lp), num_kv_heads,
                                                   gqa_group, head_dim, page_size))


def decode_workspace_bytes(prefix_lens, num_kv_heads, gqa_group, head_dim, page_size,
                           kv_dtype="bf16") -> int:
    lp = _lens(prefix_lens)
    return int(library().cw_decode_workspace_bytes(_ptr(lp), len(lp), num_kv_heads, gqa_group,
                                                   head_dim, page_size, _dtype_code(kv_dtype)))


def set_tuning(key: int, value: int):
    _check(library().cw_set_tuning(key, value))


def plan_items(prefix_lens, suffix_lens, num_kv_heads, gqa_group, head_dim, page_size) -> np.ndarray:
    """The extend work list in launch order, int32 [n, 8] (see cw_extend_plan_items)."""
    lp, ls = _lens(prefix_lens), _lens(suffix_lens)
    lib = library()
    n = lib.cw_extend_plan_items(_ptr(lp), _ptr(ls), len(lp), num_kv_heads, gqa_group, head_dim,
                                 page_size, None, 0)
    if n < 0:
        raise CWError(L.CW_ERR_UNSUPPORTED, "invalid plan arguments")
    out = np.zeros((max(n, 1), 8), dtype=np.int32)
    lib.cw_extend_plan_items(_ptr(lp), _ptr(ls), len(lp), num_kv_heads, gqa_group, head_dim,
                             page_size, out.ctypes.data, n)
    return out[:n]


def decode_plan(prefix_lens, num_kv_heads, gqa_group, head_dim, page_size, kv_dtype="bf16",
                rebuilt=False):
    """The decode work list and merge groups, int32 [n, 8] each (see
    cw_decode_plan_items): as planned, or as rebuilt from the compact form."""
    lp = _lens(prefix_lens)
    lib = library()
    ng = C.c_int64()
    dt = {"bf16": L.CW_KV_BF16, "fp8": L.CW_KV_FP8_E4M3FN}[kv_dtype]
    n = lib.cw_decode_plan_items(_ptr(lp), len(lp), num_kv_heads, gqa_group, head_dim, page_size, dt,
                                 int(rebuilt), None, 0, None, 0, C.byref(ng))
    if n < 0:
        raise CWError(L.CW_ERR_UNSUPPORTED, "invalid plan arguments")
    items = np.zeros((max(n, 1), 8), dtype=np.int32)
    groups = np.zeros((max(ng.value, 1), 8), dtype=np.int32)
    lib.cw_decode_plan_items(_ptr(lp), len(lp), num_kv_heads, gqa_group, head_dim, page_size, dt,
                             int(rebuilt), items.ctypes.data, n, groups.ctypes.data, ng.value, C.byref(ng))
    return items[:n], groups[:ng.value]


def kv_write_pages(k_new, v_new, k_pool, v_pool, block_table, prefix_lens, suffix_lens,
                   k_scale=None, v_scale=None, workspace=None):
    lp, ls = _lens_pair(prefix_lens, suffix_lens)
    num_pages, hkv, page, d = _check_call(None, k_new, v_new, k_pool, v_pool, block_table, len(lp),
                                          int(ls.sum()), 1, k_scale, v_scale)
    ws = _workspace(write_pages_workspace_bytes(len(lp)), k_pool.device, workspace)
    _check(library().cw_kv_write_pages(
        _dptr(k_new), _dptr(v_new), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale), _dptr(v_scale),
        _dptr(block_table), block_table.shape[1], num_pages, _ptr(lp), _ptr(ls), len(lp), hkv, d,
        page, _kv_dtype(k_pool), _dptr(ws), ws.numel(), _stream()))


def extend_attention(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens, suffix_lens,
                     gqa_group, softmax_scale, k_scale=None, v_scale=None, out=None, lse=None,
                     workspace=None):
    lp, ls = _lens_pair(prefix_lens, suffix_lens)
    num_pages, hkv, page, d = _check_call(q, k_new, v_new, k_pool, v_pool, block_table, len(lp),
                                          int(ls.sum()), gqa_group, k_scale, v_scale, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = _workspace(extend_workspace_bytes(lp, ls, hkv, gqa_group, d, page),
                               q.device, None)
    _check(library().cw_extend_attention(
        _dptr(q), _dptr(k_new), _dptr(v_new), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale),
        _dptr(v_scale), _dptr(block_table), block_table.shape[1], num_pages, _ptr(lp), _ptr(ls),
        len(lp), hkv, gqa_group, d, page, float(softmax_scale), _kv_dtype(k_pool), _dptr(out),
        _dptr(lse), _dptr(workspace), workspace.numel(), _stream()))
    return out


def extend_attention_noalloc(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens, suffix_lens,
                             gqa_group, softmax_scale, k_scale=None, v_scale=None, out=None,
                             lse=None):
    """extend_attention with the library's static scratch instead of a workspace
    (cw_extend_attention_noalloc; init() must have run on this device).  With
    `out` given, the call allocates nothing."""
    lp, ls = _lens_pair(prefix_lens, suffix_lens)
    num_pages, hkv, page, d = _check_call(q, k_new, v_new, k_pool, v_pool, block_table, len(lp),
                                          int(ls.sum()), gqa_group, k_scale, v_scale, out, lse)
    if out is None:
        out = torch.empty_like(q)
    _check(library().cw_extend_attention_noalloc(
        _dptr(q), _dptr(k_new), _dptr(v_new), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale),
        _dptr(v_scale), _dptr(block_table), block_table.shape[1], num_pages, _ptr(lp), _ptr(ls),
        len(lp), hkv, gqa_group, d, page, float(softmax_scale), _kv_dtype(k_pool), _dptr(out),
        _dptr(lse), _stream()))
    return out


def write_extend_attention(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens, suffix_lens,
                           gqa_group, softmax_scale, k_scale=None, v_scale=None, out=None,
                           lse=None, workspace=None):
    """kv_write_pages + extend_attention in one launch (the pools are written)."""
    lp, ls = _lens_pair(prefix_lens, suffix_lens)
    num_pages, hkv, page, d = _check_call(q, k_new, v_new, k_pool, v_pool, block_table, len(lp),
                                          int(ls.sum()), gqa_group, k_scale, v_scale, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = _workspace(extend_workspace_bytes(lp, ls, hkv, gqa_group, d, page),
                               q.device, None)
    _check(library().cw_write_extend_attention(
        _dptr(q), _dptr(k_new), _dptr(v_new), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale),
        _dptr(v_scale), _dptr(block_table), block_table.shape[1], num_pages, _ptr(lp), _ptr(ls),
        len(lp), hkv, gqa_group, d, page, float(softmax_scale), _kv_dtype(k_pool), _dptr(out),
        _dptr(lse), _dptr(workspace), workspace.numel(), _stream()))
    return out


def step_workspace_bytes(prefix_lens, suffix_lens, num_kv_heads, gqa_group, head_dim, page_size,
                         kv_dtype="bf16") -> int:
    lp, ls = _lens(prefix_lens), _lens(suffix_lens)
    return int(library().cw_step_workspace_bytes(_ptr(lp), _ptr(ls), len(lp), num_kv_heads, gqa_group,
                                                 head_dim, page_size, _dtype_code(kv_dtype)))


def step_attention(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens, suffix_lens,
                   gqa_group, softmax_scale, k_scale=None, v_scale=None, out=None, lse=None,
                   workspace=None):
    """One serving step: page write + attention, decodes on the decode kernel."""
    lp, ls = _lens_pair(prefix_lens, suffix_lens)
    num_pages, hkv, page, d = _check_call(q, k_new, v_new, k_pool, v_pool, block_table, len(lp),
                                          int(ls.sum()), gqa_group, k_scale, v_scale, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = _workspace(step_workspace_bytes(lp, ls, hkv, gqa_group, d, page, _kv_dtype(k_pool)),
                               q.device, None)
    _check(library().cw_step_attention(
        _dptr(q), _dptr(k_new), _dptr(v_new), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale),
        _dptr(v_scale), _dptr(block_table), block_table.shape[1], num_pages, _ptr(lp), _ptr(ls),
        len(lp), hkv, gqa_group, d, page, float(softmax_scale), _kv_dtype(k_pool), _dptr(out),
        _dptr(lse), _dptr(workspace), workspace.numel(), _stream()))
    return out


def swap_workspace_bytes(n: int) -> int:
    return int(library().cw_swap_workspace_bytes(n))


def _hptr(t: Optional[torch.Tensor]):
    """Pointer to a host-pool tensor: device memory or pinned (device-mapped) host memory."""
    if t is None:
        return None
    if not (t.is_cuda or t.is_pinned()):
        raise ValueError("host pools must be pinned host tensors (pin_memory=True) or on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _swap_dims(k_pool, k_host):
    num_pages, hkv, page, d = k_pool.shape
    if tuple(k_host.shape[1:]) != (hkv, page, d):
        raise ValueError(f"host pool blocks {tuple(k_host.shape[1:])} differ from pool blocks {(hkv, page, d)}")
    return num_pages, k_host.shape[0], hkv, page, d


def kv_swap_out(k_pool, v_pool, k_host, v_host, pages, host_blocks, k_scale=None, v_scale=None,
                k_scale_host=None, v_scale_host=None, workspace=None):
    """Pool page pages[i] -> host block host_blocks[i] (K, V and fp8 scales)."""
    pg, hb = _lens(pages), _lens(host_blocks)
    num_pages, n_host, hkv, page, d = _swap_dims(k_pool, k_host)
    ws = _workspace(swap_workspace_bytes(len(pg)), k_pool.device, workspace)
    _check(library().cw_kv_swap_out(
        _dptr(k_pool), _dptr(v_pool), _dptr(k_scale), _dptr(v_scale), num_pages, _hptr(k_host),
        _hptr(v_host), _hptr(k_scale_host), _hptr(v_scale_host), n_host, _ptr(pg), _ptr(hb), len(pg),
        hkv, d, page, _kv_dtype(k_pool), _dptr(ws), ws.numel(), _stream()))


def kv_swap_in(k_host, v_host, k_pool, v_pool, host_blocks, pages, k_scale_host=None,
               v_scale_host=None, k_scale=None, v_scale=None, workspace=None):
    """Host block host_blocks[i] -> pool page pages[i] (K, V and fp8 scales)."""
    pg, hb = _lens(pages), _lens(host_blocks)
    num_pages, n_host, hkv, page, d = _swap_dims(k_pool, k_host)
    ws = _workspace(swap_workspace_bytes(len(pg)), k_pool.device, workspace)
    _check(library().cw_kv_swap_in(
        _hptr(k_host), _hptr(v_host), _hptr(k_scale_host), _hptr(v_scale_host), n_host,
        _dptr(k_pool), _dptr(v_pool), _dptr(k_scale), _dptr(v_scale), num_pages, _ptr(hb), _ptr(pg),
        len(pg), hkv, d, page, _kv_dtype(k_pool), _dptr(ws), ws.numel(), _stream()))


def decode_attention(q, k_new, v_new, k_pool, v_pool, block_table, prefix_lens, gqa_group,
                     softmax_scale, k_scale=None, v_scale=None, out=None, lse=None, workspace=None):
    lp = _lens(prefix_lens)
    if lp.ndim != 1:
        raise ValueError("prefix_lens must be 1-D")
    num_pages, hkv, page, d = _check_call(q, k_new, v_new, k_pool, v_pool, block_table, len(lp),
                                          len(lp), gqa_group, k_scale, v_scale, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = _workspace(decode_workspace_bytes(lp, hkv, gqa_group, d, page,
                                                      _kv_dtype(k_pool)), q.device, None)
    _check(library().cw_decode_attention(
        _dptr(q), _dptr(k_new), _dptr(v_new), _dptr(k_pool), _dptr(v_pool), _dptr(k_scale),
        _dptr(v_scale), _dptr(block_table), block_table.shape[1], num_pages, _ptr(lp), len(lp),
        hkv, gqa_group, d, page, float(softmax_scale), _kv_dtype(k_pool), _dptr(out), _dptr(lse),
        _dptr(workspace), workspace.numel(), _stream()))
    return out


def check_block_table(block_table, prefix_lens, suffix_lens, num_pages: int, page_size: int,
                      workspace=None) -> np.ndarray:
    """Per sequence, the number of block-table entries a call with these lengths
    would read that lie outside [0, num_pages) (waits for the result)."""
    lp, ls = _lens(prefix_lens), _lens(suffix_lens)
    bad = torch.empty(max(len(lp), 1), dtype=torch.int32, device=block_table.device)
    if workspace is None:
        workspace = _workspace(write_pages_workspace_bytes(len(lp)), block_table.device, None)
    _check(library().cw_check_block_table(
        _dptr(block_table), block_table.shape[1], int(num_pages), _ptr(lp), _ptr(ls), len(lp),
        int(page_size), _dptr(bad), _dptr(workspace), workspace.numel(), _stream()))
    return bad[:len(lp)].cpu().numpy()


# measured ceilings (include/cw_ceiling.h): not part of the attention path

def ceiling_mfma_bf16(workgroups: int, iters: int, sink: torch.Tensor, random: bool = True) -> float:
    """Enqueues the matrix-core loop (random operand bits, or the low-entropy
    patterns with `random=False`); returns the FLOPs it performs."""
    kind = L.CW_CEILING_RANDOM if random else L.CW_CEILING_LOW_ENTROPY
    _check(library().cw_ceiling_mfma_bf16(int(workgroups), int(iters), kind, _dptr(sink), _stream()))
    return float(workgroups) * 8 * iters * 131072


def ceiling_stream_read(src: torch.Tensor, sink: torch.Tensor) -> int:
    """Enqueues a streaming read of `src`; returns the bytes it moves."""
    n = src.numel() * src.element_size()
    _check(library().cw_ceiling_stream_read(_dptr(src), n, _dptr(sink), _stream()))
    return n


def ceiling_stream_copy(src: torch.Tensor, dst: torch.Tensor) -> int:
    """Enqueues a streaming copy of `src` into `dst`; returns the bytes it moves."""
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < n:
        raise ValueError("dst is smaller than src")
    _check(library().cw_ceiling_stream_copy(_dptr(src), _dptr(dst), n, _stream()))
    return 2 * n
