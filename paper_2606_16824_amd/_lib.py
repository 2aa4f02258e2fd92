"""ctypes declarations of libcw.so (the C ABI declared in include/cw.h,
include/cw_ceiling.h and include/cw_policy.h)."""
from __future__ import annotations

import ctypes as C
import os

# CW_LIBRARY names another build of the same library (the sanitizer build of
# the host code, for the CPU tests); by default the in-tree libcw.so
LIB_PATH = os.environ.get("CW_LIBRARY") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libcw.so")

(CW_OK, CW_ERR_NULL, CW_ERR_UNSUPPORTED, CW_ERR_BAD_LENS, CW_ERR_ALIGN, CW_ERR_WORKSPACE, CW_ERR_HIP,
 CW_ERR_ALIAS, CW_ERR_INIT) = range(9)
CW_KV_BF16, CW_KV_FP8_E4M3FN = 0, 1
CW_TUNE_KV_CHUNK_TILES, CW_TUNE_TARGET_WGS, CW_TUNE_EXTEND_KERNEL, CW_TUNE_DEAL_ROUNDS, CW_TUNE_PLAN_DIRECT, CW_TUNE_SUFFIX_WEIGHT = 0, 1, 2, 3, 4, 5
CW_TUNE_COMPACT_DECODE, CW_TUNE_ARG_PLANS = 6, 7
CW_CEILING_LOW_ENTROPY, CW_CEILING_RANDOM = 0, 1

_i32p = C.POINTER(C.c_int32)
_fp = C.POINTER(C.c_float)
_vp = C.c_void_p
_i32 = C.c_int32
_sz = C.c_size_t

# name: (restype, argtypes)
SIGNATURES = {
    "cw_write_pages_workspace_bytes": (_sz, [_i32]),
    "cw_kv_write_pages": (C.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _i32,
                                    _i32, _i32, _i32, C.c_int, _vp, _sz, _vp]),
    "cw_extend_workspace_bytes": (_sz, [_vp, _vp, _i32, _i32, _i32, _i32, _i32]),
    "cw_extend_attention": (C.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp,
                                      _i32, _i32, _i32, _i32, _i32, C.c_float, C.c_int, _vp, _vp,
                                      _vp, _sz, _vp]),
    "cw_write_extend_attention": (C.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp,
                                            _vp, _i32, _i32, _i32, _i32, _i32, C.c_float, C.c_int,
                                            _vp, _vp, _vp, _sz, _vp]),
    "cw_decode_workspace_bytes": (_sz, [_vp, _i32, _i32, _i32, _i32, _i32, _i32]),
    "cw_swap_workspace_bytes": (_sz, [_i32]),
    "cw_step_workspace_bytes": (_sz, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32]),
    "cw_step_attention": (C.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp,
                                    _i32, _i32, _i32, _i32, _i32, C.c_float, C.c_int, _vp, _vp,
                                    _vp, _sz, _vp]),
    "cw_kv_swap_out": (C.c_int, [_vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _i32,
                                 _i32, _i32, _i32, C.c_int, _vp, _sz, _vp]),
    "cw_kv_swap_in": (C.c_int, [_vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _i32,
                                _i32, _i32, _i32, C.c_int, _vp, _sz, _vp]),
    "cw_decode_attention": (C.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp,
                                      _i32, _i32, _i32, _i32, _i32, C.c_float, C.c_int, _vp, _vp,
                                      _vp, _sz, _vp]),
    "cw_check_block_table": (C.c_int, [_vp, _i32, _i32, _vp, _vp, _i32, _i32, _vp, _vp, _sz, _vp]),
    "cw_set_tuning": (C.c_int, [C.c_int, _i32]),
    "cw_set_timing_events": (C.c_int, [_vp, _vp]),
    "cw_extend_plan_items": (C.c_int64, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, C.c_int64]),
    "cw_decode_plan_items": (C.c_int64, [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, C.c_int64, _vp,
                                         C.c_int64, _vp]),
    "cw_init": (C.c_int, []),
    "cw_extend_attention_noalloc": (C.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp,
                                              _vp, _i32, _i32, _i32, _i32, _i32, C.c_float, C.c_int,
                                              _vp, _vp, _vp]),
    "cw_pinned_allocations": (C.c_int64, []),
    "cw_arg_plan_calls": (C.c_int64, []),
    "cw_status_string": (C.c_char_p, [C.c_int]),
    "cw_last_error_message": (C.c_char_p, []),
    "cw_version": (_i32, []),
    # include/cw_ceiling.h (measurement kernels)
    "cw_ceiling_mfma_bf16": (C.c_int, [_i32, _i32, _i32, _vp, _vp]),
    "cw_ceiling_stream_read": (C.c_int, [_vp, _sz, _vp, _vp]),
    "cw_ceiling_stream_copy": (C.c_int, [_vp, _vp, _sz, _vp]),
    # include/cw_policy.h (host-only)
    "cw_policy_simulate": (C.c_int, [_vp, _vp, _vp, _vp, C.c_int64]),
    "cw_policy_predict": (C.c_int, [_vp, _i32, C.c_double, _vp]),
    "cw_policy_simulate_log": (C.c_int, [_vp, _vp, _vp, _vp]),
    "cw_bm_create": (C.c_int, [_i32, _i32, _vp]),
    "cw_bm_destroy": (C.c_int, [_vp]),
    "cw_bm_add_session": (C.c_int, [_vp, _i32, _i32, _i32]),
    "cw_bm_admit": (C.c_int, [_vp, _i32, C.c_int64, C.c_int64, C.c_int64, _vp, _i32, _vp, _vp, _vp]),
    "cw_bm_release": (C.c_int, [_vp, _i32, C.c_double]),
    "cw_bm_rebuild": (C.c_int, [_vp, _vp, _vp, _i32]),
    "cw_bm_stats": (C.c_int, [_vp, _vp, _vp]),
    "cw_bm_create_with_host_pool": (C.c_int, [_i32, _i32, _i32, _vp]),
    "cw_bm_admit_swaps": (C.c_int, [_vp, _i32, C.c_int64, C.c_int64, C.c_int64, _vp, _i32, _vp, _vp, _vp,
                                    _vp]),
    "cw_bm_host_stats": (C.c_int, [_vp, _vp, _vp]),
}

_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Loads libcw.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} not found: build the HIP library first "
            "(python -m paper_2606_16824_amd.build)")
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib
