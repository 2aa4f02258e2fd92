"""The C ABI on the CPU: symbols, argument validation, status strings, the planner.

No call here reaches the GPU: invalid arguments are rejected before any HIP
call, and the planner is host code.
"""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2606_16824_amd as cwlib
from paper_2606_16824_amd import _lib as L

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
HEADERS = sorted(os.path.join(INCLUDE, h) for h in os.listdir(INCLUDE) if h.endswith(".h"))


def lib():
    return cwlib.library()


def test_exports_every_declared_symbol():
    text = "".join(open(h).read() for h in HEADERS)
    names = set(re.findall(r"\b(cw_[a-z0-9_]+)\s*\(", text))
    assert {"cw_kv_write_pages", "cw_extend_attention", "cw_decode_attention"} <= names
    for n in sorted(names):
        assert hasattr(lib(), n), n
    assert names == set(L.SIGNATURES), "binding and header disagree"
    assert lib().cw_version() >= 100


def test_status_strings():
    for s in range(8):
        assert lib().cw_status_string(s).decode().startswith("CW_")


FAKE = 0x100000  # a 16-byte-aligned address that is never dereferenced


def _step(**over):
    lp = np.array(over.pop("lp", [10, 20]), dtype=np.int32)
    ls = np.array(over.pop("ls", [5, 6]), dtype=np.int32)
    a = dict(q=FAKE, k_new=FAKE, v_new=FAKE, k_pool=FAKE, v_pool=FAKE, k_scale=None, v_scale=None,
             block_table=FAKE, bt_stride=4, num_pages=100, num_kv_heads=2, gqa_group=4,
             head_dim=128, page_size=16, scale=0.088, kv_dtype=0, out=FAKE, lse=None,
             workspace=FAKE, workspace_bytes=1 << 40)
    a.update(over)
    return lib().cw_step_attention(
        a["q"], a["k_new"], a["v_new"], a["k_pool"], a["v_pool"], a["k_scale"], a["v_scale"],
        a["block_table"], a["bt_stride"], a["num_pages"], lp.ctypes.data, ls.ctypes.data, len(lp),
        a["num_kv_heads"], a["gqa_group"], a["head_dim"], a["page_size"], a["scale"],
        a["kv_dtype"], a["out"], a["lse"], a["workspace"], a["workspace_bytes"], None)


def _extend(fused=False, **over):
    if fused == "step":
        return _step(**over)
    lp = np.array(over.pop("lp", [10, 20]), dtype=np.int32)
    ls = np.array(over.pop("ls", [5, 6]), dtype=np.int32)
    a = dict(q=FAKE, k_new=FAKE, v_new=FAKE, k_pool=FAKE, v_pool=FAKE, k_scale=None, v_scale=None,
             block_table=FAKE, bt_stride=4, num_pages=100, num_kv_heads=2, gqa_group=4,
             head_dim=128, page_size=16, scale=0.088, kv_dtype=0, out=FAKE, lse=None,
             workspace=FAKE, workspace_bytes=1 << 40)
    a.update(over)
    fn = lib().cw_write_extend_attention if fused else lib().cw_extend_attention
    return fn(
        a["q"], a["k_new"], a["v_new"], a["k_pool"], a["v_pool"], a["k_scale"], a["v_scale"],
        a["block_table"], a["bt_stride"], a["num_pages"], lp.ctypes.data, ls.ctypes.data, len(lp),
        a["num_kv_heads"], a["gqa_group"], a["head_dim"], a["page_size"], a["scale"],
        a["kv_dtype"], a["out"], a["lse"], a["workspace"], a["workspace_bytes"], None)


@pytest.mark.parametrize("over,status", [
    (dict(q=None), L.CW_ERR_NULL),
    (dict(out=None), L.CW_ERR_NULL),
    (dict(block_table=None), L.CW_ERR_NULL),
    (dict(kv_dtype=1), L.CW_ERR_NULL),  # fp8 without scales
    (dict(head_dim=96), L.CW_ERR_UNSUPPORTED),
    (dict(page_size=32), L.CW_ERR_UNSUPPORTED),
    (dict(gqa_group=0), L.CW_ERR_UNSUPPORTED),
    (dict(gqa_group=17), L.CW_ERR_UNSUPPORTED),
    (dict(num_kv_heads=0), L.CW_ERR_UNSUPPORTED),
    (dict(scale=0.0), L.CW_ERR_UNSUPPORTED),
    (dict(scale=float("inf")), L.CW_ERR_UNSUPPORTED),
    (dict(kv_dtype=7), L.CW_ERR_UNSUPPORTED),
    (dict(lp=[-1, 3]), L.CW_ERR_BAD_LENS),
    (dict(ls=[2, -3]), L.CW_ERR_BAD_LENS),
    (dict(lp=[60, 0], ls=[5, 1]), L.CW_ERR_BAD_LENS),  # 65 > bt_stride * P = 64
    (dict(bt_stride=0), L.CW_ERR_BAD_LENS),
    (dict(q=FAKE + 8), L.CW_ERR_ALIGN),
    (dict(k_pool=FAKE + 2), L.CW_ERR_ALIGN),
    (dict(workspace=FAKE + 4), L.CW_ERR_ALIGN),
    (dict(workspace_bytes=16), L.CW_ERR_WORKSPACE),
    (dict(workspace=None), L.CW_ERR_WORKSPACE),
])
@pytest.mark.parametrize("fused", [False, True, "step"])
def test_extend_rejects_before_any_gpu_work(over, status, fused):
    assert _extend(fused=fused, **over) == status
    assert lib().cw_last_error_message().decode()


def test_fused_write_needs_the_pools_even_without_a_prefix():
    # the plain extend reads no pool when every prefix is empty; the fused call writes it
    assert _extend(lp=[0, 0], k_pool=None, v_pool=None, workspace_bytes=1) == L.CW_ERR_WORKSPACE
    assert _extend(fused=True, lp=[0, 0], k_pool=None) == L.CW_ERR_NULL
    assert _extend(fused=True, lp=[0, 0], v_pool=None) == L.CW_ERR_NULL


def test_all_empty_suffixes_is_a_no_op():
    assert _extend(ls=[0, 0], q=None, out=None) == L.CW_OK


def test_lp_plus_ls_exactly_fills_table_is_valid_until_workspace():
    assert _extend(lp=[48, 0], ls=[16, 1], workspace_bytes=1) == L.CW_ERR_WORKSPACE


def test_write_pages_validation():
    lp = np.array([3, 0], dtype=np.int32)
    ls = np.array([2, 4], dtype=np.int32)
    ws = lib().cw_write_pages_workspace_bytes(2)
    assert ws >= 32 and ws % 256 == 0

    def call(**o):
        a = dict(k_new=FAKE, v_new=FAKE, k_pool=FAKE, v_pool=FAKE, k_scale=None, v_scale=None,
                 bt=FAKE, stride=1, d=128, p=16, dt=0, ws=FAKE, wsb=ws)
        a.update(o)
        return lib().cw_kv_write_pages(a["k_new"], a["v_new"], a["k_pool"], a["v_pool"],
                                       a["k_scale"], a["v_scale"], a["bt"], a["stride"], 10,
                                       lp.ctypes.data, ls.ctypes.data, 2, 2, a["d"], a["p"],
                                       a["dt"], a["ws"], a["wsb"], None)
    assert call(k_pool=None) == L.CW_ERR_NULL
    assert call(dt=1) == L.CW_ERR_NULL
    assert call(d=80) == L.CW_ERR_UNSUPPORTED
    assert call(v_new=FAKE + 1) == L.CW_ERR_ALIGN
    assert call(wsb=8) == L.CW_ERR_WORKSPACE


def test_workspace_query_rejects_bad_args():
    lp = np.array([5], dtype=np.int32)
    ls = np.array([-1], dtype=np.int32)
    assert lib().cw_extend_workspace_bytes(lp.ctypes.data, ls.ctypes.data, 1, 1, 1, 64, 16) == 0
    assert lib().cw_extend_workspace_bytes(lp.ctypes.data, lp.ctypes.data, 1, 1, 1, 72, 16) == 0
    assert lib().cw_extend_workspace_bytes(lp.ctypes.data, lp.ctypes.data, 1, 1, 1, 64, 24) == 0
    assert lib().cw_extend_workspace_bytes(lp.ctypes.data, lp.ctypes.data, 1, 1, 1, 64, 16) > 0
    assert lib().cw_decode_workspace_bytes(lp.ctypes.data, 1, 1, 1, 64, 16, 7) == 0
    assert lib().cw_decode_workspace_bytes(lp.ctypes.data, 1, 1, 1, 72, 16, 0) == 0
    assert lib().cw_decode_workspace_bytes(ls.ctypes.data, 1, 1, 1, 64, 16, 0) == 0
    for dt in (0, 1):
        assert lib().cw_decode_workspace_bytes(lp.ctypes.data, 1, 1, 1, 64, 16, dt) > 0


def test_tuning_keys():
    assert lib().cw_set_tuning(0, -1) == L.CW_ERR_UNSUPPORTED
    assert lib().cw_set_tuning(9, 1) == L.CW_ERR_UNSUPPORTED
    assert lib().cw_set_tuning(0, 0) == L.CW_OK
    assert lib().cw_set_tuning(1, 0) == L.CW_OK
    # extend kernel choice: 0/1 eight waves, 2 four waves of 64 rows, nothing else
    for v in (0, 1, 2):
        assert lib().cw_set_tuning(L.CW_TUNE_EXTEND_KERNEL, v) == L.CW_OK
    assert lib().cw_set_tuning(L.CW_TUNE_EXTEND_KERNEL, 3) == L.CW_ERR_UNSUPPORTED
    assert lib().cw_set_tuning(L.CW_TUNE_EXTEND_KERNEL, 0) == L.CW_OK
    assert lib().cw_set_tuning(L.CW_TUNE_DEAL_ROUNDS, 0) == L.CW_OK
    assert lib().cw_set_tuning(L.CW_TUNE_DEAL_ROUNDS, 1) == L.CW_OK
    assert lib().cw_set_tuning(L.CW_TUNE_PLAN_DIRECT, 1) == L.CW_OK
    assert lib().cw_set_tuning(L.CW_TUNE_PLAN_DIRECT, 0) == L.CW_OK
    assert lib().cw_set_tuning(L.CW_TUNE_SUFFIX_WEIGHT, 0) == L.CW_ERR_UNSUPPORTED
    assert lib().cw_set_tuning(L.CW_TUNE_SUFFIX_WEIGHT, 10001) == L.CW_ERR_UNSUPPORTED
    assert lib().cw_set_tuning(L.CW_TUNE_SUFFIX_WEIGHT, 125) == L.CW_OK


def _swap(out=True, **over):
    pages = np.array(over.pop("pages", [3, 7, 1]), dtype=np.int32)
    host = np.array(over.pop("host", [0, 2, 1]), dtype=np.int32)
    a = dict(pool_k=FAKE, pool_v=FAKE, ks=None, vs=None, num_pages=10, host_k=FAKE, host_v=FAKE,
             hks=None, hvs=None, num_host=4, n=len(pages), num_kv_heads=2, head_dim=128,
             page_size=16, kv_dtype=0, workspace=FAKE, workspace_bytes=1 << 20)
    a.update(over)
    if out:
        return lib().cw_kv_swap_out(a["pool_k"], a["pool_v"], a["ks"], a["vs"], a["num_pages"],
                                    a["host_k"], a["host_v"], a["hks"], a["hvs"], a["num_host"],
                                    pages.ctypes.data, host.ctypes.data, a["n"], a["num_kv_heads"],
                                    a["head_dim"], a["page_size"], a["kv_dtype"], a["workspace"],
                                    a["workspace_bytes"], None)
    return lib().cw_kv_swap_in(a["host_k"], a["host_v"], a["hks"], a["hvs"], a["num_host"],
                               a["pool_k"], a["pool_v"], a["ks"], a["vs"], a["num_pages"],
                               host.ctypes.data, pages.ctypes.data, a["n"], a["num_kv_heads"],
                               a["head_dim"], a["page_size"], a["kv_dtype"], a["workspace"],
                               a["workspace_bytes"], None)


@pytest.mark.parametrize("over,status", [
    (dict(pool_k=None), L.CW_ERR_NULL),
    (dict(host_v=None), L.CW_ERR_NULL),
    (dict(kv_dtype=1), L.CW_ERR_NULL),  # fp8 without scales
    (dict(kv_dtype=5), L.CW_ERR_UNSUPPORTED),
    (dict(head_dim=96), L.CW_ERR_UNSUPPORTED),
    (dict(page_size=8), L.CW_ERR_UNSUPPORTED),
    (dict(pages=[3, 10, 1]), L.CW_ERR_BAD_LENS),   # page id past the pool
    (dict(host=[0, 4, 1]), L.CW_ERR_BAD_LENS),     # host block past the host pool
    (dict(pages=[-1, 7, 1]), L.CW_ERR_BAD_LENS),
    (dict(n=-1), L.CW_ERR_BAD_LENS),
    (dict(host_k=FAKE + 4), L.CW_ERR_ALIGN),
    (dict(workspace_bytes=8), L.CW_ERR_WORKSPACE),
    (dict(workspace=None), L.CW_ERR_WORKSPACE),
])
@pytest.mark.parametrize("out", [True, False])
def test_swap_rejects_before_any_gpu_work(over, status, out):
    assert _swap(out, **over) == status
    assert lib().cw_last_error_message().decode()


def test_swap_destinations_must_be_distinct():
    # swap-out writes host blocks, swap-in writes pool pages
    assert _swap(True, host=[0, 2, 0]) == L.CW_ERR_BAD_LENS
    assert _swap(False, pages=[3, 3, 1]) == L.CW_ERR_BAD_LENS
    # repeated sources are allowed; these calls fail only at the workspace check
    assert _swap(True, pages=[3, 3, 1], workspace_bytes=8) == L.CW_ERR_WORKSPACE
    assert _swap(False, host=[0, 0, 1], workspace_bytes=8) == L.CW_ERR_WORKSPACE


def test_empty_swap_is_a_no_op():
    assert _swap(True, pages=[], host=[], pool_k=None, workspace=None) == L.CW_OK
    assert lib().cw_swap_workspace_bytes(0) >= 256 and lib().cw_swap_workspace_bytes(-1) == 0


def test_ceiling_calls_reject_before_any_gpu_work():
    L_ = lib()
    R = L.CW_CEILING_RANDOM
    assert L_.cw_ceiling_mfma_bf16(256, 10, R, None, None) == L.CW_ERR_NULL
    assert L_.cw_ceiling_mfma_bf16(0, 10, R, 16, None) == L.CW_ERR_UNSUPPORTED
    assert L_.cw_ceiling_mfma_bf16(256, 0, R, 16, None) == L.CW_ERR_UNSUPPORTED
    assert L_.cw_ceiling_mfma_bf16(65537, 10, R, 16, None) == L.CW_ERR_UNSUPPORTED
    for bad in (2, -1, 7):
        assert L_.cw_ceiling_mfma_bf16(256, 10, bad, 16, None) == L.CW_ERR_UNSUPPORTED
    assert L_.cw_ceiling_stream_read(None, 1024, 16, None) == L.CW_ERR_NULL
    assert L_.cw_ceiling_stream_read(16, 0, 16, None) == L.CW_ERR_UNSUPPORTED
    assert L_.cw_ceiling_stream_read(24, 1024, 16, None) == L.CW_ERR_ALIGN
    assert L_.cw_ceiling_stream_read(16, 1000, 16, None) == L.CW_ERR_ALIGN
    assert L_.cw_ceiling_stream_copy(16, None, 1024, None) == L.CW_ERR_NULL
    assert L_.cw_ceiling_stream_copy(4096, 4096 + 512, 1024, None) == L.CW_ERR_UNSUPPORTED
    assert b"overlap" in L_.cw_last_error_message()


def test_check_block_table_rejects_before_any_gpu_work():
    L_ = lib()
    lp = np.array([10, 20], dtype=np.int32)
    ls = np.array([5, 6], dtype=np.int32)

    def call(bt=FAKE, stride=4, num_pages=100, lp=lp, ls=ls, page=16, bad=FAKE, ws=FAKE,
             ws_bytes=1 << 20):
        return L_.cw_check_block_table(bt, stride, num_pages, lp.ctypes.data, ls.ctypes.data,
                                       len(lp), page, bad, ws, ws_bytes, None)

    assert call(bt=None) == L.CW_ERR_NULL
    assert call(bad=None) == L.CW_ERR_NULL
    assert call(page=32) == L.CW_ERR_UNSUPPORTED
    assert call(num_pages=-1) == L.CW_ERR_BAD_LENS
    assert call(lp=np.array([60, 0], dtype=np.int32)) == L.CW_ERR_BAD_LENS  # 65 > 4 * 16
    assert call(ls=np.array([-1, 0], dtype=np.int32)) == L.CW_ERR_BAD_LENS
    assert call(bt=FAKE + 2) == L.CW_ERR_ALIGN
    assert call(ws=FAKE + 4) == L.CW_ERR_ALIGN
    assert call(ws_bytes=16) == L.CW_ERR_WORKSPACE
    assert call(ws=None) == L.CW_ERR_WORKSPACE
    assert L_.cw_last_error_message()


def test_binding_fails_loudly_without_the_library(tmp_path):
    # no fallback path: with the library absent, the first call raises
    import subprocess
    import sys
    code = ("import paper_2606_16824_amd as cw\n"
            "try:\n"
            "    cw.write_pages_workspace_bytes(1)\n"
            "except RuntimeError as e:\n"
            "    print('raised:', e)\n"
            "else:\n"
            "    print('no error')\n")
    env = dict(os.environ, CW_LIBRARY=str(tmp_path / "absent" / "libcw.so"))
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], env=env, cwd=root, capture_output=True,
                       text=True, timeout=300)
    assert "raised:" in r.stdout and "not found" in r.stdout, r.stdout + r.stderr


# distinct, far-apart fake ranges; sizes for the default call: 11 rows x 8 heads x 128 x 2 B
_BASES = dict(q=0x10000000, k_new=0x20000000, v_new=0x30000000, k_pool=0x40000000,
              v_pool=0x50000000, block_table=0x60000000, out=0x70000000, workspace=0x80000000)
_ROWS_Q = 11 * 8 * 128 * 2


@pytest.mark.parametrize("fused", [False, True, "step"])
@pytest.mark.parametrize("over,culprit", [
    (dict(out=_BASES["q"] + 16), "q"),
    (dict(out=_BASES["q"] - _ROWS_Q + 16), "q"),                 # tail of out over the head of q
    (dict(out=_BASES["k_pool"] + 4096), "k_pool"),
    (dict(out=_BASES["block_table"] - 64), "block_table"),
    (dict(out=_BASES["workspace"] + (1 << 20)), "workspace"),
    (dict(lse=_BASES["v_new"] + 4), "v_new"),
    (dict(lse=_BASES["out"] + 512), "lse"),                       # out and lse overlap
])
def test_outputs_that_alias_inputs_are_rejected(fused, over, culprit):
    args = dict(_BASES, workspace_bytes=1 << 24)
    args.update(over)
    assert _extend(fused=fused, **args) == L.CW_ERR_ALIAS
    msg = lib().cw_last_error_message().decode()
    assert culprit in msg and "overlaps" in msg, msg


def test_decode_output_alias_is_rejected():
    lp = np.array([10, 20], dtype=np.int32)
    r = lib().cw_decode_attention(
        _BASES["q"], _BASES["k_new"], _BASES["v_new"], _BASES["k_pool"], _BASES["v_pool"], None,
        None, _BASES["block_table"], 4, 100, lp.ctypes.data, 2, 2, 4, 128, 16, 0.088, 0,
        _BASES["k_new"] + 128, None, _BASES["workspace"], 1 << 24, None)
    assert r == L.CW_ERR_ALIAS and b"k_new" in lib().cw_last_error_message()


def test_plan_larger_than_a_staging_slot_is_rejected_before_any_gpu_work():
    # 20000 one-token decodes x 8 kv heads = 160000 work items: a 5 MB plan, more than
    # one 4 MiB staging slot (the ring is never grown)
    n = 20000
    lp = np.zeros(n, dtype=np.int32)
    gb = 1 << 30
    st = lib().cw_decode_attention(FAKE, FAKE + gb, FAKE + 2 * gb, FAKE + 3 * gb, FAKE + 4 * gb,
                                   None, None, FAKE + 5 * gb, 1, 1, lp.ctypes.data, n, 8, 4, 128,
                                   16, 0.088, 0, FAKE + 6 * gb, None, FAKE + 7 * gb, 1 << 29, None)
    assert st == L.CW_ERR_UNSUPPORTED
    assert "staging slot" in lib().cw_last_error_message().decode()


@pytest.mark.parametrize("header", ["cw.h", "cw_policy.h", "cw_ceiling.h"])
@pytest.mark.parametrize("lang", ["c", "c++"])
def test_header_compiles_alone(header, lang, tmp_path):
    """Each public header compiles on its own as C11 and as C++17 (plain host
    compilers, no HIP compiler), so a C caller can use the boundary directly."""
    import shutil
    import subprocess
    cc = shutil.which("gcc" if lang == "c" else "g++")
    if cc is None:
        pytest.skip("no host compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    src = tmp_path / "use.c"
    src.write_text(f'#include "{header}"\nint main(void) {{ return 0; }}\n')
    std = "-std=c11" if lang == "c" else "-std=c++17"
    r = subprocess.run([cc, std, "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I",
                        os.path.join(root, "include"), "-I", "/opt/rocm/include", "-fsyntax-only",
                        "-x", lang, str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
