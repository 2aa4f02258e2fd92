"""Builds libcw.so (the C-ABI library) in-tree with hipcc for gfx950.

Usage: python -m paper_2606_16824_amd.build [--jobs N] [--sanitize]
Every .hip / .cpp under csrc/ is compiled to an object in _build/ (in
parallel), then linked into paper_2606_16824_amd/libcw.so; the C programs under
tests/native/ are then compiled against it (build_native_tests).

--sanitize builds the host side of every source with AddressSanitizer and
UndefinedBehaviorSanitizer (device code is built as usual) into
_build/sanitize/libcw.so, for running the CPU tests (argument validation,
planner, host policy simulator) under the sanitizers:

    python -m paper_2606_16824_amd.build --sanitize
    LD_PRELOAD=$(hipcc -print-file-name=libclang_rt.asan-x86_64.so) \
    ASAN_OPTIONS=detect_leaks=0 CW_LIBRARY=_build/sanitize/libcw.so \
    python -m pytest tests -m "not gpu"
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libcw.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Wno-unused-function", "-Wno-unused-command-line-argument",
    # no packed-FP32 VALU instructions in generated device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def sources():
    out = []
    for dirpath, _, files in os.walk(CSRC):
        for f in sorted(files):
            if f.endswith((".hip", ".cpp")):
                out.append(os.path.join(dirpath, f))
    return sorted(out)


# host-side sanitizers only: each -fsanitize= applies to the host pass
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]


def _obj(src, build_dir=BUILD):
    rel = os.path.relpath(src, CSRC).replace(os.sep, "__")
    return os.path.join(build_dir, rel + ".o")


def _compile(src, extra=(), build_dir=BUILD):
    obj = _obj(src, build_dir)
    lang = ["-x", "hip"]
    cmd = [HIPCC, *COMMON, *extra, *lang, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    return src, r.returncode, r.stdout + r.stderr, cmd


def build(jobs: int = 8, verbose: bool = False, sanitize: bool = False) -> str:
    build_dir = os.path.join(BUILD, "sanitize") if sanitize else BUILD
    lib_path = os.path.join(build_dir, "libcw.so") if sanitize else LIB
    extra = SANITIZE if sanitize else []
    os.makedirs(build_dir, exist_ok=True)
    srcs = sources()
    errors = []
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        for src, rc, log, cmd in ex.map(lambda s_: _compile(s_, extra, build_dir), srcs):
            if verbose or rc != 0:
                print(" ".join(cmd), file=sys.stderr)
            # the host pass does not know the packed-fp32 feature; drop that warning
            log = "\n".join(l for l in log.splitlines() if "packed-fp32-ops" not in l)
            if log.strip() and (verbose or rc != 0):
                print(log, file=sys.stderr)
            if rc != 0:
                errors.append(src)
    if errors:
        raise RuntimeError("hipcc failed for: " + ", ".join(errors))
    tmp = lib_path + ".tmp"
    link_extra = ["-fsanitize=address,undefined", "-shared-libsan"] if sanitize else []
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *link_extra, "-o", tmp,
           *[_obj(s, build_dir) for s in srcs]]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        print(" ".join(cmd), "\n", r.stdout, r.stderr, file=sys.stderr)
        raise RuntimeError("link of libcw.so failed")
    os.replace(tmp, lib_path)
    return lib_path


NATIVE = os.path.join(ROOT, "tests", "native")


def build_native_tests() -> list:
    """Compiles the C programs under tests/native/ (host code that drives the C
    ABI with no Python) against libcw.so into tests/native/<name>.bin."""
    cc = shutil.which("gcc") or "gcc"
    out = []
    for f in sorted(os.listdir(NATIVE)) if os.path.isdir(NATIVE) else []:
        if not f.endswith(".c"):
            continue
        exe = os.path.join(NATIVE, f[:-2] + ".bin")
        cmd = [cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
               "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
               os.path.join(NATIVE, f), "-L", PKG, "-lcw", "-L", "/opt/rocm/lib", "-lamdhip64", "-lm",
               "-Wl,-rpath,$ORIGIN/../../paper_2606_16824_amd", "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            print(" ".join(cmd), "\n", r.stdout, r.stderr, file=sys.stderr)
            raise RuntimeError(f"build of {f} failed")
        out.append(exe)
    return out


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=8)
    ap.add_argument("-v", "--verbose", action="store_true")
    ap.add_argument("--sanitize", action="store_true",
                    help="host-side ASan + UBSan build into _build/sanitize/libcw.so")
    a = ap.parse_args()
    print(build(a.jobs, a.verbose, a.sanitize))
    if not a.sanitize:
        print("\n".join(build_native_tests()))
