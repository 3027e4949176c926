"""Build libepikv.so (gfx950) in-tree with hipcc, and beside it the
benchmark's streaming-copy probe libcopyprobe.so (measurement only; not part
of the eviction step's C ABI).

    python -m paper_2606_26472_amd.build
    python -m paper_2606_26472_amd.build --host-asan   # _build/asan/libepikv.so

The second form instruments the host code (argument validation, layouts,
launch set-up) with AddressSanitizer; the device code is built as usual.  It
is meant for the C-ABI validation tests on a machine without a GPU:

    EPIKV_LIB=_build/asan/libepikv.so ASAN_OPTIONS=detect_leaks=0 \
    LD_PRELOAD=$(ls /opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so) \
    python -m pytest tests/test_abi.py -k "not only_the_c_abi"
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libepikv.so")
PROBE_LIB = os.path.join(PKG, "libcopyprobe.so")
PROBE_SOURCES = ["copy_probe.hip"]

SOURCES = ["epikv_api.hip", "score_hs.hip", "score_lagkv.hip", "zscore.hip",
           "select.hip", "compact.hip", "compact_inplace.hip", "score_tokens.hip",
           "score_select.hip", "select_multi.hip", "noalloc.hip"]

ARCH = "gfx950"
CXXFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-fvisibility=hidden", "-Wall", "-Wno-unused-function",
    # no packed fp32 instructions (v_pk_*_f32) anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc",
                 shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libepikv)")


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("command failed:\n" + " ".join(cmd) + "\n"
                           + r.stdout + r.stderr)
    return r


ASAN_HOST = ["-Xarch_host", "-fsanitize=address",
             "-Xarch_host", "-fno-omit-frame-pointer"]


def build(verbose: bool = False, host_asan: bool = False) -> str:
    """Compile every source and link libepikv.so; returns its path."""
    cc = hipcc()
    out_dir = os.path.join(BUILD, "asan") if host_asan else BUILD
    lib = os.path.join(out_dir, "libepikv.so") if host_asan else LIB
    flags = CXXFLAGS + (ASAN_HOST if host_asan else [])
    os.makedirs(out_dir, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        cmd = [cc, *flags, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        _run(cmd)
        return obj

    def link(objs, target):
        tmp = target + ".tmp"
        # (an instrumented library takes its sanitizer runtime from
        # LD_PRELOAD)
        cmd = [cc, "-shared", f"--offload-arch={ARCH}", "-fvisibility=hidden",
               "-o", tmp, *objs]
        if verbose:
            print(" ".join(cmd), flush=True)
        _run(cmd)
        os.replace(tmp, target)

    todo = SOURCES + ([] if host_asan else PROBE_SOURCES)
    with ThreadPoolExecutor(max_workers=min(8, len(todo))) as ex:
        objs = dict(zip(todo, ex.map(compile_one, todo)))
    link([objs[s] for s in SOURCES], lib)
    if not host_asan:
        link([objs[s] for s in PROBE_SOURCES], PROBE_LIB)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, host_asan="--host-asan" in sys.argv))
