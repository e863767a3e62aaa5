"""Build the rosa HIP library (librosa.so) in-tree for gfx950 with hipcc.

    python -m paper_2607_01088_amd.build             # compile + link
    python -m paper_2607_01088_amd.build --sanitize  # librosa_san.so: host code
                                                     # under AddressSanitizer and
                                                     # UndefinedBehaviorSanitizer

The sanitized library checks the host side only (planner, validation, the
schedulers; device code is built as usual).  It is for CPU runs of the host
tests, with the sanitizer runtime preloaded and ROSA_LIB_PATH pointing at it:

    LD_PRELOAD=$(/opt/rocm/llvm/bin/clang -print-file-name=libclang_rt.asan-x86_64.so) \
    ASAN_OPTIONS=detect_leaks=0 ROSA_LIB_PATH=paper_2607_01088_amd/librosa_san.so \
    python -m pytest tests/test_abi_cpu.py tests/test_s1_batching.py tests/test_homogeneous_lib.py
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "librosa.so")
LIB_SAN = os.path.join(PKG, "librosa_san.so")
SOURCES = ["k_time.hip", "k_rows.hip", "k_gemm.hip", "k_attn.hip", "k_probe.hip", "k_prefill.hip", "rosa_api.cpp",
           "rosa_prefill.cpp", "rosa_sched.cpp"]
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wno-unused-result",
         # packed fp32 VALU ops stay disabled: compiler-formed packed fp32 forms are avoided
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in [shutil.which("hipcc"), "/opt/rocm/bin/hipcc"]:
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the rosa library needs ROCm's hipcc to build")


# Host-side sanitizers only: each -fsanitize is scoped to the host pass.
SAN_FLAGS = ["-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]


def _compile(src: str, san: bool = False) -> str:
    obj = os.path.join(BUILD + ("_san" if san else ""), os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *FLAGS, *(SAN_FLAGS if san else []), "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stderr}")
    return obj


def build(verbose: bool = True, sanitize: bool = False) -> str:
    out = LIB_SAN if sanitize else LIB
    os.makedirs(BUILD + ("_san" if sanitize else ""), exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda src: _compile(src, sanitize), SOURCES))
    tmp = out + ".tmp"
    cmd = [hipcc(), "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    if sanitize:
        cmd[2:2] = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(sanitize="--sanitize" in sys.argv[1:])
    sys.exit(0)
