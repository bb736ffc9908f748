"""Build libmgi.so: the engine's host core and HIP kernels for gfx950.

Run as ``python -m paper_1907_01989_amd.build_lib``; the shared library is
written next to this file, where the Python binding loads it.

``--sanitize`` builds ``libmgi_asan.so`` instead: the host code instrumented
with AddressSanitizer and UndefinedBehaviorSanitizer (device code is built as
usual).  Load it by setting MGI_LIB_PATH, with the ASan runtime preloaded,
for the CPU test tiers:

  MGI_LIB_PATH=paper_1907_01989_amd/libmgi_asan.so \
  LD_PRELOAD=$(/opt/rocm/llvm/bin/clang -print-file-name=libclang_rt.asan-x86_64.so) \
  ASAN_OPTIONS=detect_leaks=0 UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
  python -m pytest tests -m "not gpu"
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libmgi.so")
LIB_ASAN = os.path.join(HERE, "libmgi_asan.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["mgi_graph.cpp", "mgi_planner.cpp", "mgi_finalize.cpp", "mgi_runtime.cpp",
           "gemm.hip", "ops.hip", "dwpw.hip", "pwdw.hip", "stemdw.hip", "irb.hip"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Wall",
          # packed fp32 instructions are kept out of every device code object
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(HERE, "..", "include")]


# host-side sanitizers only: each -fsanitize applies to the host compilation
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]


def _compile(src: str, sanitize: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ("_asan.o" if sanitize else ".o"))
    cmd = [HIPCC] + COMMON + (SANITIZE if sanitize else []) + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, sanitize: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(lambda src: _compile(src, sanitize), SOURCES))
    out = LIB_ASAN if sanitize else LIB
    tmp = out + f".tmp{os.getpid()}"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if sanitize:
        cmd[3:3] = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-shared-libsan"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv[1:])
    sys.exit(0)
