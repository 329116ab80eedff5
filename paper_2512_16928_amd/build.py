"""Builds libdion2.so (the HIP kernels and the C ABI) for gfx950, in-tree.

    python -m paper_2512_16928_amd.build [--jobs N] [--verbose] [--sanitize-host]

Every source is compiled with hipcc for gfx950 only; the shared library is
written next to this file, where the Python binding loads it from.

--sanitize-host builds a copy whose host code (validation, planning,
workspace layout, launch set-up) carries AddressSanitizer and
UndefinedBehaviorSanitizer checks, the device code unchanged, into
_build/san/libdion2.so. The CPU tests run against it with

    ASAN_OPTIONS=detect_leaks=0 \
    LD_PRELOAD=$(clang -print-file-name=libclang_rt.asan-x86_64.so) \
    python -m pytest tests -m "not gpu" --dion2-lib _build/san/libdion2.so
"""
from __future__ import annotations

import argparse
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
LIB = os.path.join(PKG, "libdion2.so")
ARCH = "gfx950"

SOURCES = ["dion2_api.hip", "k_momentum.hip", "k_select.hip", "k_gather.hip",
           "k_gemm.hip", "k_apply.hip"]

# -ffp-contract=off: the elementwise stages must round exactly as written
# (fl32(M + G), fl32(mu * M), fp64 products then differences).
# -packed-fp32-ops off: no packed fp32 VALU instructions are generated.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libdion2.so)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


# host code only: each -fsanitize= goes to the host compilation
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_LIB = os.path.join(BUILD, "san", "libdion2.so")


def build(jobs: int = 8, verbose: bool = False, sanitize_host: bool = False) -> str:
    out_dir = os.path.dirname(SAN_LIB) if sanitize_host else BUILD
    lib = SAN_LIB if sanitize_host else LIB
    extra = SAN_FLAGS if sanitize_host else []
    os.makedirs(out_dir, exist_ok=True)
    cc = hipcc()
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmds.append([cc, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=max(1, min(jobs, len(cmds)))) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = lib + ".tmp"
    link_extra = ["-shared-libsan", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
                  "-fsanitize=undefined"] if sanitize_host else []
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *link_extra, "-o", tmp, *objs], verbose)
    os.replace(tmp, lib)
    return lib


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--jobs", type=int, default=8)
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--sanitize-host", action="store_true",
                    help="host code with AddressSanitizer and UBSan, into _build/san/libdion2.so")
    args = ap.parse_args(argv)
    print(build(args.jobs, args.verbose, args.sanitize_host))


if __name__ == "__main__":
    sys.exit(main())
