"""Build libcas.so (HIP for gfx950) in-tree with hipcc.

    python -m paper_2606_04557_amd.build
    python -m paper_2606_04557_amd.build --sanitize

--sanitize builds _build_san/libcas_san.so with AddressSanitizer and
UndefinedBehaviorSanitizer on the host code only (device code is compiled as
usual), for running the host-side tests (validation, planning) under the
sanitizers without a GPU:

    CAS_LIB=_build_san/libcas_san.so LD_PRELOAD=<clang asan runtime>:$LD_PRELOAD \
        ASAN_OPTIONS=detect_leaks=0 python -m pytest tests/test_host_lib.py
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG, "libcas.so")
SAN_DIR = os.path.join(ROOT, "_build_san")
SAN_LIB_PATH = os.path.join(SAN_DIR, "libcas_san.so")
# Host-only sanitizers: each -fsanitize= goes to the host compilation alone.
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
             "-O1", "-g"]
SOURCES = ["cas_api.cpp", "cas_pool.cpp", "cas_fwd.hip", "cas_bwd.hip", "cas_bf16.hip", "cas_adam.hip", "cas_decode.hip",
           "cas_noalloc.hip"]
ARCH = "gfx950"

# -packed-fp32-ops: no packed fp32 ALU instructions are generated on gfx950.
COMMON_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


# The bf16 kernels produce no NaN of their own (masked scores are -inf, never
# NaN), so max/min need not quiet signalling NaNs: without this every fmaxf
# on an MFMA result costs an extra canonicalising instruction.
#
# The optimizer step rounds once per operation in a documented order, so no
# multiply-add contraction there.
FILE_FLAGS = {"cas_bf16.hip": ["-fno-honor-nans"], "cas_adam.hip": ["-ffp-contract=off"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # The host pass does not know the gfx950 feature flag; drop that notice.
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile every source and link libcas.so (or, with sanitize, the
    host-sanitized _build_san/libcas_san.so); returns its path."""
    cc = hipcc()
    bdir, lib = (SAN_DIR, SAN_LIB_PATH) if sanitize else (BUILD_DIR, LIB_PATH)
    extra = SAN_FLAGS if sanitize else []
    os.makedirs(bdir, exist_ok=True)
    objs = []
    jobs = []
    for src in SOURCES:
        obj = os.path.join(bdir, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        jobs.append([cc, *COMMON_FLAGS, *FILE_FLAGS.get(src, []), *extra, "-c", os.path.join(CSRC, src),
                     "-o", obj])
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        for out in ex.map(_run, jobs):
            if verbose and out.strip():
                print(out)
    tmp = lib + ".tmp"
    link_extra = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-shared-libasan"] if sanitize else []
    out = _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *link_extra, "-o", tmp, *objs])
    if verbose and out.strip():
        print(out)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
