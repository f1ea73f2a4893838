"""Build libcompactattn.so (and its debug variant libcompactattn_debug.so,
compiled with CA_DEBUG_CHECKS) in-tree with hipcc for gfx950."""
from __future__ import annotations

import glob
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libcompactattn.so")
DEBUG_LIB = os.path.join(PKG, "libcompactattn_debug.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # keep the compiler from forming packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


def build_library(verbose: bool = False, debug: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    out = DEBUG_LIB if debug else LIB
    tmp = out + ".tmp"
    extra = ["-DCA_DEBUG_CHECKS=1"] if debug else []
    cmd = [hipcc, *HIPCC_FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-o", tmp,
           *sources()]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    os.replace(tmp, out)
    return out


def build_all(verbose: bool = False) -> list:
    """Both libraries, compiled in parallel."""
    from concurrent.futures import ThreadPoolExecutor

    with ThreadPoolExecutor(2) as ex:
        jobs = [ex.submit(build_library, verbose, dbg) for dbg in (False, True)]
        return [j.result() for j in jobs]


if __name__ == "__main__":
    print(build_all(verbose=True))
