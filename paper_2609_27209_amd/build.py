"""Build the HIP library ``liberc.so`` in-tree for gfx950.

    python -m paper_2609_27209_amd.build

Compiles ``csrc/erc_kernels.hip``, ``csrc/erc_draw.hip``, ``csrc/erc_probe.hip``,
``csrc/erc_static.hip`` and ``csrc/erc_host.cpp`` with
hipcc and links them into ``paper_2609_27209_amd/liberc.so``.  Packed fp32 instructions are disabled in
device code (``-packed-fp32-ops``); the host pass warns that it does not know the
feature, which is harmless.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "liberc.so")
ARCH = os.environ.get("ERC_OFFLOAD_ARCH", "gfx950")

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-pass-failed",
          "-Wno-unused-command-line-argument"]
DEVICE = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}")
    return r


def build(verbose: bool = False) -> str:
    """Compile and link ``liberc.so``; returns its path."""
    hipcc = _hipcc()
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = []
    jobs = []
    for name in ("erc_kernels", "erc_draw", "erc_probe", "erc_static"):
        objs.append(os.path.join(objdir, name + ".o"))
        jobs.append([hipcc, f"--offload-arch={ARCH}", *COMMON, *DEVICE, "-c",
                     os.path.join(CSRC, name + ".hip"), "-o", objs[-1]])
    objs.append(os.path.join(objdir, "erc_host.o"))
    jobs.append([hipcc, *COMMON, "-c", os.path.join(CSRC, "erc_host.cpp"), "-o", objs[-1]])
    with ThreadPoolExecutor(len(jobs)) as ex:
        for f in [ex.submit(_run, j, verbose) for j in jobs]:
            f.result()
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
