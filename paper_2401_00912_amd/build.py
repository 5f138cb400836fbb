"""Build libsla.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2401_00912_amd.build          # compile every source, link

Always recompiles (the caller decides when a build is due).  The library lands
next to this file so that it travels with the source tree.
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
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsla.so")
SOURCES = ["sla_builder.hip", "sla_attn.hip", "sla_proj.hip", "sla_proj_bwd.hip", "sla_cwi.hip", "sla_naive.hip", "sla_xca.hip", "sla_api.hip"]
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-fvisibility=hidden",
    # never emit packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-I", CSRC,
]


def hipcc() -> str:
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found; a ROCm toolchain is required to build libsla")
    return exe


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False, defines=(), out: str = LIB, build_dir: str = BUILD) -> str:
    """Compile and link.  `defines` (e.g. ["SLA_GRID_WGS=1024"]) and `out` /
    `build_dir` exist for building tuning variants next to the default library."""
    os.makedirs(build_dir, exist_ok=True)
    cc = hipcc()
    objs = [os.path.join(build_dir, s.replace(".hip", ".o")) for s in SOURCES]
    dflags = [f"-D{d}" for d in defines]
    cmds = [[cc, *HIPCC_FLAGS, *dflags, "-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
    with ThreadPoolExecutor(max_workers=len(cmds)) as ex:
        for cmd, err in zip(cmds, ex.map(_run, cmds)):
            if verbose:
                print(" ".join(cmd))
            if err.strip() and verbose:
                print(err)
    tmp = out + ".tmp"
    link = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    _run(link)
    os.replace(tmp, out)
    if verbose:
        print("built", out)
    return out


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
