"""Build the HIP/C++ library ``libppconv.so`` in-tree for gfx950.

    python -m paper_2004_11250_amd.build            # build (always recompiles)
    python -m paper_2004_11250_amd.build --host     # also the g++-only packer library

Every HIP translation unit is compiled with packed-FP32 instructions disabled
(``-Xclang -target-feature -Xclang -packed-fp32-ops``); the host pass warns
that it does not know the feature, which is harmless.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libppconv.so")
HOST_LIB = os.path.join(PKG, "libppconv_host.so")
OBJDIR = os.path.join(PKG, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# -structurizecfg-skip-uniform-regions: the pattern dispatch of the pruned
# conv is a wave-uniform branch tree; left unstructurized it needs no
# accumulator copies at the joins (the structurized form duplicates them).
# -simplifycfg-sink-common=false: otherwise the eight pattern cases, which
# have the same shape, are merged into one FMA block fed by register copies.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Xclang", "-target-feature",
             "-Xclang", "-packed-fp32-ops", "-mllvm", "-structurizecfg-skip-uniform-regions",
             "-mllvm", "-simplifycfg-sink-common=false", "-Wno-pass-failed", f"-I{INCLUDE}", f"-I{CSRC}"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    objs = []
    jobs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        for s in srcs:
            o = os.path.join(OBJDIR, os.path.basename(s) + ".o")
            objs.append(o)
            cmd = [HIPCC] + HIP_FLAGS + (["-x", "hip"] if s.endswith(".hip") else []) + ["-c", s, "-o", o]
            jobs.append(ex.submit(_run, cmd))
        for j in jobs:
            out = j.result()
            if verbose and out.strip():
                print(out)
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs)
    os.replace(tmp, LIB)
    return LIB


def build_host() -> str:
    """The packer, the pruning projections and blob validation alone, built
    with g++ (no HIP)."""
    tmp = HOST_LIB + ".tmp"
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", f"-I{INCLUDE}", f"-I{CSRC}",
          os.path.join(CSRC, "pack.cpp"), os.path.join(CSRC, "project.cpp"), "-o", tmp])
    os.replace(tmp, HOST_LIB)
    return HOST_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    if "--host" in sys.argv:
        print(build_host())
