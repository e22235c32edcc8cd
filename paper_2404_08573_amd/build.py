"""Build libff.so for gfx950 in-tree with hipcc.

``python -m paper_2404_08573_amd.build`` (or ``__graft_entry__.build()``)
compiles every HIP/C++ source of the library.  Packed-fp32 instructions are
disabled for device code (the host pass prints a harmless warning that it
does not know the feature).

Per-lane arrays must stay in registers.  LLVM may otherwise move a
dynamically indexed one into LDS, indexed by the flat work-item id, which
every wave then computes from the workgroup size read out of the dispatch
packet in host memory (a many-microsecond stall when all CUs do it at once).
That promotion is switched off, so such an array would land in scratch
instead, and the build fails if any kernel reports scratch use.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libff.so")
SOURCES = ["ff_kernels.hip", "ff_api.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-disable-promote-alloca-to-lds",
         "-Wall", "-Wno-unused-function", f"-I{os.path.join(ROOT, 'include')}"]
KERNELS = "ff_kernels.hip"  # compiled with the resource-usage report


def scratch_users(report: str) -> list:
    """Kernels with a nonzero ScratchSize in hipcc's resource-usage remarks."""
    users, name = [], None
    for line in report.splitlines():
        if "remark: Function Name:" in line:
            name = line.split("Function Name:", 1)[1].split("[-Rpass")[0].strip()
        elif "ScratchSize [bytes/lane]:" in line and name:
            n = int(line.split("ScratchSize [bytes/lane]:", 1)[1].split()[0])
            if n:
                users.append((name, n))
    return users


def build(verbose: bool = False) -> str:
    objs = []
    for src in SOURCES:
        obj = os.path.join(CSRC, "_build", src + ".o")
        os.makedirs(os.path.dirname(obj), exist_ok=True)
        report = ["-Rpass-analysis=kernel-resource-usage"] if src == KERNELS else []
        cmd = [HIPCC, *FLAGS, *report, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        noise = ("is not a recognized feature for this target", "-Rpass-analysis=kernel-resource")
        err = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                        if not any(n in l for n in noise))
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{err}")
        if report:
            users = scratch_users(r.stderr)
            if users:
                raise RuntimeError("kernels using scratch memory (per-lane arrays out of "
                                   "registers):\n" + "\n".join(f"  {n}: {b} B/lane" for n, b in users))
        if err.strip() and verbose:
            print(err)
        objs.append(obj)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", f"--offload-arch={ARCH}", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
