"""Build libaep.so (the gfx950 HIP kernels + the C ABI) in-tree with hipcc.

    python -m paper_2505_08944_amd.build        # or build() from Python

Every source is compiled for gfx950 only.  Packed-FP32 instruction selection
is switched off (``-packed-fp32-ops``): all float math is plain scalar VALU or
MFMA.  Objects go to ``_build/``; the library lands next to this file.
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
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libaep.so")

SOURCES = ["api.hip", "k_route.hip", "k_rebatch.hip", "k_ffn.hip", "k_combine.hip", "k_pool.hip", "sched.hip"]
ARCH = "gfx950"
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libaep)")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host pass does not know the packed-fp32 feature and says so; drop that noise
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    return r.returncode, out


def build(verbose: bool = False, jobs: int = 0) -> str:
    """Compile every source and link libaep.so; returns the library path."""
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmds.append([cc, *CFLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
    jobs = jobs or min(len(cmds), os.cpu_count() or 4, 16)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        results = list(ex.map(_run, cmds))
    for cmd, (rc, out) in zip(cmds, results):
        if verbose or rc:
            sys.stderr.write(" ".join(cmd) + "\n" + out + ("\n" if out else ""))
        if rc:
            raise RuntimeError(f"hipcc failed on {cmd[-3]}")
    tmp = LIB + ".tmp"
    rc, out = _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp,
                    *[c[-1] for c in cmds]])
    if verbose or rc:
        sys.stderr.write(out + ("\n" if out else ""))
    if rc:
        raise RuntimeError("linking libaep.so failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
