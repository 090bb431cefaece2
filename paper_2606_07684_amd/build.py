"""Build the SCD codec's HIP library (libscd.so) in-tree for gfx950.

Usage: ``python -m paper_2606_07684_amd.build`` or ``build()`` from Python.  Compiles every HIP and
C++ source under ``csrc/`` with hipcc into ``paper_2606_07684_amd/libscd.so``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG_DIR, "csrc")
ROOT = os.path.dirname(PKG_DIR)
LIB_PATH = os.path.join(PKG_DIR, "libscd.so")
ARCH = "gfx950"

SOURCES = ["scd_gemm.hip", "scd_patch.hip", "scd_decode.hip", "scd_encode.hip", "scd_fit.hip",
           "scd_fold.hip", "scd_api.cpp"]

FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    # never let the compiler form packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the SCD library needs ROCm's hipcc to build")


def _filter(text: str) -> str:
    # hipcc's host pass warns that it does not know the packed-fp32 feature flag; that is expected
    return "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)


def build(verbose: bool = False) -> str:
    """Compile libscd.so (always recompiles) and return its path.

    Every source is compiled to an object in its own hipcc process (in parallel), then the objects
    are linked into one shared library."""
    cc = hipcc()
    with tempfile.TemporaryDirectory(prefix="scd_build_") as tmpdir:
        procs = []
        objs = []
        for src in SOURCES:
            obj = os.path.join(tmpdir, src + ".o")
            cmd = [cc, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
        failed = []
        for src, proc in procs:
            out = _filter(proc.communicate()[0])
            if proc.returncode != 0:
                failed.append(f"{src} ({proc.returncode}):\n{out}")
            elif verbose and out.strip():
                print(out)
        if failed:
            raise RuntimeError("hipcc failed: " + "\n".join(failed))
        tmp = LIB_PATH + ".tmp"
        cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"link failed ({res.returncode}):\n{_filter(res.stdout + res.stderr)}")
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
