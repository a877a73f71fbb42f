"""Build libmeq.so (HIP kernels for gfx950 + the C ABI) in-tree with hipcc.

Usage: ``python -m paper_2609_35701_amd.build`` (or ``__graft_entry__.build()``).
The library is written next to this file so that it travels with the source tree.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libmeq.so")

ARCH = "gfx950"
# Packed-fp32 VALU forms are disabled for all device code (plain float code only).
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", f"-I{INCLUDE}", f"-I{CSRC}",
          "-fvisibility=hidden", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# Per-source extra flags.
SOURCES = {
    "k_ns_gemm.hip": [],
    "k_stream.hip": [],
    "k_aux.hip": [],
    "meq_api.cpp": [],
    "meq_static.hip": [],
}


def hipcc() -> str:
    path = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the MeqMuon HIP library cannot be built")
    return path


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libmeq.so; returns the library path."""
    cc = hipcc()
    with tempfile.TemporaryDirectory(prefix="meq_build_") as tmp:
        objs = []
        for src, extra in SOURCES.items():
            obj = os.path.join(tmp, src + ".o")
            lang = ["-x", "hip"] if src.endswith(".hip") else []
            cmd = [cc, *COMMON, *extra, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            res = subprocess.run(cmd, stdout=subprocess.PIPE if not verbose else None,
                                 stderr=subprocess.STDOUT if not verbose else None, text=True)
            if res.returncode != 0:
                raise RuntimeError(f"hipcc failed on {src}:\n{res.stdout or ''}")
            objs.append(obj)
        out_tmp = LIB + ".tmp"
        # -z defs: an entry point whose kernel source is missing fails here, not at load time
        cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,-z,defs", *objs, "-o", out_tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
