"""Build the host-only check library: the planner of libmeq.so (meq_api.cpp) linked with the
recording launchers of launch_record.cpp instead of the HIP kernels, compiled by g++ (no device
code), optionally with AddressSanitizer and UndefinedBehaviorSanitizer.  Test infrastructure."""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2609_35701_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def compiler() -> str:
    cc = shutil.which("g++")
    if not cc:
        raise RuntimeError("g++ not found")
    return cc


def build(out_path: str, sanitize: bool) -> str:
    cmd = [compiler(), "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
           f"-I{ROCM}/include", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", "-Wno-unused-result",
           *(SANITIZE if sanitize else []),
           os.path.join(CSRC, "meq_api.cpp"), os.path.join(HERE, "launch_record.cpp"),
           f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", out_path]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError("host check build failed:\n" + " ".join(cmd) + "\n" + res.stdout)
    return out_path


def sanitizer_preload() -> str:
    """The sanitizer runtimes a non-instrumented Python must preload to load the instrumented library."""
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        p = subprocess.run([compiler(), f"-print-file-name={name}"], stdout=subprocess.PIPE, text=True).stdout.strip()
        if not os.path.isabs(p):
            raise RuntimeError(f"{name} not found")
        libs.append(os.path.realpath(p))
    return ":".join(libs)
