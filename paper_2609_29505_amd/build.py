"""Build libsgd.so (HIP kernels + C ABI) for gfx950 with hipcc.

    python -m paper_2609_29505_amd.build        # from the repository root

Objects go to ``paper_2609_29505_amd/_build``; the library to
``paper_2609_29505_amd/lib/libsgd.so``.
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
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libsgd.so")

SOURCES = ["api.cpp", "dynamic.cpp", "schedule.cpp", "gemm.hip", "gemm_bf16.hip", "attention.hip", "norm.hip", "elementwise.hip", "spectral.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    "-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}",
    # packed fp32 instructions stay off: the compiler would otherwise pair fp32 math
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
    "-Wno-unused-result",
]


def _spills(remarks: str) -> list:
    """Kernels whose resource-usage remarks report spilled registers."""
    out, name = [], None
    for line in remarks.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:", 1)[1].split("[")[0].strip()
        elif "Spill:" in line:
            n = line.split("Spill:", 1)[1].split("[")[0].strip()
            if n.isdigit() and int(n) > 0:
                out.append(f"{name}: {line.split('remark:', 1)[-1].split('[')[0].strip()}")
    return out


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd.append("-Rpass-analysis=kernel-resource-usage")
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    # every kernel keeps its registers: a spill goes through scratch memory in the hot loops
    spills = _spills(r.stderr)
    if spills:
        raise RuntimeError(f"register spills in {src}:\n" + "\n".join(spills))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    workers = min(len(SOURCES), max(1, min(os.cpu_count() or 1, 16)))
    with ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
