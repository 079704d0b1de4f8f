"""Build libdmc.so (gfx950) in-tree with hipcc.

Usage: python paper_2403_09636_amd/csrc/build.py [--verbose]
(run by path: importing the package first would load the library it builds)
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libdmc.so")
SOURCES = [os.path.join(HERE, "dmc_api.cpp"), os.path.join(HERE, "dmc_kernels.hip"),
           os.path.join(HERE, "dmc_prompt.hip"), os.path.join(HERE, "dmc_train.hip")]
ARCH = "gfx950"

# Packed-fp32 VALU forms are disabled for every HIP translation unit.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-function", "-Wno-unknown-warning-option",
             "-I", os.path.join(ROOT, "include"), "-I", HERE]


def hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = (res.stdout + res.stderr).strip()
    # hipcc's host pass does not know the packed-fp32 target feature; that warning is expected.
    lines = [ln for ln in out.splitlines() if "packed-fp32-ops" not in ln and ln.strip()]
    return res.returncode, lines


def build(verbose: bool = False) -> str:
    """Compile every source to an object in parallel, then link libdmc.so."""
    from concurrent.futures import ThreadPoolExecutor
    tmp = LIB + f".tmp{os.getpid()}"
    with tempfile.TemporaryDirectory(prefix="dmc_build_") as objdir:
        objs = [os.path.join(objdir, os.path.basename(src) + ".o") for src in SOURCES]
        cmds = [[hipcc(), *HIP_FLAGS, "-c", "-o", obj, src] for src, obj in zip(SOURCES, objs)]
        with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
            results = list(ex.map(lambda c: _run(c, verbose), cmds))
        failed = [ln for rc, lines in results if rc != 0 for ln in lines]
        if failed:
            raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
        rc, lines = _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-o", tmp, *objs], verbose)
        if rc != 0:
            raise RuntimeError("link failed:\n" + "\n".join(lines))
    if verbose:
        for _, ls in results:
            if ls:
                print("\n".join(ls))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="--verbose" in sys.argv))
