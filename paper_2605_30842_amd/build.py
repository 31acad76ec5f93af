"""Build libcomem_attn.so (HIP, gfx950) in-tree with hipcc.

Usage: python -m paper_2605_30842_amd.build   (or call build_library()).
Every call compiles from source; nothing is cached between calls.
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
LIB_NAME = "libcomem_attn.so"
SOURCES = ["api.cpp", "api_prefill.cpp", "kernel_mfma.hip", "kernel_valu.hip", "kernel_append.hip", "kernel_prefill.hip",
           "noalloc.hip", "cost_model.cpp"]
PROBE_LIB_NAME = "libcomem_probe.so"
PROBE_SOURCES = ["probe.hip"]
ARCH = "gfx950"

# Packed fp32 VALU instructions are kept out of the generated code.
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature and says so; drop that line only
    err = "\n".join(line for line in r.stderr.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def _build_one(name, sources, out_dir, verbose):
    hipcc = _hipcc()
    obj_dir = os.path.join(ROOT, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    objs = []
    cmds = []
    for src in sources:
        obj = os.path.join(obj_dir, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmds.append([hipcc, *HIP_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", *lang, "-c",
                     os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=len(cmds)) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    out = os.path.join(out_dir, name)
    tmp = out + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, out)
    return out


def build_library(out_dir: str = PKG, verbose: bool = False) -> str:
    """Build the decode-attention library and the measurement probe library; return the former's path."""
    with ThreadPoolExecutor(max_workers=2) as ex:
        main = ex.submit(_build_one, LIB_NAME, SOURCES, out_dir, verbose)
        probe = ex.submit(_build_one, PROBE_LIB_NAME, PROBE_SOURCES, out_dir, verbose)
        probe.result()
        return main.result()


if __name__ == "__main__":
    print(build_library(verbose="-v" in sys.argv))
