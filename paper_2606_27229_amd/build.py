"""Build libcarve.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

The library is built in-tree next to this file so it travels with the
repository; nothing is installed.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libcarve.so")
# (source, object name, extra flags): carve_variant.hip is compiled once per
# layer variant (decay given / formed in the kernels x full / scalar write
# gate, and the input activations inside the layer)
SOURCES = [("carve_abi.hip", "carve_abi", []), ("carve_fwd_chain.hip", "carve_fwd_chain", []),
           ("carve_bwd.hip", "carve_bwd", []), ("carve_norm.hip", "carve_norm", [])] + [
    ("carve_variant.hip", f"carve_variant{v}", [f"-DCARVE_VARIANT={v}"]) for v in range(5)]

BUILD = os.path.join(HERE, "_build")
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed f32 ops are kept off: hipcc forms them from plain float code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for p in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if p and os.path.exists(p):
            return p
    return "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
    return r.returncode


def build(verbose: bool = False) -> str:
    """Compile every translation unit (in parallel) and link libcarve.so."""
    os.makedirs(BUILD, exist_ok=True)
    objs, cmds = [], []
    for src, name, extra in SOURCES:
        obj = os.path.join(BUILD, name + ".o")
        objs.append(obj)
        cmds.append([hipcc()] + HIPCC_FLAGS + extra + ["-c", "-o", obj, os.path.join(CSRC, src)])
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
        rcs = list(ex.map(lambda c: _run(c, verbose), cmds))
    if any(rcs):
        raise RuntimeError("hipcc failed compiling libcarve")
    tmp = LIB + ".tmp"
    if _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs, verbose):
        raise RuntimeError("hipcc failed linking libcarve.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
