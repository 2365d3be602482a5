"""Build libember.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

Run ``python -m paper_2607_01455_amd.build`` (or ``__graft_entry__.build()``).
The library is written next to this file and loaded from there.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libember.so")
SOURCES = ["ember_kernels.hip", "ember_coalesce.hip", "ember_lmhead.hip", "ember_probe.hip", "ember_api.cpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed-fp32 VALU forms are disabled for all device code; hipcc's host pass
# warns that it does not know the feature, which is harmless.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd, verbose: bool) -> None:
    p = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in p.stderr.splitlines() if noise not in l)
    if p.returncode != 0:
        sys.stderr.write(err + "\n")
        raise RuntimeError(f"build step failed ({p.returncode}): {' '.join(cmd)}")
    if verbose and err.strip():
        sys.stderr.write(err + "\n")


def build(verbose: bool = False, extra_flags=(), out: str = LIB) -> str:
    """Compile and link the library to `out`; extra_flags go to every compile
    (e.g. -O2, or -save-temps to inspect the code)."""
    objs = []
    tag = str(abs(hash((tuple(extra_flags), out))))
    try:
        for src in SOURCES:
            obj = os.path.join(CSRC, f"{src}.{tag}.o")
            objs.append(obj)
            lang = ["-x", "hip"] if src.endswith(".hip") else []
            cmd = [HIPCC, f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
                   "-ffp-contract=fast", "-Wall", "-Wno-unused-function",
                   "-I", INCLUDE, "-I", CSRC, *DEVICE_FLAGS, *extra_flags, *lang, "-c",
                   os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            _run(cmd, verbose)
        tmp = out + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        _run(cmd, verbose)
        os.replace(tmp, out)
    finally:
        # objects are intermediate: none is left behind, also when a step fails
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
