"""Build the gfx950 shared library ``_lib/libmoe_stage.so`` with hipcc.

Run as ``python -m paper_2607_19539_amd.build``.  Cross-compiles without a GPU.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "libmoe_stage.so")
SOURCES = ["kernels.hip", "combine.hip", "plan_device.hip", "plan.cpp", "api.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# -packed-fp32-ops: never emit packed fp32 VALU ops (v_pk_add/mul/fma_f32).
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-command-line-argument",
          f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]


def build(verbose: bool = False) -> str:
    os.makedirs(LIBDIR, exist_ok=True)
    with tempfile.TemporaryDirectory(prefix="moe_build_") as tmp:
        objs = []
        for src in SOURCES:
            obj = os.path.join(tmp, src + ".o")
            # api.cpp holds the no-allocation entry point's device array, so it is HIP source too.
            lang = ["-x", "hip"] if src.endswith(".hip") or src == "api.cpp" else []
            cmd = [HIPCC, *COMMON, *DEVICE_FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
            _run(cmd, verbose)
            objs.append(obj)
        out_tmp = LIB + ".tmp"
        _run([HIPCC, *DEVICE_FLAGS, "-shared", "-fPIC", *objs, "-o", out_tmp], verbose)
        os.replace(out_tmp, LIB)
    return LIB


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = ("packed-fp32-ops", "is not a recognized feature")
    err = "\n".join(l for l in (r.stderr or "").splitlines() if not any(n in l for n in noise))
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
