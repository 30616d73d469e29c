"""Build the gfx950 shared libraries in-tree with hipcc: libbcjr.so (the
C ABI of include/bcjr.h) and libissue_rates.so (the VALU issue-rate probe
the benchmark prices its roofline with).

libbcjr.so links two translation units: bcjr_capi.hip (the C ABI and every
kernel family) and bcjr_rot.hip (the rotating-exchange kernel of the
S = 65536, k = 2 fwd + dW call), which is compiled with the AMDGPU max-ilp
instruction scheduler; each object carries its own code object."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libbcjr.so")
# (source, extra compiler flags)
UNITS = [(os.path.join(CSRC, "bcjr_capi.hip"), []),
         (os.path.join(CSRC, "bcjr_rot.hip"), ["-mllvm", "-amdgpu-sched-strategy=max-ilp"])]
SOURCES = [u[0] for u in UNITS]
RATES_SRC = os.path.join(CSRC, "issue_rates.hip")
RATES_LIB = os.path.join(PKG, "libissue_rates.so")
DEPENDS = SOURCES + [os.path.join(CSRC, f) for f in (
    "bcjr_device.h", "bcjr_kernels.h", "bcjr_vec_kernels.h", "bcjr_qat.h", "bcjr_internal.h",
    "bcjr_generic_kernels.h", "bcjr_ldlq_kernels.h", "bcjr_rot_kernels.h", "bcjr_pruned_kernels.h")] + [
    os.path.join(INCLUDE, "bcjr.h")]

BASE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
              # packed FP32 math stays off (v_pk_* fp32 forms)
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              "-Wno-unused-command-line-argument"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the gfx950 library cannot be built")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out_text = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                         if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{out_text}")
    if verbose and out_text.strip():
        print(out_text)


def _compile(sources, out, verbose):
    tmp = out + ".tmp"
    _run([hipcc()] + BASE_FLAGS + ["-shared", "-I", INCLUDE, "-I", CSRC, "-o", tmp] + sources, verbose)
    os.replace(tmp, out)
    return out


def _compile_units(units, out, verbose):
    """Each unit to an object with its own flags, then one shared library."""
    tmp = out + ".tmp"
    with tempfile.TemporaryDirectory(prefix="bcjr_build_") as d:
        objs = []
        for src, flags in units:
            obj = os.path.join(d, os.path.splitext(os.path.basename(src))[0] + ".o")
            _run([hipcc()] + BASE_FLAGS + flags + ["-c", "-I", INCLUDE, "-I", CSRC, "-o", obj, src], verbose)
            objs.append(obj)
        _run([hipcc(), "--offload-arch=gfx950", "-fPIC", "-shared", "-o", tmp] + objs, verbose)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    _compile([RATES_SRC], RATES_LIB, verbose)
    return _compile_units(UNITS, LIB, verbose)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
