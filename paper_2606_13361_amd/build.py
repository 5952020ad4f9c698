"""Compile libkvr.so (gfx950) in place with hipcc.

The library is the whole product path: HIP kernels plus the C ABI declared in
include/kvr.h.  Built in-tree so it travels with the source tree.
"""
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libkvr.so")
# the decoder layer around the attention: its own library, linked against
# libkvr's public ABI and hipBLASLt
MODEL_LIB = os.path.join(PKG, "libkvr_model.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # no packed fp32 instructions in any generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs: keeps the loop-carried attention
    # accumulators out of AGPR <-> VGPR copies around the softmax updates
    "-mllvm", "-amdgpu-mfma-vgpr-form",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.isabs(cand) and os.path.exists(cand) or not os.path.isabs(cand)):
            return cand
    return "hipcc"


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def model_sources():
    return sorted(glob.glob(os.path.join(CSRC, "model", "*.hip")))


def build(verbose=False):
    """Always recompile both libraries."""
    _build_one(LIB, sources(), [], verbose)
    _build_one(MODEL_LIB, model_sources(),
               ["-L" + PKG, "-lkvr", "-Wl,-rpath,$ORIGIN", "-L/opt/rocm/lib", "-lhipblaslt"], verbose)
    return LIB


def _build_one(lib, srcs, link, verbose):
    """Compile srcs into lib, written atomically."""
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + ["-I" + INCLUDE, "-I" + CSRC] + srcs + ["-o", tmp] + link
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    msgs = [ln for ln in res.stdout.splitlines() if noise not in ln]
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if msgs and verbose:
        print("\n".join(msgs), file=sys.stderr)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
