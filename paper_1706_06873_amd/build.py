"""Build the MEC HIP library in-tree: ``paper_1706_06873_amd/libmec.so``.

    python paper_1706_06873_amd/build.py

Compiles every source under ``csrc/`` for gfx950 with hipcc into one shared
library exporting the C ABI of ``include/mec.h``. Packed-fp32 instructions are
disabled for all device code.
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
REPO = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(REPO, "include")
LIB = os.path.join(PKG, "libmec.so")
SOURCES = ["mec_api.cpp", "mec_lower.hip", "mec_im2col.hip", "mec_gemm.hip", "mec_gemm_fixed.hip",
           "mec_gemm_ring.hip", "mec_grad.hip"]
ARCH = "gfx950"
# Per-source flags. The flat-window kernel keeps its accumulators in
# architectural VGPRs: with the default heuristic the compiler holds them in
# AGPRs for the MFMAs but copies them through VGPRs at every loop back edge.
EXTRA_FLAGS = {"mec_gemm_ring.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}

HIPCC_FLAGS = [
    "--offload-arch=" + ARCH,
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]


def build(verbose: bool = False) -> str:
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = (["hipcc"] + HIPCC_FLAGS + EXTRA_FLAGS.get(src, []) + lang +
               ["-c", os.path.join(CSRC, src), "-o", obj])
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["hipcc", "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv))
