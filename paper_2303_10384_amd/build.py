"""Builds the HIP library librnnt_mi355x.so in-tree for gfx950.

    python -m paper_2303_10384_amd.build          (or __graft_entry__.build())
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB_NAME = "librnnt_mi355x.so"
SOURCES = ["csrc/rnnt_api.hip", "csrc/rnnt_arc_plan.cpp"]
HEADERS = ["csrc/rnnt_device.h", "csrc/rnnt_k1_populate.h", "csrc/rnnt_k2_lattice.h", "csrc/rnnt_k2_viterbi.h",
           "csrc/rnnt_k3_grad.h", "csrc/rnnt_arc_layout.h", "csrc/rnnt_arc_kernels.h"]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the library)")


def compile_flags():
    return [
        "--offload-arch=gfx950",
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-shared",
        "-Wall",
        # packed fp32 VALU ops stay off: ordinary float code only
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"),
        "-I", os.path.join(PKG, "csrc"),
    ]


def build(verbose=True, extra_flags=()):
    out = os.path.join(PKG, LIB_NAME)
    tmp = out + ".tmp"
    cmd = [hipcc()] + compile_flags() + list(extra_flags) + [os.path.join(PKG, s) for s in SOURCES] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    build(verbose=True, extra_flags=sys.argv[1:])
