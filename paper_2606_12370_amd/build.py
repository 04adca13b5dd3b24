"""Build libspecverify.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2606_12370_amd.build

The library lands next to this file so that it travels with the source tree.
"""

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libspecverify.so")
ARCH = "gfx950"

SOURCES = ["specverify.hip"]
HEADERS = ["sv_device.h", "verify_kernel.h", "tv_kernel.h", "variants_kernel.h", "gumbel_kernel.h", "kl_kernel.h"]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def compile_cmd(out=LIB, extra=()):
    return [
        hipcc(), "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
        # code objects the ROCm 7.0 runtime bundled with PyTorch can load
        "-mcode-object-version=5",
        # expressions are evaluated as written: the comparisons 1[q <= p] must
        # see the same rounded products everywhere they are formed
        "-ffp-contract=off",
        # no packed FP32 instructions
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-I" + INCLUDE, "-I" + CSRC,
        *extra,
        "-o", out,
    ] + [os.path.join(CSRC, s) for s in SOURCES]


def build(verbose=False):
    """Compile the library (always, even if a built copy exists)."""
    tmp = LIB + ".tmp"
    cmd = compile_cmd(out=tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + msgs)
    if verbose and msgs.strip():
        print(msgs)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
