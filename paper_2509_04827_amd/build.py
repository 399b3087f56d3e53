"""Build libvdecode.so in-tree with hipcc for gfx950 (MI355X) only.

    python -m paper_2509_04827_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", f) for f in ("vdecode.hip", "gemm.hip")]
HEADER = os.path.join(ROOT, "include", "vdecode.h")
LIB = os.path.join(HERE, "libvdecode.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]
# per source: MFMA accumulators in ordinary VGPRs.  The attention kernels'
# online-softmax rescale touches them with VALU ops, and the GEMM tiles'
# accumulators fit the VGPRs; in AGPRs the compiler copies them back and forth
# inside the K loop (over 200 accumulator moves per stage of the LDS-fed tiles)
SRC_FLAGS = {
    "vdecode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so; harmless
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s" % (res.returncode, err))
    if err.strip() and verbose:
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    """Compile each source with its flags, then link the shared library."""
    tag = ".tmp%d" % os.getpid()
    objs = []
    try:
        for src in SRCS:
            obj = os.path.join(HERE, os.path.basename(src) + tag + ".o")
            objs.append(obj)
            _run([hipcc(), *HIPCC_FLAGS, *SRC_FLAGS[os.path.basename(src)], "-I",
                  os.path.join(ROOT, "include"), "-c", "-o", obj, src], verbose)
        tmp = LIB + tag
        _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
        os.replace(tmp, LIB)
    finally:
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
