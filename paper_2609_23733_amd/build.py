"""Build libvggtprime.so (gfx950) in-tree with hipcc.

Every .hip file under csrc/ is compiled in parallel to an object, then all are
linked into ``paper_2609_23733_amd/libvggtprime.so``.  Packed fp32 VALU
instructions are disabled for device code.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libvggtprime.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

CFLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # Loop heads on 64-byte boundaries: the FULL-head kernel's inner loops
    # otherwise land at addresses that cost it a few percent, differently
    # from one build to the next.
    "-falign-loops=64",
]
# MFMA results in arch VGPRs: the softmax reads S directly instead of copying
# it out of accumulation registers every tile.  Not for the block GEMM, whose
# 256 accumulators per lane live in the AGPRs.
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=true"]
AGPR_ACC_SOURCES = {"block.hip"}


def _compile(src: str, extra) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    form = [] if os.path.basename(src) in AGPR_ACC_SOURCES else VGPR_FORM
    cmd = [HIPCC] + CFLAGS + form + list(extra) + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s" % (src, msgs))
    if msgs.strip():
        sys.stderr.write(msgs + "\n")
    return obj


def build(extra=(), verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, extra), srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    extra = sys.argv[1:]
    build(extra, verbose=True)
