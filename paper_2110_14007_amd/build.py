"""Build libtod.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libtod.so")
SOURCES = ["api.hip", "prep.hip", "select.hip", "lof.hip", "tile_f32.hip", "tile_f16.hip",
           "tile_bf16.hip", "mtile_f16.hip", "mtile_bf16.hip", "order.hip",
           "rtile_f16.hip", "rtile_bf16.hip", "nwr.hip", "score.hip", "loci.hip"]
# The fused tile kernels take maxima of MFMA accumulators (fmax, so that the
# compiler sees the reads and inserts the wait states an MFMA result needs
# before a VALU reads it).  Their operands are never NaN (prep rejects
# non-finite input; masked entries are -inf), and -fno-honor-nans lets the
# compiler form v_max3_f32 without quieting every operand first.
NO_NAN_SOURCES = {"mtile_f16.hip", "mtile_bf16.hip", "tile_f32.hip", "tile_f16.hip",
                  "tile_bf16.hip"}
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def build(verbose: bool = False) -> str:
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)

    def compile_one(src: str) -> str:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        extra = ["-fno-honor-nans"] if src in NO_NAN_SOURCES else []
        cmd = [HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        out = "\n".join(line for line in (r.stdout + r.stderr).splitlines()
                        if "packed-fp32-ops" not in line)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed for %s:\n%s" % (src, out))
        if verbose and out.strip():
            print(out, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s%s" % (r.stdout, r.stderr))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
