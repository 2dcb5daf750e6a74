"""Build ``liblpv.so`` (the HIP kernels and the C ABI of include/lpv.h) for gfx950.

Cross-compiles with hipcc; no GPU is needed to build.  Every build recompiles
from source.
"""
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "liblpv.so")
SOURCES = ["api.hip", "pack.hip", "linear.hip", "mask.hip", "backward.hip", "delta.hip", "encoder.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "-std=c++17", "-O3", "--offload-arch=" + ARCH, "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: the kept-tile walk branches
    # around each tile's instructions, and accumulators in AGPRs would then be
    # copied across every branch
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
]


# Kernels whose LDS ring counts every vector-memory instruction a wave issues
# (vmcnt): a register spill to scratch would add uncounted ones, so any
# scratch use there fails the build.
NO_SCRATCH = ("k_linear16",)


def check_resources(remarks):
    """Parse hipcc's kernel-resource-usage remarks; return the offending lines."""
    bad, kernel = [], None
    for line in remarks:
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            kernel = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and kernel and any(k in kernel for k in NO_SCRATCH) and int(m.group(1)) > 0:
            bad.append("%s: %s bytes of scratch per lane" % (kernel, m.group(1)))
    return bad


def build(verbose: bool = False, extra=()) -> str:
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-Rpass-analysis=kernel-resource-usage", "-fno-caret-diagnostics"] + list(extra) + srcs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    p = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature and says so
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"
    lines = [l for l in (p.stdout + p.stderr).splitlines() if noise not in l]
    remarks = [l for l in lines if "remark:" in l]
    msgs = [l for l in lines if "remark:" not in l]
    if p.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s" % (p.returncode, "\n".join(msgs)))
    bad = check_resources(remarks)
    if bad:
        os.unlink(tmp)
        raise RuntimeError("register spills in ring kernels:\n" + "\n".join(bad))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
