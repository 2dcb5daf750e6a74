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
    "-std=c++17", "-O3", "--offload-arch=" + ARCH, "-fPIC",
    "-Wall", "-Wno-unused-function",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
# Per-source flags.  The matrix-core kernels keep their accumulators in
# ordinary VGPRs: they branch around each tile's instructions, and at their
# register counts accumulators in AGPRs would be copied across every branch.
_VGPR_MFMA = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
SOURCE_FLAGS = {"linear.hip": _VGPR_MFMA, "backward.hip": _VGPR_MFMA, "encoder.hip": _VGPR_MFMA}
BUILD_DIR = os.path.join(HERE, "_build")


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
    """Compile every source to an object (in parallel), then link the shared
    library; resource remarks are checked per object."""
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(BUILD_DIR, exist_ok=True)
    noise = "'-packed-fp32-ops' is not a recognized feature for this target"

    def compile_one(src):
        obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
        cmd = ([HIPCC] + FLAGS + SOURCE_FLAGS.get(src, []) +
               ["-Rpass-analysis=kernel-resource-usage", "-fno-caret-diagnostics"] + list(extra) +
               ["-c", os.path.join(CSRC, src), "-o", obj])
        if verbose:
            print(" ".join(cmd), flush=True)
        p = subprocess.run(cmd, capture_output=True, text=True)
        lines = [l for l in (p.stdout + p.stderr).splitlines() if noise not in l]
        return src, obj, p.returncode, lines

    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        results = list(ex.map(compile_one, SOURCES))
    bad = []
    for src, obj, rc, lines in results:
        msgs = [l for l in lines if "remark:" not in l]
        if rc != 0:
            raise RuntimeError("hipcc failed on %s (%d):\n%s" % (src, rc, "\n".join(msgs)))
        bad += check_resources([l for l in lines if "remark:" in l])
        if verbose and msgs:
            print("\n".join(msgs))
    if bad:
        raise RuntimeError("register spills in ring kernels:\n" + "\n".join(bad))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC"] + [r[1] for r in results] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError("link failed (%d):\n%s" % (p.returncode, p.stdout + p.stderr))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
