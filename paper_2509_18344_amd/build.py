"""Build step of the native library: compiles csrc/ with hipcc for gfx950 into
``libsubspec.so`` next to this file (in-tree, so that it travels with the tree)."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsubspec.so")
HOST_SOURCES = ["api.cpp"]
DEVICE_SOURCES = ["kernels_qlinear.hip", "kernels_qmma.hip", "kernels_qmma_b2.hip", "kernels_qmma_b3.hip",
                  "kernels_qmma_b4.hip", "kernels_prep.hip", "kernels_tree.hip", "kernels_attn.hip",
                  "noalloc.hip"]
OBJDIR = os.path.join(ROOT, "_build")

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
    "-ffp-contract=off",
    # keep the compiler from emitting packed fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: the per-group scale/offset FMAs
    # read them directly instead of copying them out of AGPRs first
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wno-unused-command-line-argument",
]


HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("build step failed: " + " ".join(cmd[:2]) + " ... " + cmd[-1])


def build(verbose: bool = False) -> str:
    """Compile every source (always, even when a built library exists)."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJDIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    jobs = []
    for s in HOST_SOURCES:
        o = os.path.join(OBJDIR, s + ".o")
        jobs.append((["g++", *HOST_FLAGS, *inc, "-c", os.path.join(CSRC, s), "-o", o], o))
    for s in DEVICE_SOURCES:
        o = os.path.join(OBJDIR, s + ".o")
        jobs.append(([hipcc, *HIPCC_FLAGS, *inc, "-c", os.path.join(CSRC, s), "-o", o], o))
    # the translation units are independent: compile them side by side
    with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1, 8)) as ex:
        list(ex.map(lambda j: _run(j[0], verbose), jobs))
    objs = [o for _, o in jobs]
    _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", LIB + ".tmp"], verbose)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
