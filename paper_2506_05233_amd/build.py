"""Build libmesa (hipcc, gfx950) in-tree: paper_2506_05233_amd/_lib/libmesa.so."""
from __future__ import annotations

import concurrent.futures
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_DIR = os.path.join(HERE, "_lib")
LIB_PATH = os.path.join(LIB_DIR, "libmesa.so")
OFFLOAD_ARCH = "gfx950"

HIPCC_FLAGS = [
    "--offload-arch=" + OFFLOAD_ARCH,
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: the CG vectors they produce are
    # consumed by VALU code, so this avoids AGPR <-> VGPR copies
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-I" + INCLUDE,
    "-I" + CSRC,
]


# Per-source additions.  The instruction scheduler's ILP strategy (instead of the default
# occupancy-driven one) measured faster for the single-pass CG kernel (~1%) and the chunk
# state scans (2% single product, 9% split product) and slower for the split-operand CG and
# backward kernels, so it applies to those two sources only.
EXTRA_FLAGS = {
    "chunk_cg_bf16.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "chunk_state.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
}


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(verbose: bool = False) -> str:
    """Compile every HIP source into libmesa.so (always recompiles): one object per
    source, compiled side by side, then one shared-library link."""
    os.makedirs(LIB_DIR, exist_ok=True)
    obj_dir = os.path.join(LIB_DIR, "obj")
    os.makedirs(obj_dir, exist_ok=True)
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tag = "%d" % os.getpid()
    jobs = []
    for src in sources():
        obj = os.path.join(obj_dir, os.path.basename(src)[:-4] + "." + tag + ".o")
        extra = EXTRA_FLAGS.get(os.path.basename(src), [])
        jobs.append((src, obj, [hipcc] + HIPCC_FLAGS + extra + ["-c", "-o", obj, src]))
    workers = max(1, min(len(jobs), int(os.environ.get("MAX_JOBS", "0")) or os.cpu_count() or 1, 16))
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        for src, obj, cmd in jobs:
            if verbose:
                print(" ".join(cmd), flush=True)
        list(ex.map(lambda j: subprocess.run(j[2], check=True), jobs))
    tmp = LIB_PATH + ".tmp" + tag
    link = [hipcc, "--offload-arch=" + OFFLOAD_ARCH, "-shared", "-fPIC", "-o", tmp] + [j[1] for j in jobs]
    if verbose:
        print(" ".join(link), flush=True)
    subprocess.run(link, check=True)
    os.replace(tmp, LIB_PATH)
    for _, obj, _ in jobs:
        os.remove(obj)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
