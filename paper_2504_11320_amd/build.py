"""Build the HIP library (gfx950) in-tree: paper_2504_11320_amd/libwait_sim.so.

Each source is compiled to an object in parallel, then the objects are
linked into one shared library."""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
import time
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SRC_NAMES = ("wait_sim_host.hip", "sim_known_wait.hip", "sim_known_fcfs.hip",
             "sim_nested.hip", "sim_known_wait_tv.hip", "sim_known_fcfs_tv.hip",
             "sim_nested_tv.hip", "sim_fcfs_dist.hip", "sim_wait_many.hip")
SRCS = [os.path.join(CSRC, f) for f in SRC_NAMES]
INC = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libwait_sim.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # identical IEEE operations on both sides of the parity tests
    "-ffp-contract=off", "-fno-fast-math",
    # no packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


# Instruction-scheduling strategy per translation unit (LLVM's AMDGPU
# scheduler), as measured: the known-length WAIT and the Nested WAIT kernels
# gain from the ILP-maximising one, the FCFS kernels lose.
SCHED_FLAGS = {
    "sim_known_wait.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "sim_known_wait_tv.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "sim_wait_many.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "sim_nested.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "sim_nested_tv.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
}


def flags_for(src: str) -> list:
    """hipcc options for one source file."""
    return HIPCC_FLAGS + SCHED_FLAGS.get(os.path.basename(src), [])


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if c and (os.path.exists(c) or c == "hipcc"):
            return c
    return "hipcc"


# Host-side AddressSanitizer and UndefinedBehaviorSanitizer (device code is
# built as usual): each -fsanitize= goes right after -Xarch_host.
SANITIZE_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def build(verbose: bool = False, defines=(), out: str = LIB, sanitize: bool = False) -> str:
    """Compile every source for gfx950 and link `out` (default: the in-tree
    library).  `defines` are extra -D options; `sanitize` instruments the host
    code with ASan and UBSan (load the result with the clang ASan runtime
    preloaded)."""
    dflags = [f"-D{d}" for d in defines] + (SANITIZE_FLAGS if sanitize else [])
    with tempfile.TemporaryDirectory(prefix="wait_sim_build_") as tmp:
        def compile_one(src: str):
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            cmd = [hipcc()] + flags_for(src) + dflags + ["-I", INC, "-I", CSRC, "-c", "-o", obj, src]
            if verbose:
                print(" ".join(cmd), flush=True)
            t0 = time.perf_counter()
            subprocess.run(cmd, check=True)
            if verbose:
                print(f"  {os.path.basename(src)}: {time.perf_counter() - t0:.1f} s", flush=True)
            return obj

        workers = max(1, min(len(SRCS), os.cpu_count() or 1))
        with ThreadPoolExecutor(workers) as ex:
            objs = list(ex.map(compile_one, SRCS))
        cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", out + ".tmp"] + objs
        if sanitize:
            cmd += ["-fsanitize=address,undefined", "-shared-libasan"]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
