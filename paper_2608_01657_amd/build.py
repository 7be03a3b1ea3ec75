"""Builds libpcreplay.so (the HIP library behind include/pc.h) for gfx950,
and two test builds of the same sources:
  - libpcreplay_phases.so, with per-phase cycle counters (-DPC_PROFILE; the
    counters replace the stats record of group 63);
  - libpcreplay_jitter.so, the race-detection build (-DPC_JITTER): every
    replay barrier is followed by a pseudo-random per-wavefront delay, so
    results that depend on wavefront timing differ from the oracle's.

    python -m paper_2608_01657_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libpcreplay.so")
LIB_PHASES = os.path.join(HERE, "libpcreplay_phases.so")
LIB_JITTER = os.path.join(HERE, "libpcreplay_jitter.so")
BUILD_DIR = os.path.join(ROOT, "_build")

SOURCES = ["pc_hash.hip", "pc_replay.hip", "pc_replay_global.hip", "pc_abi.cpp"]
ARCH = os.environ.get("PC_OFFLOAD_ARCH", "gfx950")
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
         # packed FP32 instructions stay off (none are needed: the path is integer)
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-result"]
# Machine schedulers of the replay kernels, each the fastest measured for
# its layouts (results are identical under every one):
#  - all-LDS layout (pc_replay.hip): the scheduler that maximises
#    instruction-level parallelism, 3.5 % less replay time than the default
#    one on the one-touch C = 4096 batch (one instance per CU);
#  - hybrid and workspace layouts (pc_replay_global.hip, two instances per
#    CU, state partly or wholly in global memory): the iterative scheduler
#    that keeps the occupancy target, 2.4 % less time than the ILP one on
#    the 1,024-instance batch (hybrid) and 1.9 % on the C = 16,384 chat
#    instances (workspace); it costs the all-LDS kernels 2.2-2.6 %, hence
#    the separate translation unit.
# The loops that must be unrolled say so (#pragma unroll); the compiler's
# own unrolling of the others only lengthens the instruction stream and
# raises register pressure (another 3.7 % less replay time without it).
SOURCE_FLAGS = {"pc_replay.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp", "-fno-unroll-loops"],
                "pc_replay_global.hip": ["-mllvm", "-amdgpu-sched-strategy=iterative-maxocc", "-fno-unroll-loops"]}


def _hipcc() -> str:
    for c in ("/opt/rocm/bin/hipcc", "hipcc"):
        if os.path.sep not in c or os.path.exists(c):
            return c
    return "hipcc"


def build(verbose: bool = False) -> str:
    variants = [(LIB, BUILD_DIR, []),
                (LIB_PHASES, os.path.join(BUILD_DIR, "phases"), ["-DPC_PROFILE"]),
                (LIB_JITTER, os.path.join(BUILD_DIR, "jitter"), ["-DPC_JITTER"])]
    with ThreadPoolExecutor(max_workers=len(variants)) as ex:
        for f in [ex.submit(_build_one, lib, d, extra, verbose) for lib, d, extra in variants]:
            f.result()
    return LIB


def _build_one(lib_path, build_dir, extra, verbose):
    os.makedirs(build_dir, exist_ok=True)
    hipcc = _hipcc()

    def compile_one(src):
        obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc, *FLAGS, *SOURCE_FLAGS.get(src, []), *extra, "-c", os.path.join(CSRC, src), "-o", obj]
        if src.endswith(".cpp"):
            cmd = [hipcc, *FLAGS, *extra, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
        if verbose and r.stderr.strip():
            print(r.stderr, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = lib_path + f".tmp{os.getpid()}"
    r = subprocess.run([hipcc, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, lib_path)
    return lib_path


if __name__ == "__main__":
    print(build(verbose=True))
