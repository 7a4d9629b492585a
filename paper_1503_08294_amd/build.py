"""Build ``libgsn.so`` (the C ABI of include/gsn.h) for gfx950 with hipcc, in-tree.

Each source is compiled to an object on its own (in parallel), then linked into the shared
library.  Flags:
  -ffp-contract=off      the distance and update expressions are defined operation by
                         operation in binary32; no multiply-add contraction;
  -Xclang -target-feature -Xclang -packed-fp32-ops
                         no packed fp32 instructions are generated;
  -mllvm -amdgpu-mfma-vgpr-form
                         matrix-core results are written to ordinary VGPRs, so the vector
                         unit reads them without accumulator-register copies;
  no fast-math, IEEE denormals (default for gfx950 fp32).
"""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libgsn.so")
OBJ_DIR = os.path.join(HERE, "_build")
SOURCES = ["gsn_host.hip", "find_winners.hip", "staging.hip", "find_screened.hip",
           "find_mfma.hip", "find_f16.hip", "update.hip", "update_winner.hip", "grow.hip",
           "schedule.hip", "find_grid.hip", "resolve_greedy.hip", "find_small.hip"]
ARCH = "gfx950"

FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC",
         "-ffp-contract=off", "-fno-fast-math",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-mfma-vgpr-form",
         "-Wall", "-Wno-unused-result"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def _jobs() -> int:
    return max(1, min(8, int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))


def build(verbose: bool = False, extra=()) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    cmds = []
    objs = []
    for s in SOURCES:
        obj = os.path.join(OBJ_DIR, os.path.splitext(s)[0] + ".o")
        objs.append(obj)
        cmds.append([hipcc(), *FLAGS, *extra, "-c", os.path.join(CSRC, s), "-o", obj])
    if verbose:
        for c in cmds:
            print(" ".join(c), flush=True)
    with ThreadPoolExecutor(_jobs()) as pool:
        results = list(pool.map(lambda c: subprocess.run(c, capture_output=True, text=True),
                                cmds))
    failed = False
    for c, r in zip(cmds, results):
        if r.returncode != 0 or (verbose and r.stderr.strip()):
            msg = "\n".join(ln for ln in r.stderr.splitlines()
                            if "packed-fp32-ops" not in ln)
            if msg.strip():
                print(msg, flush=True)
        failed |= r.returncode != 0
    if failed:
        raise subprocess.CalledProcessError(1, "hipcc (see the messages above)")
    tmp = LIB + ".tmp"
    link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(link), flush=True)
    subprocess.run(link, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
