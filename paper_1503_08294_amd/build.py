"""Build ``libgsn.so`` (the C ABI of include/gsn.h) for gfx950 with hipcc, in-tree.

Flags:
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

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libgsn.so")
SOURCES = ["gsn_host.hip", "find_winners.hip", "staging.hip", "find_screened.hip",
           "find_mfma.hip", "find_f16.hip", "update.hip", "update_winner.hip", "grow.hip",
           "schedule.hip", "find_grid.hip", "resolve_greedy.hip"]
ARCH = "gfx950"

FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-shared",
         "-ffp-contract=off", "-fno-fast-math",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-mfma-vgpr-form",
         "-Wall", "-Wno-unused-result"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def build(verbose: bool = False, extra=()) -> str:
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *FLAGS, *extra, *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
