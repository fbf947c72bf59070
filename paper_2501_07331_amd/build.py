"""Build libsnn.so (HIP, gfx950) in-tree with hipcc.

Flags: -O3, no FP contraction (bit-reproducible fp32 forward), fp32
denormals preserved, packed-fp32 instructions disabled (hipcc forms them
from scalar code otherwise).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = sorted(os.path.join(HERE, "csrc", f) for f in os.listdir(os.path.join(HERE, "csrc"))
              if f.endswith(".hip"))
OUT = os.path.join(HERE, "libsnn.so")
ARCH = os.environ.get("SNN_OFFLOAD_ARCH", "gfx950")


def build(verbose: bool = False) -> str:
    cmd = ["hipcc", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Wall", "-Wno-unused-result",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
           "-o", OUT + ".tmp"] + SRCS
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature and says so
    msgs = [l for l in (res.stdout + res.stderr).splitlines()
            if "packed-fp32-ops" not in l and l.strip()]
    if msgs and (verbose or res.returncode):
        print("\n".join(msgs), file=sys.stderr)
    if res.returncode:
        raise RuntimeError(f"hipcc failed ({res.returncode})")
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
