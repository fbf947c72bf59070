"""Build libsnn.so (HIP, gfx950) in-tree with hipcc, one object per source.

Flags: -O3, no FP contraction (bit-reproducible fp32 forward), fp32
denormals preserved, packed-fp32 instructions disabled (hipcc forms them
from scalar code otherwise).
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = sorted(os.path.join(HERE, "csrc", f) for f in os.listdir(os.path.join(HERE, "csrc"))
              if f.endswith(".hip"))
OUT = os.path.join(HERE, "libsnn.so")
ARCH = os.environ.get("SNN_OFFLOAD_ARCH", "gfx950")


FLAGS = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-result"]
OBJDIR = os.path.join(HERE, "_build")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature and says so
    msgs = [l for l in (res.stdout + res.stderr).splitlines()
            if "packed-fp32-ops" not in l and l.strip()]
    return res.returncode, msgs


def build(verbose: bool = False, jobs: int = 0) -> str:
    """Compiles every csrc/*.hip to an object (in parallel), then links."""
    os.makedirs(OBJDIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
    jobs = jobs or min(8, os.cpu_count() or 1)
    objs, cmds = [], []
    for src in SRCS:
        obj = os.path.join(OBJDIR, os.path.basename(src)[:-4] + ".o")
        objs.append(obj)
        cmds.append(["hipcc", f"--offload-arch={ARCH}", *FLAGS, *inc, "-c", "-o", obj, src])
    with ThreadPoolExecutor(max_workers=jobs) as pool:
        results = list(pool.map(lambda c: _run(c, verbose), cmds))
    failed = False
    for (rc, msgs), src in zip(results, SRCS):
        if msgs and (verbose or rc):
            print("\n".join(msgs), file=sys.stderr)
        if rc:
            print(f"hipcc failed ({rc}) on {os.path.basename(src)}", file=sys.stderr)
            failed = True
    if failed:
        raise RuntimeError("hipcc failed")
    rc, msgs = _run(["hipcc", f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", OUT + ".tmp"] + objs,
                    verbose)
    if msgs and (verbose or rc):
        print("\n".join(msgs), file=sys.stderr)
    if rc:
        raise RuntimeError(f"hipcc link failed ({rc})")
    os.replace(OUT + ".tmp", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
