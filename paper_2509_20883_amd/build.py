"""Build librecis_mi355x.so (the HIP kernels + C ABI) in-tree for gfx950 with hipcc."""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "librecis_mi355x.so")
SOURCES = ["dedup_idmap.hip", "ids_partition.hip", "feature_ops.hip", "pool.hip", "backward.hip", "probes.hip", "ids_static.hip", "api.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # bit-exact row init and plain fp32 optimizer arithmetic: no contraction
    "-ffp-contract=off",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-variable", "-Wno-unused-command-line-argument",
]


def build(verbose: bool = False, jobs: int = 4, out: str = LIB, defines=()) -> str:
    """Compile every source and link `out` (default: the in-tree library);
    `defines` are extra -D options (tuning variants)."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objs = []
    procs = []
    for src in SOURCES:
        obj = out + "." + src + ".o"
        cmd = [hipcc, *HIPCC_FLAGS, *[f"-D{d}" for d in defines], "-c", "-I", os.path.join(ROOT, "include"), "-I",
               CSRC, os.path.join(CSRC, src), "-o", obj]
        cmd.remove("-shared")
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd))
        objs.append(obj)
        if len(procs) >= jobs:
            if procs.pop(0).wait() != 0:
                raise RuntimeError("hipcc failed")
    for p in procs:
        if p.wait() != 0:
            raise RuntimeError("hipcc failed")
    cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    for o in objs:
        os.remove(o)
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
