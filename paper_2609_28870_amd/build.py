"""Build libpc (the HIP library) for gfx950 with hipcc, in-tree.

Output: ``paper_2609_28870_amd/_lib/libpc.so``.  Every call recompiles."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC_DIR = os.path.join(HERE, "csrc")
SOURCES = ["pc_api.hip", "pc_hash.hip", "pc_sort.hip", "pc_chain.hip", "pc_stackdist.hip", "pc_runs.hip", "pc_session.hip", "pc_profile.hip", "pc_mrc.hip",
           "pc_noalloc.hip", "pc_belady.hip"]
OUT = os.path.join(HERE, "_lib", "libpc.so")
ARCH = os.environ.get("PC_OFFLOAD_ARCH", "gfx950")

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    "--offload-arch=" + ARCH,
    # no packed-FP32 instructions anywhere in this library
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def build(verbose: bool = False) -> str:
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    tmp = OUT + ".tmp%d" % os.getpid()
    cmd = ["hipcc"] + FLAGS + ["-I", os.path.join(ROOT, "include")] + \
        [os.path.join(SRC_DIR, s) for s in SOURCES] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.check_call(cmd)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
