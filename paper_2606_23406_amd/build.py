"""Build libhq.so (gfx950 kernels + host plan + C ABI) in-tree with hipcc.

    python -m paper_2606_23406_amd.build
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libhq.so")
SOURCES = [os.path.join(CSRC, "hq_kernels.hip"), os.path.join(CSRC, "hq_host.cpp")]
DEPS = SOURCES + [os.path.join(CSRC, "hq_internal.h"), os.path.join(CSRC, "calib_table.inc"),
                  os.path.join(os.path.dirname(HERE), "include", "hq.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # every fp32 rounding in the kernels is the one written; no fused contractions
    "-ffp-contract=off",
    # no packed fp32 vector instructions (v_pk_*_f32) are generated
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(d) > t for d in DEPS)


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [HIPCC] + FLAGS + ["-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed building libhq.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
