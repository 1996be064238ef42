"""Build libgadeips.so (host library + gfx950 kernels) in-tree with hipcc.

Flags:
  -ffp-contract=off     no fused multiply-add: every product and sum rounds on
                        its own, as sequential binary32 steps do (the kernel
                        file also says so with a pragma)
  -Xclang -target-feature -Xclang -packed-fp32-ops
                        keep the compiler from emitting packed fp32 ops
  --offload-arch=gfx950 MI355X (CDNA4) only
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libgadeips.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = [os.path.join(CSRC, "ps_server.cpp"), os.path.join(CSRC, "ps_kernels.hip")]

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wextra", "-Wno-unused-parameter",
    "-I", INCLUDE, "-I", CSRC,
]


def build(verbose: bool = False, out: str = LIB, extra=()) -> str:
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *extra, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed building " + os.path.basename(out))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
