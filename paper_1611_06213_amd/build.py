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
# the same source with contraction allowed (fused multiply-adds); within 1e-6
# relative of the oracle instead of bitwise
LIB_FMA = os.path.join(HERE, "libgadeips_fma.so")
FMA_FLAGS = ["-ffp-contract=fast", "-DPS_FP_CONTRACT=1"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = [os.path.join(CSRC, "ps_server.cpp"), os.path.join(CSRC, "ps_protocol.cpp"),
           os.path.join(CSRC, "ps_layout.cpp"), os.path.join(CSRC, "ps_kernels.hip")]

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wextra", "-Wno-unused-parameter",
    "-I", INCLUDE, "-I", CSRC,
]


def build(verbose: bool = False, out: str = LIB, extra=()) -> str:
    tmp = out + ".tmp"
    flags = list(FLAGS)
    if any(x.startswith("-ffp-contract=") for x in extra):
        flags = [f for f in flags if not f.startswith("-ffp-contract=")]
    cmd = [HIPCC, *flags, *extra, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed building " + os.path.basename(out))
    os.replace(tmp, out)
    return out


def build_all(verbose: bool = False):
    """Both flavours: the bitwise default and the contraction-allowed one."""
    return build(verbose), build(verbose, out=LIB_FMA, extra=FMA_FLAGS)


# a plain C program that drives the C ABI without Python (tests/test_c_abi.py)
C_SMOKE_SRC = os.path.join(ROOT, "tests", "c_abi_smoke.c")
C_SMOKE = os.path.join(ROOT, "tests", "c_abi_smoke")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build_c_smoke(verbose: bool = False) -> str:
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", INCLUDE, "-I", os.path.join(ROCM, "include"), C_SMOKE_SRC,
           "-L", HERE, "-lgadeips", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../paper_1611_06213_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib"),
           "-o", C_SMOKE + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("gcc failed building the C ABI smoke program")
    os.replace(C_SMOKE + ".tmp", C_SMOKE)
    return C_SMOKE


if __name__ == "__main__":
    print(build_all(verbose=True))
