"""Compile the C oracle into oracle/liboracle.so and the paper-style CPU
server into oracle/libcpups.so (test infrastructure).

gcc in GNU mode contracts a*b-c into an FMA on FMA-capable hosts by default,
so contraction is switched off explicitly; no fast-math, C99, scalar SSE.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "asgd_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-std=c99", "-O2", "-ffp-contract=off", "-fno-fast-math", "-mfpmath=sse",
          "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror"]


# the paper-style CPU server (OpenMP threads, same roundings as the oracle)
CPS_SRC = os.path.join(HERE, "cpu_ps.c")
CPS_LIB = os.path.join(HERE, "libcpups.so")
CPS_CFLAGS = ["-std=c99", "-O3", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
              "-mfpmath=sse", "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror"]


def build(verbose: bool = False) -> str:
    for flags, src, lib in ((CFLAGS, SRC, LIB), (CPS_CFLAGS, CPS_SRC, CPS_LIB)):
        cmd = ["gcc", *flags, src, "-o", lib + ".tmp"]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(lib + ".tmp", lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
