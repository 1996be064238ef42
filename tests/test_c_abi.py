"""The C ABI from a plain C program (tests/c_abi_smoke.c): no Python and no
torch in that process, device memory from the HIP runtime, results checked
against closed forms that are exact in binary32."""
import os
import subprocess

import pytest

from paper_1611_06213_amd import build as lib_build


@pytest.mark.gpu
def test_c_program_drives_the_abi(spawner, tmp_path):
    """Started by the session's launcher (tests/spawner.py), which never
    touches the GPU; the program's output goes to a file."""
    if not os.path.exists(lib_build.C_SMOKE):
        pytest.fail("tests/c_abi_smoke is not built (run __graft_entry__.build())")
    out = tmp_path / "c_abi.out"
    sh = f"exec {lib_build.C_SMOKE} > {out} 2>&1"
    r = spawner.run([["/bin/sh", "-c", sh]], timeout=120)
    text = out.read_text()
    assert r == {"rc": [0], "timed_out": False}, text[-2000:]
    assert "c abi ok" in text
    for line in text.splitlines():
        if line.startswith("tiny loop"):
            print(line, flush=True)


def test_c_program_builds_and_links():
    """On the CPU: the program compiles warning-free against include/ps.h and
    links against the library (built by __graft_entry__.build)."""
    if not os.path.exists(lib_build.LIB):
        pytest.fail("libgadeips.so is not built (run __graft_entry__.build())")
    lib_build.build_c_smoke()
    assert os.access(lib_build.C_SMOKE, os.X_OK)
    r = subprocess.run(["ldd", lib_build.C_SMOKE], capture_output=True, text=True)
    assert "libgadeips.so" in r.stdout and "not found" not in r.stdout, r.stdout
