import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


class Spawner:
    """Client of tests/spawner.py, a launcher started before this process
    touches the GPU (see there)."""

    def __init__(self):
        self.p = subprocess.Popen([sys.executable, "-u", os.path.join(ROOT, "tests", "spawner.py")],
                                  stdin=subprocess.PIPE, stdout=subprocess.PIPE, text=True,
                                  cwd=ROOT)

    def run(self, cmds, timeout, cwd=None):
        self.p.stdin.write(json.dumps({"cmds": cmds, "timeout": timeout, "cwd": cwd}) + "\n")
        self.p.stdin.flush()
        reply = json.loads(self.p.stdout.readline())
        if "error" in reply:
            raise RuntimeError("launcher: " + reply["error"])
        return reply

    def close(self):
        if self.p.poll() is None:
            self.p.stdin.close()
            self.p.wait(timeout=30)


_SPAWNER = None


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running")
    global _SPAWNER
    # started here, before any test can initialise the GPU in this process
    if _SPAWNER is None:
        _SPAWNER = Spawner()


def pytest_unconfigure(config):
    global _SPAWNER
    if _SPAWNER is not None:
        _SPAWNER.close()
        _SPAWNER = None


@pytest.fixture(scope="session")
def spawner():
    return _SPAWNER
