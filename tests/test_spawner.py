"""The launcher that starts the multi-process tests' programs (CPU)."""
import sys


def test_spawner_runs_concurrently_and_reports(spawner, tmp_path):
    a, b = tmp_path / "a", tmp_path / "b"
    # the two wait for each other: they must run at the same time
    prog = ("import os, sys, time\n"
            "me, other = sys.argv[1], sys.argv[2]\n"
            "open(me, 'w').close()\n"
            "t = time.time()\n"
            "while not os.path.exists(other):\n"
            "    assert time.time() - t < 20\n"
            "    time.sleep(0.01)\n"
            "print('child', me, flush=True)\n"
            "sys.exit(int(sys.argv[3]))\n")
    r = spawner.run([[sys.executable, "-c", prog, str(a), str(b), "0"],
                     [sys.executable, "-c", prog, str(b), str(a), "3"]], timeout=60)
    assert r == {"rc": [0, 3], "timed_out": False}


def test_spawner_kills_at_the_limit(spawner):
    r = spawner.run([[sys.executable, "-c", "import time; time.sleep(60)"],
                     [sys.executable, "-c", "pass"]], timeout=2)
    assert r["timed_out"] and r["rc"][0] is None and r["rc"][1] == 0
