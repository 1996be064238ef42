"""A process launcher that never touches the GPU.

The test session starts it before any test initialises HIP, so the programs
that multi-process tests need (a parameter server and its learners, each in
its own address space) are started by a process that never initialised the
GPU, and no process that did ever starts another one.

Protocol, one JSON object per line on stdin, one reply per line on stdout:
  {"cmds": [[argv...], ...], "timeout": seconds, "cwd": dir}
    -> {"rc": [code or null if killed at the limit, ...], "timed_out": bool}
Every command's stdout and stderr go to the launcher's stderr (its stdout
carries the replies). All commands of one request
start together and run concurrently; past the time limit the launcher kills
the ones still running (by their own process ids) and reports them.
EOF-on-stdin ends the launcher.
"""
import json
import os
import subprocess
import sys
import time


def run(req):
    procs = []
    for argv in req["cmds"]:
        procs.append(subprocess.Popen(argv, cwd=req.get("cwd") or None,
                                      stdin=subprocess.DEVNULL, stdout=sys.stderr.fileno(),
                                      env=os.environ.copy()))
    deadline = time.monotonic() + float(req.get("timeout", 60))
    rcs = [None] * len(procs)
    timed_out = False
    while any(r is None for r in rcs):
        for i, p in enumerate(procs):
            if rcs[i] is None:
                rcs[i] = p.poll()
        if all(r is not None for r in rcs):
            break
        if time.monotonic() > deadline:
            timed_out = True
            for i, p in enumerate(procs):
                if rcs[i] is None:
                    p.kill()
                    p.wait()
            break
        time.sleep(0.02)
    return {"rc": rcs, "timed_out": timed_out}


def main():
    for line in sys.stdin:
        line = line.strip()
        if not line:
            continue
        try:
            reply = run(json.loads(line))
        except Exception as e:   # report, keep serving
            reply = {"error": repr(e)}
        sys.stdout.write(json.dumps(reply) + "\n")
        sys.stdout.flush()


if __name__ == "__main__":
    main()
