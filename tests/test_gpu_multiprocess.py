"""Learners as separate processes (Sec. 4.1, 4.3), on one GPU.

A server process and four learner processes share the server's rows through
HIP IPC (tests/mp_ps.py). The processes are started by the session's
launcher (tests/spawner.py), which never touches the GPU. One learner may
stop mid-schedule with gradients still in its slots; the server then
retires it (its queued gradients apply exactly once, Theorem 2) or drops it.
The server's log of every protocol call is replayed through the oracle:
order, staleness, queued counts at the death, final weights, velocity and
every finished learner's last replica must match bit for bit.
"""
import hashlib
import json
import os
import sys

import numpy as np
import pytest

from oracle import server as orc
from paper_1611_06213_amd import ps
from paper_1611_06213_amd import workloads as wl
from tests import mp_ps, parity

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def torch():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    ps.load_library()
    return torch


def run_processes(spawner, tmp_path, conf):
    """Start the server and the learners together; returns the server log."""
    sock_dir = f"/tmp/mp_ps_{os.getpid()}_{abs(hash(str(tmp_path))) % 100000}"
    os.makedirs(sock_dir, exist_ok=True)
    os.makedirs(tmp_path, exist_ok=True)
    conf = dict(conf, sock=os.path.join(sock_dir, "s"), out=str(tmp_path))
    if os.path.exists(conf["sock"]):
        os.unlink(conf["sock"])
    path = tmp_path / "conf.json"
    path.write_text(json.dumps(conf))
    prog = os.path.join(ROOT, "tests", "mp_ps.py")
    cmds = [[sys.executable, "-u", prog, "server", str(path)]]
    cmds += [[sys.executable, "-u", prog, "learner", str(path), str(l)]
             for l in range(conf["learners"])]
    print(f"[mp] starting 1 server + {conf['learners']} learners, die={conf['die']} "
          f"mode={conf['dead_mode']}", file=sys.stderr, flush=True)
    r = spawner.run(cmds, timeout=100)
    assert not r["timed_out"] and r["rc"] == [0] * len(cmds), r
    with open(tmp_path / "server.json") as f:
        return conf, json.load(f)


def replay(torch, conf, log, o=None):
    """The oracle through the server's calls, in the server's order (from a
    given oracle state, for the run after a restart)."""
    cfg = mp_ps.workload(conf)
    pool = {}
    if o is None:
        w0 = parity.np_bits(wl.make_w0(cfg, "cuda"))
        o = orc.OracleServer(w0, conf["lr"], conf["momentum"], depth=conf["depth"])
        if conf.get("queue", "rr") == "rr":
            assert o.set_queue_mode(orc.ROUND_ROBIN, conf["slots"]) == orc.OK
    deaths = []
    for e in log:
        if e[0] == "push":
            _, l, _, j = e
            if j not in pool:
                pool[j] = parity.np_bits(wl.make_grad(cfg, j, "cuda"))
            assert o.push(l, pool[j]) == orc.OK
        elif e[0] == "apply":
            n0 = len(o.staleness)
            o.apply_pending()
            assert o.applied_order[n0:] == e[1] and o.staleness[n0:] == e[2], e
        elif e[0] == "pull":
            for l in e[1]:
                o.pull(l, ("replica", l), orc.F32)
        elif e[0] == "retire":
            assert o.retire_learner(e[1]) == e[2]
            deaths.append(e)
        elif e[0] == "drop":
            assert o.drop_learner(e[1]) == e[2]
            deaths.append(e)
        elif e[0] == "checkpoint":
            assert o.pending() == 0 and o.ts == e[1]
        elif e[0] == "resume":
            assert o.restart() == orc.OK and o.ts == e[1]
        else:
            raise AssertionError(e)
    return o, deaths


CONF = {"n": 1_000_003, "lr": 0.005, "momentum": 0.9, "learners": 4, "slots": 3, "depth": 4,
        "pool": 16, "pushes": [10, 10, 10, 10], "limit": 80}


@pytest.mark.parametrize("dead_mode,die,extra", [
    ("retire", {}, {}),
    ("retire", {"2": 7}, {}),
    ("drop", {"2": 7}, {}),
    ("retire", {"1": 6}, {"workload": "mixed", "queue": "fifo", "lr": 0.001, "depth": 6}),
], ids=["all-finish", "retire", "drop", "bf16-fifo-retire"])
def test_learner_processes_share_server_rows(torch, spawner, tmp_path, dead_mode, die, extra):
    """Round-robin queues with fp32 gradients (the first three), and one FIFO
    queue of 6 with bf16 gradients in bf16 rows."""
    conf, out = run_processes(spawner, tmp_path, dict(CONF, die=die, dead_mode=dead_mode, **extra))
    log = out["log"]
    o, deaths = replay(torch, conf, log)
    assert o.ts == out["ts"] and o.pending() == 0
    w = np.load(tmp_path / "w.npy")
    v = np.load(tmp_path / "v.npy")
    assert parity.bitwise(w, o.w) and parity.bitwise(v, o.v)
    pushes = [sum(1 for e in log if e[0] == "push" and e[1] == l) for l in range(4)]
    applied = [o.applied_order.count(l) for l in range(4)]
    for l in range(4):
        if str(l) in die:
            assert pushes[l] == die[str(l)]
            assert len(deaths) == 1 and deaths[0][1] == l
            assert deaths[0][2] >= 1, "the learner died with nothing queued"
            if dead_mode == "retire":          # exactly once, dead or alive
                assert applied[l] == pushes[l]
            else:
                assert applied[l] == pushes[l] - deaths[0][2]
            assert not os.path.exists(tmp_path / f"learner{l}.json")
        else:
            assert pushes[l] == applied[l] == conf["pushes"][l]
            with open(tmp_path / f"learner{l}.json") as f:
                got = json.load(f)
            assert got["ts"] == o.ts
            want = hashlib.sha256(o.replicas[("replica", l)].tobytes()).hexdigest()
            assert got["replica_sha256"] == want
    if not die:
        assert deaths == []


def test_restart_from_checkpoint_in_new_processes(torch, spawner, tmp_path):
    """Sec. 4.3's restart across processes: after 5 applies the server takes
    no more pushes, tells its learners to stop (they detach), applies what
    is queued, writes a checkpoint and exits. A new server process loads it
    and four new learner processes push on. Both runs' logs replayed through
    one oracle (with its restart between them: pull history starts afresh,
    learners keep their timestamps) give the final w, v and replicas bit for
    bit."""
    ckpt = str(tmp_path / "ps.ckpt")
    base = dict(CONF, die={}, dead_mode="retire")
    c1, out1 = run_processes(spawner, tmp_path / "first",
                             dict(base, stop_after=5, checkpoint=ckpt))
    assert out1["log"][-1][0] == "checkpoint"
    c2, out2 = run_processes(spawner, tmp_path / "second",
                             dict(base, resume=ckpt, push_offset=3, pushes=[6, 6, 6, 6]))
    assert out2["log"][0] == ["resume", out1["ts"]]
    o, _ = replay(torch, c1, out1["log"])
    o, _ = replay(torch, c2, out2["log"], o)
    assert o.ts == out2["ts"] and o.pending() == 0
    second = tmp_path / "second"
    assert parity.bitwise(np.load(second / "w.npy"), o.w)
    assert parity.bitwise(np.load(second / "v.npy"), o.v)
    for l in range(4):
        with open(second / f"learner{l}.json") as f:
            got = json.load(f)
        assert got["ts"] == o.ts
        assert got["replica_sha256"] == hashlib.sha256(o.replicas[("replica", l)].tobytes()).hexdigest()
