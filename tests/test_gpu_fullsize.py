"""Whole-vector parity at full size (Eq. gd / Eq. asgd hold per coordinate).

The first full K-batches of every workload (all 200 of Tiny) with all
their pulls, in the launch configuration bench.py times (gradient pool and
replicas in server rows, the apply and the fan-out as separate calls). Every
replica written by every pull event is snapshotted on the device; then the
oracle runs block by block (at most 16M coordinates, gradient blocks copied
from the device pool per block, so host memory stays small) and every
coordinate of w, v and every snapshot is compared bit for bit.
"""
import sys

import numpy as np
import pytest

from oracle import server as orc
from paper_1611_06213_amd import ps
from paper_1611_06213_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu

BLOCK = 16 << 20


@pytest.fixture(scope="module")
def torch():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    ps.load_library()
    return torch


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def first_batches(cfg, count):
    """The schedule up to and including the pulls after its count-th apply."""
    out, applies = [], 0
    for ev in wl.schedule(cfg):
        if isinstance(ev, wl.Push) and applies == count:
            break
        out.append(ev)
        applies += isinstance(ev, wl.Apply)
    return out


@pytest.mark.parametrize("name,batches,mode", [
    ("vgg16", 3, "fifo"), ("mixed", 2, "fifo"), ("alexnet", 2, "fifo"), ("textcnn", 3, "fifo"),
    ("vgg16_shard8", 4, "fifo"), ("tiny", 200, "fifo"), ("vgg16", 3, "round-robin"),
    ("vgg16", 2, "ssgd")])
def test_workload_full_size_whole_vector(torch, name, batches, mode):
    """mode: fifo (the default queue), round-robin (per-learner queues of K
    slots, as bench.py --queue rr), ssgd (each apply a synchronous step over
    the batch, Eq. ssgd)."""
    cfg = wl.CONFIGS[name]
    events = first_batches(cfg, batches)
    n = cfg.n
    say(f"[whole] {name} {mode} n={n:,} events={len(events)}")
    rdt = torch.bfloat16 if cfg.pull_dtype == wl.BF16 else torch.float32
    srv = ps.ParameterServer(n, cfg.lr, cfg.momentum, queue_depth=cfg.depth)
    srv.set_stream(torch.cuda.current_stream())
    if mode == "round-robin":
        srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, cfg.depth)
    pool = srv.alloc_rows(cfg.pool, torch.bfloat16 if cfg.grad_dtype == wl.BF16 else torch.float32)
    reps = srv.alloc_rows(cfg.replicas, rdt)
    for j in range(cfg.pool):
        pool[j].copy_(wl.make_grad(cfg, j, "cuda"))
    for r in reps:
        r.zero_()
    w0 = wl.make_w0(cfg, "cuda")
    srv.set_weights(w0)
    snaps = []            # per pull event: {learner: device copy of its replica}
    stale = []
    for ev in events:
        if isinstance(ev, wl.Push):
            assert srv.push(ev.learner, pool[ev.buf])
        elif isinstance(ev, wl.Apply):
            if mode == "ssgd":
                srv.apply_sync()
            else:
                srv.apply_pending()
            stale += srv.last_staleness()
        else:
            for rnd in parity.pull_rounds(ev.learners):
                srv.pull_many(rnd, [reps[l] for l in rnd])
            snaps.append({l: reps[l].clone() for l in dict.fromkeys(ev.learners)})
    w = srv.weights_copy()
    v = srv.velocity_copy()
    torch.cuda.synchronize()
    say(f"[whole] {name}: GPU run done, {len(snaps)} pull events")

    bad = []
    for lo in range(0, n, BLOCK):
        hi = min(n, lo + BLOCK)
        o = orc.OracleServer(parity.np_bits(w0[lo:hi]), cfg.lr, cfg.momentum, depth=cfg.depth)
        if mode == "round-robin":
            assert o.set_queue_mode(orc.ROUND_ROBIN, cfg.depth) == orc.OK
        grads = {}
        k = 0
        for ev in events:
            if isinstance(ev, wl.Push):
                if ev.buf not in grads:
                    grads[ev.buf] = parity.np_bits(pool[ev.buf][lo:hi])
                assert o.push(ev.learner, grads[ev.buf]) == orc.OK
            elif isinstance(ev, wl.Apply):
                assert (o.apply_sync() if mode == "ssgd" else o.apply_pending()) == orc.OK
            else:
                for rnd in parity.pull_rounds(ev.learners):
                    for l in rnd:
                        o.pull(l, l, cfg.pull_dtype)
                for l, t in snaps[k].items():
                    if not parity.bitwise(parity.np_bits(t[lo:hi]), o.replicas[l]):
                        bad.append(f"pull event {k} learner {l} block {lo}")
                k += 1
        if not parity.bitwise(parity.np_bits(w[lo:hi]), o.w):
            bad.append(f"w block {lo}")
        if v is not None and not parity.bitwise(parity.np_bits(v[lo:hi]), o.v):
            bad.append(f"v block {lo}")
        if lo == 0:
            assert stale == o.staleness and srv.timestamp == o.ts
        del grads
        assert not bad, bad[:10]
    say(f"[whole] {name}: w, v and {sum(len(s) for s in snaps)} replicas equal over all "
        f"{n:,} coordinates")
    del snaps, pool, reps
    srv.close()
    torch.cuda.empty_cache()
