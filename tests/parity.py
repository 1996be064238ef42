"""Replay one workload schedule on the GPU (through the C ABI) and in the
oracle, on the same seeded inputs, and compare what both produce.

The GPU run keeps the whole vector; the oracle runs on coordinate ranges
(every step is per coordinate, so a range run is the full run restricted to
those coordinates). For each pull event the replicas it refreshed are
snapshotted on both sides and compared, as are the final weights, the
velocity, each applied gradient's staleness and the counters.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from oracle import server as orc
from paper_1611_06213_amd import ps
from paper_1611_06213_amd import workloads as wl


def np_bits(t) -> np.ndarray:
    """CPU numpy view of a torch tensor: float32 values or bf16 bit patterns."""
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def pull_rounds(learners: Sequence[int]) -> List[List[int]]:
    """Split a pull event into calls without repeated learners (first
    occurrences, then second occurrences, ...), applied in order."""
    rounds: List[List[int]] = []
    seen: Dict[int, int] = {}
    for l in learners:
        k = seen.get(l, 0)
        seen[l] = k + 1
        if k == len(rounds):
            rounds.append([])
        rounds[k].append(l)
    return rounds


def gpu_replay(cfg: wl.Config, events, pool, w0, ranges: Sequence[Tuple[int, int]],
               fused: bool = False, pull_skip: bool = True, stream=None, fusion=None,
               replicas=None, round_robin: bool = False):
    """fused: drive apply+pull through ps_apply_pull; fusion: the replica
    count up to which that call writes replicas from the apply pass;
    replicas: the replica tensors (default: workloads.Rows); round_robin:
    per-learner queues of `depth` slots served round-robin (as bench.py
    --queue rr sets them)."""
    import torch
    srv = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=cfg.depth)
    if round_robin:
        srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, cfg.depth)
    srv.set_pull_skip(pull_skip)
    if fusion is not None:
        srv.set_pull_fusion(fusion)
    srv.set_stream(stream or torch.cuda.current_stream())
    srv.set_weights(w0)
    rdt = torch.bfloat16 if cfg.pull_dtype == wl.BF16 else torch.float32
    if replicas is None:
        replicas = wl.Rows(cfg.replicas, cfg.n, rdt, "cuda")
        replicas.buf.zero_()
    else:
        for r in replicas:
            r.zero_()
    snaps, stale = [], []

    widths = [hi - lo for lo, hi in ranges]

    def snap(learners):
        # one gather and one device-to-host copy per pull event
        ls = list(dict.fromkeys(learners))
        rows = np_bits(torch.stack([torch.cat([replicas[l][lo:hi] for lo, hi in ranges])
                                    for l in ls]))
        d = {}
        for j, l in enumerate(ls):
            parts, off = [], 0
            for wdt in widths:
                parts.append(rows[j, off:off + wdt].copy())
                off += wdt
            d[l] = parts
        snaps.append(d)

    i = 0
    while i < len(events):
        ev = events[i]
        if isinstance(ev, wl.Push):
            assert srv.push(ev.learner, pool[ev.buf])
        elif isinstance(ev, wl.Apply):
            nxt = events[i + 1] if i + 1 < len(events) else None
            if fused and isinstance(nxt, wl.Pull):
                rounds = pull_rounds(nxt.learners)
                srv.apply_pull(rounds[0], [replicas[l] for l in rounds[0]])
                stale += srv.last_staleness()
                for r in rounds[1:]:
                    srv.pull_many(r, [replicas[l] for l in r])
                snap(nxt.learners)
                i += 2
                continue
            srv.apply_pending()
            stale += srv.last_staleness()
        else:
            for r in pull_rounds(ev.learners):
                srv.pull_many(r, [replicas[l] for l in r])
            snap(ev.learners)
        i += 1
    w = srv.weights_copy()
    v = srv.velocity_copy()
    st = srv.stats()
    out = {
        "w": [np_bits(w[lo:hi]) for lo, hi in ranges],
        "v": None if v is None else [np_bits(v[lo:hi]) for lo, hi in ranges],
        "snaps": snaps,
        "staleness": stale,
        "ts": srv.timestamp,
        "counts": (st.pushes_accepted, st.pushes_applied, st.pulls, st.pulls_skipped),
    }
    srv.close()
    del replicas
    return out


def oracle_replay(cfg: wl.Config, events, pool_slices, w0_slices, ranges, pull_skip: bool = True,
                  round_robin: bool = False):
    """pool_slices[r][buf] is pool buffer `buf` restricted to range r."""
    per_range = []
    for r, (lo, hi) in enumerate(ranges):
        s = orc.OracleServer(w0_slices[r], cfg.lr, cfg.momentum, depth=cfg.depth,
                             pull_skip=pull_skip)
        if round_robin:
            assert s.set_queue_mode(orc.ROUND_ROBIN, cfg.depth) == orc.OK
        snaps = []

        def on_pull(learners, srv, snaps=snaps):
            snaps.append({l: srv.replicas[l].copy() for l in learners})

        def grads(buf, r=r):
            return pool_slices[r][buf]

        for ev in events:
            if isinstance(ev, wl.Pull):
                for rnd in pull_rounds(ev.learners):
                    for l in rnd:
                        s.pull(l, l, cfg.pull_dtype)
                on_pull(ev.learners, s)
            elif isinstance(ev, wl.Push):
                assert s.push(ev.learner, grads(ev.buf)) == orc.OK
            else:
                s.apply_pending()
        per_range.append((s, snaps))
    s0 = per_range[0][0]
    return {
        "w": [s.w for s, _ in per_range],
        "v": None if s0.v is None else [s.v for s, _ in per_range],
        "snaps": [{l: [per_range[r][1][k][l] for r in range(len(ranges))] for l in per_range[0][1][k]}
                  for k in range(len(per_range[0][1]))],
        "staleness": s0.staleness,
        "ts": s0.ts,
        "counts": (s0.ts + s0.pending(), s0.ts, s0.pulls, s0.pulls_skipped),
    }


def host_inputs(cfg: wl.Config, pool, w0, ranges):
    """Slices of the device inputs for the oracle (same bits)."""
    pool_slices = [[np_bits(pool[b][lo:hi]) for b in range(cfg.pool)] for lo, hi in ranges]
    w0_slices = [np_bits(w0[lo:hi]) for lo, hi in ranges]
    return pool_slices, w0_slices


def bitwise(a: np.ndarray, b: np.ndarray) -> bool:
    a = np.asarray(a)
    b = np.asarray(b)
    if a.dtype == np.float32:
        a = a.view(np.uint32)
    if b.dtype == np.float32:
        b = b.view(np.uint32)
    return a.shape == b.shape and bool(np.array_equal(a, b))


def compare(gpu, ora, ranges) -> List[str]:
    """All mismatches between a GPU run and an oracle run ([] = identical)."""
    bad = []
    for r in range(len(ranges)):
        if not bitwise(gpu["w"][r], ora["w"][r]):
            d = np.nonzero(gpu["w"][r].view(np.uint32) != ora["w"][r].view(np.uint32))[0]
            bad.append(f"w range {ranges[r]}: {d.size} coords differ, first at +{d[0]}")
        if (gpu["v"] is None) != (ora["v"] is None):
            bad.append("velocity presence differs")
        elif gpu["v"] is not None and not bitwise(gpu["v"][r], ora["v"][r]):
            bad.append(f"v range {ranges[r]} differs")
    if len(gpu["snaps"]) != len(ora["snaps"]):
        bad.append(f"pull events {len(gpu['snaps'])} vs {len(ora['snaps'])}")
    else:
        for k, (gs, os_) in enumerate(zip(gpu["snaps"], ora["snaps"])):
            for l in os_:
                for r in range(len(ranges)):
                    if not bitwise(gs[l][r], os_[l][r]):
                        bad.append(f"pull event {k} learner {l} range {ranges[r]} differs")
                        break
    if gpu["staleness"] != ora["staleness"]:
        bad.append("staleness differs")
    if gpu["ts"] != ora["ts"]:
        bad.append(f"ts {gpu['ts']} vs {ora['ts']}")
    if gpu["counts"] != ora["counts"]:
        bad.append(f"counts {gpu['counts']} vs {ora['counts']}")
    return bad
