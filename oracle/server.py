"""Sequential ASGD parameter server, written plainly (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
module; the product path never imports it.

What it follows (GaDei, arXiv 1611.06213):
  * Sec. 2.1, Fig. "design_base": learners push gradients to the server and
    pull weights from it; they never talk to each other.
  * Eq. "asgd" with the step of Eq. "gd": each received gradient is applied on
    its own, in the order it was received.
  * Sec. 2.1: the server's scalar timestamp grows by one per update; the
    staleness of a gradient is the server timestamp minus the timestamp of
    the weights the learner held.
  * Sec. 4.1 and Lemma 1 / Theorem 2 (Sec. 4.2): gradients wait in a FIFO with
    a fixed number of slots; a full queue refuses the pusher; each queued
    gradient is applied exactly once.
  * Sec. 4.1: a pull is skipped when the learner's copy already carries the
    server's timestamp.

Synchronous SGD (Eq. "ssgd") is also provided: apply_sync() averages the
pending gradients (one per learner), summed in queue order, and applies one
update.

Round-robin mode (set_queue_mode(ROUND_ROBIN, slots)) follows Sec. 4.1 more
literally: every learner has its own FIFO with a fixed number of slots (the
lambda single-producer single-consumer queues) and a push on a full one is
refused (Lemma 1 per learner). The server visits the learners in increasing
id order, cyclically, starting after the learner it served last, and takes
one gradient per visit of a non-empty queue; an apply takes up to `depth`
gradients this way. A synchronous step takes one gradient from every
non-empty queue, summed in increasing learner order (Eq. "ssgd" sums over
l = 1..lambda).

Dead learners (Sec. 4.3): drop_learner discards a dead learner's queued
gradients (its buffers may have died with it); retire_learner keeps them
queued, to be applied exactly once in their turn, as the paper's stateless
server does with gradients already in its shared slots.

Readings where the paper is silent:
  * one global FIFO in push-call order stands in for the per-learner queues;
  * a batch of K pending gradients is applied as K sequential steps, each over
    the whole vector, oldest first;
  * a full queue returns EFULL instead of blocking;
  * momentum, when non-zero, is heavy-ball kept on the server (v0 = +0);
  * the staleness of a push uses the timestamp the learner held when it
    pushed; every learner starts holding w0 at timestamp 0;
  * a pull is skipped iff the same learner pulls into the same buffer with
    the same dtype and the timestamp has not moved since its last pull.

Parity unpinned against the paper (pinned only to the reading itself, by the
tests' closed forms and hand-worked scripts): the momentum step, which the
paper does not have, and round-robin service taking one gradient per visit,
which the paper states in a listing that is not in its text.

The oracle can be run on any coordinate range [lo, hi) of a workload: every
step is per coordinate (Eq. "gd" is written for the k-th parameter), so the
range run is exactly the full run restricted to those coordinates.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Tuple

import numpy as np

FIFO = 0
ROUND_ROBIN = 1

OK = 0
EINVAL = -1
EFULL = -2
ESTATE = -5

F32 = 0
BF16 = 1

MAX_DEPTH = 64

_HERE = os.path.dirname(os.path.abspath(__file__))
_lib = None


def lib():
    """Load oracle/liboracle.so, compiling it with gcc if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    path = os.path.join(_HERE, "liboracle.so")
    src = os.path.join(_HERE, "asgd_oracle.c")
    if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(src):
        from . import build
        build.build()
    L = ctypes.CDLL(path)
    fp = ctypes.POINTER(ctypes.c_float)
    up = ctypes.POINTER(ctypes.c_uint16)
    sz = ctypes.c_size_t
    fl = ctypes.c_float
    L.orc_step_f32.argtypes = [fp, fp, sz, fl]
    L.orc_step_mom_f32.argtypes = [fp, fp, fp, sz, fl, fl]
    L.orc_step_bf16.argtypes = [fp, up, sz, fl]
    L.orc_step_mom_bf16.argtypes = [fp, fp, up, sz, fl, fl]
    L.orc_pull_f32.argtypes = [fp, fp, sz]
    L.orc_pull_bf16.argtypes = [up, fp, sz]
    L.orc_widen_bf16.argtypes = [fp, up, sz]
    L.orc_widen_bf16.restype = None
    L.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
    L.orc_bf16_to_f32.restype = ctypes.c_float
    L.orc_f32_to_bf16.argtypes = [ctypes.c_float]
    L.orc_f32_to_bf16.restype = ctypes.c_uint16
    L.orc_ssgd_step.argtypes = [fp, fp, ctypes.POINTER(ctypes.c_void_p), ctypes.c_int,
                                ctypes.c_int, sz, fl, fl]
    for f in ("orc_step_f32", "orc_step_mom_f32", "orc_step_bf16", "orc_step_mom_bf16",
              "orc_pull_f32", "orc_pull_bf16", "orc_ssgd_step"):
        getattr(L, f).restype = None
    _lib = L
    return L


def _fp(a: np.ndarray):
    assert a.dtype == np.float32 and a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _up(a: np.ndarray):
    assert a.dtype == np.uint16 and a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16))


# ------------------------------------------------------------ single steps

def step(w: np.ndarray, g: np.ndarray, lr: float, v: Optional[np.ndarray] = None,
         momentum: float = 0.0) -> None:
    """One ASGD step in place on w (and v). g is float32, or uint16 holding
    bf16 bit patterns. With v given, the momentum form is used."""
    L = lib()
    n = w.size
    assert g.size == n
    if v is None:
        if g.dtype == np.uint16:
            L.orc_step_bf16(_fp(w), _up(g), n, lr)
        else:
            L.orc_step_f32(_fp(w), _fp(g), n, lr)
    else:
        if g.dtype == np.uint16:
            L.orc_step_mom_bf16(_fp(w), _fp(v), _up(g), n, lr, momentum)
        else:
            L.orc_step_mom_f32(_fp(w), _fp(v), _fp(g), n, lr, momentum)


def ssgd_step(w: np.ndarray, grads, lr: float, v: Optional[np.ndarray] = None,
              momentum: float = 0.0) -> None:
    """One synchronous step (Eq. "ssgd") in place: average of `grads` (all
    float32, or all uint16 bf16 bit patterns) in list order, then one step."""
    L = lib()
    n = w.size
    is_bf16 = grads[0].dtype == np.uint16
    for g in grads:
        assert g.size == n and (g.dtype == np.uint16) == is_bf16 and g.flags.c_contiguous
    ptrs = (ctypes.c_void_p * len(grads))(*[g.ctypes.data for g in grads])
    vp = _fp(v) if v is not None else None
    L.orc_ssgd_step(_fp(w), vp, ptrs, len(grads), int(is_bf16), n, lr, momentum)


def pull_copy(w: np.ndarray, dtype: int) -> np.ndarray:
    """The replica a pull writes: w itself (fp32) or w rounded to bf16 bits."""
    L = lib()
    if dtype == F32:
        out = np.empty_like(w)
        L.orc_pull_f32(_fp(out), _fp(w), w.size)
    else:
        out = np.empty(w.size, np.uint16)
        L.orc_pull_bf16(_up(out), _fp(w), w.size)
    return out


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    return pull_copy(np.ascontiguousarray(x, dtype=np.float32), BF16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    out = np.empty(b.size, np.float32)
    lib().orc_widen_bf16(_fp(out), _up(b), b.size)
    return out


# ------------------------------------------------------------ the server

class OracleServer:
    """Single-threaded sequential ASGD server over a coordinate range."""

    def __init__(self, w0: np.ndarray, lr: float, momentum: float = 0.0, depth: int = 32,
                 pull_skip: bool = True):
        self.w = np.array(w0, dtype=np.float32, copy=True)
        self.lr = float(np.float32(lr))
        self.momentum = float(np.float32(momentum))
        self.v = np.zeros_like(self.w) if self.momentum != 0.0 else None
        if not 1 <= depth <= MAX_DEPTH:
            raise ValueError("depth")
        self.depth = depth
        self.pull_skip = pull_skip
        self.ts = 0
        self.queue: List[Tuple[int, np.ndarray, int]] = []   # (learner, grad, learner ts)
        self.learner_ts: Dict[int, int] = {}
        self.last_pull: Dict[int, Tuple[object, int, int]] = {}
        self.replicas: Dict[object, np.ndarray] = {}
        self.staleness: List[int] = []        # one entry per applied push, in order
        self.applied_order: List[int] = []    # learner of each applied push
        self.pulls = 0
        self.pulls_skipped = 0
        self.mode = FIFO
        self.slots = 0
        self.per_learner: Dict[int, List[Tuple[int, np.ndarray, int]]] = {}
        self.last_served = -1
        self.retired = set()

    def set_queue_mode(self, mode: int, slots: int = 1) -> int:
        if mode not in (FIFO, ROUND_ROBIN) or not 1 <= slots <= MAX_DEPTH:
            return EINVAL
        if self.pending():
            return ESTATE
        self.mode, self.slots = mode, slots
        return OK

    def pending(self) -> int:
        if self.mode == ROUND_ROBIN:
            return sum(len(q) for q in self.per_learner.values())
        return len(self.queue)

    def push(self, learner: int, grad: np.ndarray) -> int:
        if learner < 0:
            return EINVAL
        if learner in self.retired:
            return ESTATE
        entry = (learner, grad, self.learner_ts.get(learner, 0))
        if self.mode == ROUND_ROBIN:
            q = self.per_learner.setdefault(learner, [])
            if len(q) == self.slots:
                return EFULL
            q.append(entry)
            return OK
        if len(self.queue) == self.depth:
            return EFULL
        self.queue.append(entry)
        return OK

    def _round_robin_batch(self) -> List[Tuple[int, np.ndarray, int]]:
        """Visit learners in increasing id order, cyclically, starting after
        the last one served; one gradient per visit; at most `depth`."""
        batch = []
        while len(batch) < self.depth:
            waiting = sorted(l for l, q in self.per_learner.items() if q)
            if not waiting:
                break
            after = [l for l in waiting if l > self.last_served]
            nxt = after[0] if after else waiting[0]
            batch.append(self.per_learner[nxt].pop(0))
            self.last_served = nxt
        return batch

    def apply_pending(self) -> int:
        if self.mode == ROUND_ROBIN:
            batch = self._round_robin_batch()
        else:
            batch, self.queue = self.queue, []
        for learner, g, lts in batch:
            self.staleness.append(self.ts - lts)
            self.applied_order.append(learner)
            step(self.w, g, self.lr, self.v, self.momentum)
            self.ts += 1
        return OK

    def apply_sync(self) -> int:
        """Synchronous step (Eq. "ssgd"): the average of the pending gradients
        (FIFO mode: all of them, in queue order; round-robin mode: the oldest
        of every non-empty learner queue, in increasing learner order),
        applied as one update; the timestamp grows by one. The gradients of
        a step must share a dtype."""
        if self.mode == ROUND_ROBIN:
            batch = [self.per_learner[l][0] for l in sorted(self.per_learner) if self.per_learner[l]]
        else:
            batch = list(self.queue)
        if not batch:
            return OK
        if len({g.dtype for _, g, _ in batch}) != 1:
            return EINVAL
        if self.mode == ROUND_ROBIN:
            for l, _, _ in batch:
                self.per_learner[l].pop(0)
        else:
            self.queue = []
        for learner, _, lts in batch:
            self.staleness.append(self.ts - lts)
            self.applied_order.append(learner)
        ssgd_step(self.w, [g for _, g, _ in batch], self.lr, self.v, self.momentum)
        self.ts += 1
        return OK

    def pull(self, learner: int, dst_key, dtype: int = F32) -> bool:
        """Refresh replica `dst_key` for `learner`. Returns False if skipped.
        A retired learner pulls no more (ValueError)."""
        if learner in self.retired:
            raise ValueError(f"learner {learner} has retired")
        self.pulls += 1
        key = (dst_key, dtype, self.ts)
        if self.pull_skip and self.last_pull.get(learner) == key:
            self.pulls_skipped += 1
            return False
        self.replicas[dst_key] = pull_copy(self.w, dtype)
        self.last_pull[learner] = key
        self.learner_ts[learner] = self.ts
        return True

    def retire_learner(self, learner: int) -> int:
        """A learner died (Sec. 4.3) while its gradients sat in the server's
        own slots. The server is stateless -- it processes the gradients in
        its queues without regard to who produced them -- so those gradients
        stay queued and are applied exactly once in their turn (Theorem 2);
        the dead learner pushes and pulls no more. Returns how many of its
        gradients are still queued."""
        if learner < 0:
            return EINVAL
        self.retired.add(learner)
        if self.mode == ROUND_ROBIN:
            return len(self.per_learner.get(learner, []))
        return sum(1 for e in self.queue if e[0] == learner)

    def drop_learner(self, learner: int) -> int:
        """A learner died (Sec. 4.3): its queued gradients are discarded, the
        others keep their order. Returns how many were dropped."""
        if self.mode == ROUND_ROBIN:
            q = self.per_learner.get(learner, [])
            dropped = len(q)
            self.per_learner[learner] = []
            return dropped
        keep = [e for e in self.queue if e[0] != learner]
        dropped = len(self.queue) - len(keep)
        self.queue = keep
        return dropped

    def restart(self) -> int:
        """Resume from a checkpoint (Sec. 4.3: the server restarts from its
        last checkpoint and the learners are restarted): weights, velocity,
        timestamp, every learner's timestamp and the round-robin position are
        what was saved; pull history starts afresh (the restarted learners
        pull again) and every learner is live again. Like a checkpoint it needs
        an empty queue."""
        if self.pending():
            return ESTATE
        self.last_pull = {}
        self.retired = set()
        return OK

    def set_depth(self, depth: int) -> int:
        if not 1 <= depth <= MAX_DEPTH:
            return EINVAL
        if self.mode == FIFO and depth < len(self.queue):
            return ESTATE
        self.depth = depth
        return OK
