"""Seeded synthetic workloads for the ASGD parameter server.

This module is the only code shared by the HIP path and the oracle. It holds
the five workload configurations, seeded generators for the initial weights
and the gradient pool, and the event schedules (push / apply / pull) that a
parameter-server run replays. It holds none of the update arithmetic: no
step, no momentum, no rounding of weights, no staleness.

The paper's workloads are Torch models trained on NLC, CIFAR and ImageNet
data (Sec. 5.2, Table "task_description"). The server only ever sees flat
gradient-shaped buffers, so these seeded streams, shaped like the paper's
models, stand in for them; no dataset item is reproduced.

Seeding: base seed 20161118, config i uses base + i. Sub-streams:
0 = initial weights, 1 = gradient pool (one sub-seed per pool buffer),
2 = arrival order, 3 = lags / bursts.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import List, Sequence, Tuple

import numpy as np

SEED_BASE = 20161118

F32 = 0
BF16 = 1


@dataclass(frozen=True)
class Config:
    """One synthetic workload.

    n          -- number of fp32 parameters (one flat vector)
    tensors    -- (name, numel) list in layout order; the remainder up to n is
                  padding (Text-CNN) or absent
    learners   -- lambda, number of learner ids
    pushes     -- total gradient pushes in the schedule
    depth      -- K, queue depth = pushes folded per apply
    lr, momentum
    grad_dist  -- 'normal' | 'laplace' | 'normal_heavy'
    grad_scale -- sigma (normal) or b (laplace)
    grad_dtype -- F32 | BF16
    pull_dtype -- F32 | BF16
    arrival    -- 'rr_jitter' | 'iid' | 'bursts'
    pulls      -- 'after_push' | 'batch_learners' | 'lag' | 'all'
    replicas   -- number of replica buffers (one per learner id that pulls)
    pool       -- distinct gradient buffers; push j uses buffer j mod pool
    index      -- position in the config list (selects the seed)
    """

    name: str
    n: int
    learners: int
    pushes: int
    depth: int
    lr: float
    momentum: float
    grad_dist: str
    grad_scale: float
    grad_dtype: int
    pull_dtype: int
    arrival: str
    pulls: str
    replicas: int
    pool: int
    index: int
    tensors: Tuple[Tuple[str, int], ...] = field(default=())
    drain_each_burst: bool = False

    @property
    def seed(self) -> int:
        return SEED_BASE + self.index

    def scaled(self, n: int, pushes: int | None = None, pool: int | None = None) -> "Config":
        """Same workload at a smaller parameter count (parity tests)."""
        kw = {"n": n, "tensors": ()}
        if pushes is not None:
            kw["pushes"] = pushes
        if pool is not None:
            kw["pool"] = pool
        return dataclasses.replace(self, **kw)


def _textcnn_tensors():
    t = [
        ("embedding", 50000 * 100),
        ("conv3.weight", 3 * 100 * 300), ("conv3.bias", 300),
        ("conv4.weight", 4 * 100 * 300), ("conv4.bias", 300),
        ("conv5.weight", 5 * 100 * 300), ("conv5.bias", 300),
        ("fc1.weight", 900 * 1000), ("fc1.bias", 1000),
        ("fc2.weight", 1000 * 1000), ("fc2.bias", 1000),
    ]
    return tuple(t)


def _alexnet_tensors():
    convs = [(64, 3, 11), (192, 64, 5), (384, 192, 3), (256, 384, 3), (256, 256, 3)]
    t = []
    for i, (co, ci, k) in enumerate(convs, 1):
        t.append((f"conv{i}.weight", co * ci * k * k))
        t.append((f"conv{i}.bias", co))
    for name, (o, i) in (("fc6", (4096, 9216)), ("fc7", (4096, 4096)), ("fc8", (1000, 4096))):
        t.append((f"{name}.weight", o * i))
        t.append((f"{name}.bias", o))
    return tuple(t)


def _vgg16_tensors():
    chans = [64, 64, 128, 128, 256, 256, 256, 512, 512, 512, 512, 512, 512]
    t = []
    cin = 3
    for i, co in enumerate(chans, 1):
        t.append((f"conv{i}.weight", co * cin * 9))
        t.append((f"conv{i}.bias", co))
        cin = co
    for name, (o, i) in (("fc6", (4096, 25088)), ("fc7", (4096, 4096)), ("fc8", (1000, 4096))):
        t.append((f"{name}.weight", o * i))
        t.append((f"{name}.bias", o))
    return tuple(t)


CONFIGS = {
    "tiny": Config(
        name="tiny", n=1_048_576, learners=4, pushes=200, depth=1, lr=0.01, momentum=0.0,
        grad_dist="normal", grad_scale=0.01, grad_dtype=F32, pull_dtype=F32,
        arrival="rr_jitter", pulls="after_push", replicas=4, pool=200, index=0),
    "textcnn": Config(
        name="textcnn", n=10_000_000, learners=8, pushes=2000, depth=8, lr=0.01, momentum=0.0,
        grad_dist="normal", grad_scale=1e-3, grad_dtype=F32, pull_dtype=F32,
        arrival="iid", pulls="batch_learners", replicas=8, pool=64, index=1,
        tensors=_textcnn_tensors()),
    "alexnet": Config(
        name="alexnet", n=61_100_840, learners=16, pushes=1000, depth=16, lr=0.005, momentum=0.9,
        grad_dist="normal", grad_scale=1e-3, grad_dtype=F32, pull_dtype=F32,
        arrival="iid", pulls="lag", replicas=16, pool=64, index=2,
        tensors=_alexnet_tensors()),
    "vgg16": Config(
        name="vgg16", n=138_357_544, learners=16, pushes=500, depth=32, lr=0.001, momentum=0.9,
        grad_dist="laplace", grad_scale=1e-3, grad_dtype=F32, pull_dtype=F32,
        arrival="iid", pulls="all", replicas=16, pool=64, index=3,
        tensors=_vgg16_tensors()),
    "mixed": Config(
        name="mixed", n=200_000_000, learners=32, pushes=400, depth=32, lr=0.001, momentum=0.9,
        grad_dist="normal_heavy", grad_scale=1e-3, grad_dtype=BF16, pull_dtype=BF16,
        arrival="bursts", pulls="all", replicas=32, pool=64, index=4),
    # one GPU's share of VGG-16 split eight ways by coordinates (a sharded
    # server applies the same pushes to each contiguous eighth)
    "vgg16_shard8": Config(
        name="vgg16_shard8", n=(138_357_544 + 7) // 8, learners=16, pushes=500, depth=32,
        lr=0.001, momentum=0.9, grad_dist="laplace", grad_scale=1e-3, grad_dtype=F32,
        pull_dtype=F32, arrival="iid", pulls="all", replicas=16, pool=64, index=5),
}


def tensor_offsets(cfg: Config) -> List[Tuple[str, int, int]]:
    """(name, start, numel) of each listed tensor in the flat vector."""
    out, off = [], 0
    for name, numel in cfg.tensors:
        out.append((name, off, numel))
        off += numel
    if cfg.tensors and off < cfg.n:
        out.append(("pad", off, cfg.n - off))
    return out


# ---------------------------------------------------------------- schedules

@dataclass(frozen=True)
class Push:
    learner: int
    buf: int          # index into the gradient pool


@dataclass(frozen=True)
class Apply:
    pass


@dataclass(frozen=True)
class Pull:
    learners: Tuple[int, ...]   # learner r pulls into replica buffer r


Event = object


def _rng(cfg: Config, stream: int) -> np.random.Generator:
    return np.random.default_rng([cfg.seed, stream])


def arrival_order(cfg: Config) -> Tuple[List[int], List[int]]:
    """Learner id of each push in arrival order, and burst ends (bursts only)."""
    r = _rng(cfg, 2)
    if cfg.arrival == "rr_jitter":
        # push j nominally from learner j mod lambda, key j + U(-1.5, 1.5),
        # stable sort; a learner's own pushes keep their order (keys 4 apart).
        keys = np.arange(cfg.pushes) + r.uniform(-1.5, 1.5, cfg.pushes)
        order = np.argsort(keys, kind="stable")
        return [int(j % cfg.learners) for j in order], []
    if cfg.arrival == "iid":
        return [int(x) for x in r.integers(0, cfg.learners, cfg.pushes)], []
    if cfg.arrival == "bursts":
        rb = _rng(cfg, 3)
        learners, ends = [], []
        while len(learners) < cfg.pushes:
            b = min(1 + int(rb.poisson(7.0)), cfg.learners, cfg.pushes - len(learners))
            learners.extend(int(x) for x in r.choice(cfg.learners, size=b, replace=False))
            ends.append(len(learners))
        return learners, ends
    raise ValueError(cfg.arrival)


def schedule(cfg: Config) -> List[Event]:
    """The event list a run replays, in order.

    Push j uses pool buffer j mod pool. Apply events fold the pending pushes.
    Pull events name the learners that pull (learner r into replica r).
    """
    learners, burst_ends = arrival_order(cfg)
    ev: List[Event] = []
    pending = 0
    if cfg.pulls == "lag":
        lags = _rng(cfg, 3).integers(0, 16, cfg.pushes)
        due: dict = {}
        for j, l in enumerate(learners):
            due.setdefault(j + int(lags[j]), []).append(l)
        late = []
        for j, l in enumerate(learners):
            ev.append(Push(l, j % cfg.pool))
            pending += 1
            if pending == cfg.depth:
                ev.append(Apply())
                pending = 0
            if j in due:
                ev.append(Pull(tuple(due.pop(j))))
        for k in sorted(due):
            late.extend(due[k])
        if pending:
            ev.append(Apply())
        if late:
            ev.append(Pull(tuple(late)))
        return ev

    ends = set(burst_ends) if cfg.drain_each_burst else set()
    batch: List[int] = []
    for j, l in enumerate(learners):
        ev.append(Push(l, j % cfg.pool))
        batch.append(l)
        pending += 1
        last = j == len(learners) - 1
        if pending == cfg.depth or last or (j + 1) in ends:
            ev.append(Apply())
            if cfg.pulls == "after_push":
                ev.append(Pull(tuple(dict.fromkeys(batch))))
            elif cfg.pulls == "batch_learners":
                ev.append(Pull(tuple(dict.fromkeys(batch))))
            elif cfg.pulls == "all":
                ev.append(Pull(tuple(range(cfg.replicas))))
            else:
                raise ValueError(cfg.pulls)
            batch = []
            pending = 0
    return ev


# ---------------------------------------------------------------- tensors

def _torch():
    import torch  # local: the schedule part above needs numpy only
    return torch


def _gen(device, *key: int):
    torch = _torch()
    g = torch.Generator(device=device)
    # a 63-bit seed derived from the key tuple (numpy's SeedSequence mixing)
    s = int(np.random.SeedSequence(list(key)).generate_state(2, dtype=np.uint32).view(np.uint64)[0])
    g.manual_seed(s & ((1 << 63) - 1))
    return g


def make_w0(cfg: Config, device="cpu"):
    """Initial weights w0 ~ U(-0.05, 0.05), fp32."""
    torch = _torch()
    g = _gen(device, cfg.seed, 0)
    return (torch.rand(cfg.n, generator=g, device=device, dtype=torch.float32) - 0.5) * 0.1


def make_grad_f32(cfg: Config, buf: int, device="cpu"):
    """The fp32 gradient behind pool buffer `buf` (before any bf16 rounding)."""
    torch = _torch()
    g = _gen(device, cfg.seed, 1, buf)
    n = cfg.n
    if cfg.grad_dist == "normal":
        return torch.randn(n, generator=g, device=device) * cfg.grad_scale
    if cfg.grad_dist == "laplace":
        # Laplace(0, b) as the difference of two unit exponentials, times b
        e1 = torch.empty(n, device=device).exponential_(1.0, generator=g)
        e2 = torch.empty(n, device=device).exponential_(1.0, generator=g)
        return (e1 - e2) * cfg.grad_scale
    if cfg.grad_dist == "normal_heavy":
        x = torch.randn(n, generator=g, device=device) * cfg.grad_scale
        mask = torch.rand(n, generator=g, device=device) < 0.01
        return torch.where(mask, x * 100.0, x)
    raise ValueError(cfg.grad_dist)


def make_grad(cfg: Config, buf: int, device="cpu"):
    """Pool buffer `buf` in the config's gradient dtype (bf16 by torch's cast)."""
    torch = _torch()
    x = make_grad_f32(cfg, buf, device)
    if cfg.grad_dtype == BF16:
        return x.to(torch.bfloat16)
    return x


ROW_ALIGN = 2 << 20     # bytes: each buffer starts on a 2 MiB boundary ...
ROW_STAGGER = 4096      # ... plus 4 KiB per row, so rows do not share a DRAM phase


class Rows:
    """`count` buffers of n elements, carved from one allocation on aligned,
    staggered row starts (row r at r * stride): each starts on a 2 MiB
    boundary plus r * 4 KiB, the layout of the server's own rows, here
    without a server (tests, oracle-side copies). Buffers laid out back to
    back n*4 bytes apart would start at arbitrary 32-byte offsets for most n,
    and separately allocated ones all at one offset within 2 MiB; streaming
    kernels lose bandwidth on both."""

    def __init__(self, count: int, n: int, dtype, device="cpu", align: int = ROW_ALIGN,
                 stagger: int = ROW_STAGGER):
        torch = _torch()
        es = torch.empty((), dtype=dtype).element_size()
        a, st = align // es, stagger // es
        self.stride = (n + a - 1) // a * a + st
        self.n = n
        self.count = count
        self.buf = torch.empty(count * self.stride, dtype=dtype, device=device)
        self.rows = [self.buf[i * self.stride: i * self.stride + n] for i in range(count)]

    def __getitem__(self, i):
        return self.rows[i]

    def __len__(self):
        return self.count


def make_pool(cfg: Config, device="cpu") -> Rows:
    """The gradient pool: buffer j = make_grad(cfg, j), as aligned rows."""
    torch = _torch()
    dt = torch.bfloat16 if cfg.grad_dtype == BF16 else torch.float32
    pool = Rows(cfg.pool, cfg.n, dt, device)
    for j in range(cfg.pool):
        pool[j].copy_(make_grad(cfg, j, device))
    return pool


def sample_ranges(n: int, width: int = 4096, count: int = 6, seed: int = 0) -> List[Tuple[int, int]]:
    """Coordinate ranges for sampled parity at full size: the head, the tail
    (which holds the ragged end) and seeded interior blocks."""
    width = min(width, n)
    out = [(0, width), (n - width, n)]
    r = np.random.default_rng([SEED_BASE, 99, seed])
    for _ in range(max(0, count - 2)):
        lo = int(r.integers(0, max(1, n - width)))
        out.append((lo, lo + width))
    return out
