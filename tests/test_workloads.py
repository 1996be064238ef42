"""The synthetic workloads: shapes, schedules and seeded generators."""
import numpy as np
import pytest

from paper_1611_06213_amd import workloads as wl


def test_model_sizes():
    """Tensor lists add up to the architectures' parameter counts: VGG-16
    (13 conv + 3 fc) 138,357,544; AlexNet (5 conv + 3 fc) 61,100,840; the
    Text-CNN tensors 7,262,900 (padded to 10M)."""
    tot = lambda c: sum(x for _, x in c.tensors)
    assert tot(wl.CONFIGS["vgg16"]) == 138_357_544 == wl.CONFIGS["vgg16"].n
    assert tot(wl.CONFIGS["alexnet"]) == 61_100_840 == wl.CONFIGS["alexnet"].n
    assert tot(wl.CONFIGS["textcnn"]) == 7_262_900
    offs = wl.tensor_offsets(wl.CONFIGS["textcnn"])
    assert offs[-1] == ("pad", 7_262_900, 2_737_100)


def _count(ev):
    pushes = [e for e in ev if isinstance(e, wl.Push)]
    applies, sizes, pend, pulls = 0, [], 0, 0
    for e in ev:
        if isinstance(e, wl.Push):
            pend += 1
        elif isinstance(e, wl.Apply):
            applies += 1
            sizes.append(pend)
            pend = 0
        else:
            pulls += len(e.learners)
    return len(pushes), applies, sizes, pend, pulls


@pytest.mark.parametrize("name,applies,last", [
    ("tiny", 200, 1), ("textcnn", 250, 8), ("alexnet", 63, 8), ("vgg16", 16, 20), ("mixed", 13, 16)])
def test_schedule_shape(name, applies, last):
    cfg = wl.CONFIGS[name]
    ev = wl.schedule(cfg)
    n, a, sizes, pend, pulls = _count(ev)
    assert n == cfg.pushes and a == applies and pend == 0
    assert sizes[-1] == last and all(s == cfg.depth for s in sizes[:-1])
    assert all(0 < s <= cfg.depth for s in sizes)
    for e in ev:
        if isinstance(e, wl.Push):
            assert 0 <= e.learner < cfg.learners and 0 <= e.buf < cfg.pool
        if isinstance(e, wl.Pull):
            assert all(0 <= l < cfg.replicas for l in e.learners)


def test_schedule_specifics():
    # Tiny: round-robin with jitter keeps each learner's pushes in order and
    # pulls by the pushing learner after every push
    cfg = wl.CONFIGS["tiny"]
    learners, _ = wl.arrival_order(cfg)
    assert sorted(learners) == sorted(j % 4 for j in range(200))
    ev = wl.schedule(cfg)
    for a, b, c in zip(ev, ev[1:], ev[2:]):
        if isinstance(a, wl.Push):
            assert isinstance(b, wl.Apply) and c.learners == (a.learner,)
    # VGG-16: all 16 replicas after each apply
    ev = wl.schedule(wl.CONFIGS["vgg16"])
    assert all(e.learners == tuple(range(16)) for e in ev if isinstance(e, wl.Pull))
    # Mixed: bursts of distinct learners, mean size near 8
    cfg = wl.CONFIGS["mixed"]
    learners, ends = wl.arrival_order(cfg)
    starts = [0] + ends[:-1]
    for s, e in zip(starts, ends):
        assert len(set(learners[s:e])) == e - s
    assert 6 < np.mean(np.diff([0] + ends)) < 10
    # parity variant: an apply at every burst end, variable K <= 32
    import dataclasses
    ev = wl.schedule(dataclasses.replace(cfg, drain_each_burst=True))
    _, a, sizes, _, _ = _count(ev)
    assert a >= len(ends) and max(sizes) <= 32 and min(sizes) >= 1
    # AlexNet: lagged pulls, about one per push
    _, _, _, _, pulls = _count(wl.schedule(wl.CONFIGS["alexnet"]))
    assert pulls == 1000


def test_generators_seeded_and_shaped():
    torch = pytest.importorskip("torch")
    for name in wl.CONFIGS:
        cfg = wl.CONFIGS[name].scaled(5000, pool=3)
        a = wl.make_grad(cfg, 1)
        b = wl.make_grad(cfg, 1)
        c = wl.make_grad(cfg, 2)
        assert torch.equal(a, b) and not torch.equal(a, c)
        assert a.dtype == (torch.bfloat16 if name == "mixed" else torch.float32)
        w0 = wl.make_w0(cfg)
        assert w0.dtype == torch.float32 and float(w0.abs().max()) <= 0.05
    # spread of the gradient distributions (loose: 5000 samples)
    g = wl.make_grad_f32(wl.CONFIGS["vgg16"].scaled(200000), 0)
    assert abs(float(g.abs().mean()) - 1e-3) < 5e-5          # Laplace mean |x| = b
    g = wl.make_grad_f32(wl.CONFIGS["mixed"].scaled(200000), 0)
    assert 0.005 < float((g.abs() > 5e-3).float().mean()) < 0.015   # the x100 tail


def test_sample_ranges():
    r = wl.sample_ranges(10_000_003, 4096, 6)
    assert r[0] == (0, 4096) and r[1] == (10_000_003 - 4096, 10_000_003)
    assert all(0 <= lo < hi <= 10_000_003 for lo, hi in r)
