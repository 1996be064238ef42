"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar: bitwise for fp32 weights, velocities and replicas and for bf16 replica
bits (the library is built without contraction, like the oracle); exact
integers for timestamps, staleness and counters. This holds for the
bf16-gradient variant too, against the oracle fed the same bf16 bits; against
the oracle fed the fp32 gradients before rounding, the difference is checked
against the bound the bf16 rounding of each push implies.
"""
import dataclasses
import os
import sys

import numpy as np
import pytest

from oracle import server as orc
from paper_1611_06213_amd import ps
from paper_1611_06213_amd import workloads as wl
from tests import golden_script, parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    ps.load_library()
    return torch


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def free(torch):
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# ---------------------------------------------------------------- workloads

SMALL_N = 3 * 65536 + 7   # several 256-lane tiles and a ragged tail


@pytest.mark.parametrize("fused,fusion", [(False, None), (True, None), (True, 0), (True, 64)],
                         ids=["separate", "fused", "fused-never-one-pass", "fused-one-pass"])
@pytest.mark.parametrize("name", list(wl.CONFIGS))
def test_workload_small_full_oracle(torch, name, fused, fusion):
    """Each workload's whole schedule at a reduced parameter count; the
    oracle covers every coordinate. "fused" takes ps_apply_pull's per-call
    choice (replicas from the apply pass for one, or up to 4 with at most 16
    gradients; else the tiled fan-out after it); "fused-never-one-pass"
    always the fan-out; "fused-one-pass" every replica from the apply pass."""
    cfg = wl.CONFIGS[name].scaled(SMALL_N, pool=min(wl.CONFIGS[name].pool, 64))
    say(f"[small] {name} n={cfg.n} fused={fused} fusion={fusion}")
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = [(0, cfg.n)]
    g = parity.gpu_replay(cfg, ev, pool, w0, ranges, fused=fused, fusion=fusion)
    ps_, w0s = parity.host_inputs(cfg, pool, w0, ranges)
    o = parity.oracle_replay(cfg, ev, ps_, w0s, ranges)
    assert parity.compare(g, o, ranges) == []
    del pool
    free(torch)


def test_mixed_variable_k_drain_each_burst(torch):
    """Mixed workload, parity variant: apply at every burst end (K from 1
    to 32 varies apply to apply)."""
    cfg = dataclasses.replace(wl.CONFIGS["mixed"].scaled(SMALL_N), drain_each_burst=True)
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = [(0, cfg.n)]
    for fused in (False, True):
        g = parity.gpu_replay(cfg, ev, pool, w0, ranges, fused=fused)
        ps_, w0s = parity.host_inputs(cfg, pool, w0, ranges)
        o = parity.oracle_replay(cfg, ev, ps_, w0s, ranges)
        assert parity.compare(g, o, ranges) == []
    free(torch)


def _full_ranges(cfg):
    r = wl.sample_ranges(cfg.n, 4096, 6, seed=cfg.index)
    for name, off, numel in wl.tensor_offsets(cfg)[-4:]:
        lo = max(0, off - 2048)
        r.append((lo, min(cfg.n, lo + 4096)))
    return r


@pytest.mark.parametrize("fused,fusion", [(True, None), (False, None), (True, 64)],
                         ids=["fused", "separate", "fused-one-pass"])
@pytest.mark.parametrize("name", list(wl.CONFIGS))
def test_workload_full_size_sampled(torch, name, fused, fusion):
    """Each workload at its full size, in the launch configuration the
    benchmark uses; the oracle checks sampled coordinate ranges (head, tail
    with the ragged end, seeded interior blocks, tensor boundaries) of the
    weights, velocity and every replica after every pull event."""
    cfg = wl.CONFIGS[name]
    say(f"[full] {name} n={cfg.n} fused={fused} fusion={fusion}")
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = _full_ranges(cfg)
    g = parity.gpu_replay(cfg, ev, pool, w0, ranges, fused=fused, fusion=fusion)
    ps_, w0s = parity.host_inputs(cfg, pool, w0, ranges)
    del pool
    free(torch)
    o = parity.oracle_replay(cfg, ev, ps_, w0s, ranges)
    assert parity.compare(g, o, ranges) == []


@pytest.mark.parametrize("layout", ["server", "torch"])
def test_vgg16_full_size_bench_layouts(torch, layout):
    """VGG-16 at full size with the gradient pool and replicas laid out as
    bench.py lays them out: server rows (ps_alloc_rows; one front), or one
    torch allocation per buffer (--layout torch; four fronts chosen). Sampled
    ranges against the oracle, as above."""
    cfg = wl.CONFIGS["vgg16"]
    say(f"[full] vgg16 layout={layout}")
    ev = wl.schedule(cfg)
    rdt = torch.float32
    holder = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum)
    if layout == "server":
        pool = holder.alloc_rows(cfg.pool)
        reps = holder.alloc_rows(cfg.replicas, rdt)
    else:
        pool = [torch.empty(cfg.n, device="cuda") for _ in range(cfg.pool)]
        reps = [torch.empty(cfg.n, dtype=rdt, device="cuda") for _ in range(cfg.replicas)]
    for j in range(cfg.pool):
        pool[j].copy_(wl.make_grad(cfg, j, "cuda"))
    w0 = wl.make_w0(cfg, "cuda")
    ranges = _full_ranges(cfg)
    g = parity.gpu_replay(cfg, ev, pool, w0, ranges, replicas=reps)
    ps_, w0s = parity.host_inputs(cfg, pool, w0, ranges)
    del pool, reps
    holder.close()
    free(torch)
    o = parity.oracle_replay(cfg, ev, ps_, w0s, ranges)
    assert parity.compare(g, o, ranges) == []


def test_vgg16_full_size_round_robin_sampled(torch):
    """VGG-16 at full size with per-learner queues served round-robin, as
    bench.py --queue rr runs it (K slots per learner, applies of K gradients
    in service order): sampled ranges of w, v and every replica, the
    staleness of every applied gradient and the counters against the
    oracle in the same mode."""
    cfg = wl.CONFIGS["vgg16"]
    say("[full] vgg16 round-robin")
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = _full_ranges(cfg)
    g = parity.gpu_replay(cfg, ev, pool, w0, ranges, round_robin=True)
    ps_, w0s = parity.host_inputs(cfg, pool, w0, ranges)
    del pool
    free(torch)
    o = parity.oracle_replay(cfg, ev, ps_, w0s, ranges, round_robin=True)
    assert parity.compare(g, o, ranges) == []
    # the service order differs from FIFO: the same gradients folded in
    # another order round differently (every learner pulls after every apply,
    # so the staleness sequence is the same in both modes)
    fifo = parity.oracle_replay(cfg, ev, ps_, w0s, ranges[:1])
    assert not parity.bitwise(fifo["w"][0], o["w"][0])


def test_mixed_bf16_quantisation_bound_vs_fp32_gradients(torch):
    """The bf16-gradient run against the oracle fed the original fp32
    gradients x (before rounding to bf16). Push k changes the gradient by
    e_k = widen(bf16(x_k)) - x_k, exactly computable per coordinate; the
    heavy-ball recurrence (v_k = m v_(k-1) + g_k, w_k = w_(k-1) - lr v_k) is
    linear in the gradients, so in exact arithmetic the two runs differ by
    dw = -lr * sum_k e_k * (1 - m^(T-k+1)) / (1 - m). Checked per coordinate
    on the sampled ranges: |w_bf16 - w_f32 - dw| within the binary32 rounding
    of both runs (8*T*2^-24*(max|w| + 1e-3)), which is far below the
    quantisation effect itself, and |w_bf16 - w_f32| within the triangle
    bound lr/(1-m) * sum_k |e_k| plus that rounding. The R12 relative error
    is printed for the record."""
    cfg = wl.CONFIGS["mixed"]
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = _full_ranges(cfg)
    g = parity.gpu_replay(cfg, ev, pool, w0, ranges, fused=True)
    bf_slices = [[parity.np_bits(pool[b][lo:hi]) for b in range(cfg.pool)] for lo, hi in ranges]
    del pool
    f32_slices = [[None] * cfg.pool for _ in ranges]
    for b in range(cfg.pool):
        x = wl.make_grad_f32(cfg, b, "cuda")
        for r, (lo, hi) in enumerate(ranges):
            f32_slices[r][b] = parity.np_bits(x[lo:hi])
        del x
    w0s = [parity.np_bits(w0[lo:hi]) for lo, hi in ranges]
    free(torch)
    o = parity.oracle_replay(cfg, ev, f32_slices, w0s, ranges)
    pushes = [e.buf for e in ev if isinstance(e, wl.Push)]
    T = len(pushes)
    lr, m = float(np.float32(cfg.lr)), float(np.float32(cfg.momentum))
    coef = [(1 - m ** (T - k)) / (1 - m) for k in range(T)]     # push k (0-based) of T
    tau = float(np.sqrt(np.mean(np.concatenate(w0s).astype(np.float64) ** 2)))
    worst_rel, worst_frac, worst_signed = 0.0, 0.0, 0.0
    for r in range(len(ranges)):
        err_sum = np.zeros(ranges[r][1] - ranges[r][0])
        pred = np.zeros(ranges[r][1] - ranges[r][0])
        for k, b in enumerate(pushes):
            e = orc.bf16_to_f32(bf_slices[r][b]).astype(np.float64) - f32_slices[r][b]
            err_sum += np.abs(e)
            pred -= lr * coef[k] * e
        a = g["w"][r].astype(np.float64)
        ref = o["w"][r].astype(np.float64)
        rounding = 8 * T * 2.0 ** -24 * (np.abs(ref).max() + 1e-3)
        bound = lr / (1 - m) * err_sum + rounding
        diff = np.abs(a - ref)
        assert np.all(diff <= bound), (ranges[r], float((diff / bound).max()))
        signed = np.abs(a - ref - pred)
        assert np.all(signed <= rounding), (ranges[r], float(signed.max()), rounding)
        worst_frac = max(worst_frac, float((diff / bound).max()))
        worst_signed = max(worst_signed, float(signed.max() / rounding))
        worst_rel = max(worst_rel, float((diff / np.maximum(np.abs(ref), tau)).max()))
    say(f"[bf16 vs fp32 gradients] R12 relative error {worst_rel:.3e}; largest fraction of the "
        f"triangle bound used {worst_frac:.3f}; of the rounding bound after removing the "
        f"predicted quantisation effect {worst_signed:.3f}")


# ---------------------------------------------------------------- edges

def _run_edge(torch, n, k, momentum, gdt, pdt, offset_g=0, offset_d=0, seed=0, lr=0.01, fusion=None):
    """Push k gradients (optionally at element offsets that break vector
    alignment), apply+pull into two replicas, pull into a third, compare."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1000 + seed)
    gtd = torch.bfloat16 if gdt == ps.PS_BF16 else torch.float32
    ptd = torch.bfloat16 if pdt == ps.PS_BF16 else torch.float32
    w0 = ((torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1).contiguous()
    big = (torch.randn(k, n + 8, generator=gen, device="cuda") * 1e-2).to(gtd)
    grads = [big[j, offset_g:offset_g + n] for j in range(k)]
    dbig = torch.zeros(3, n + 8, dtype=ptd, device="cuda")
    dsts = [dbig[r, offset_d:offset_d + n] for r in range(3)]
    srv = ps.ParameterServer(n, lr, momentum, queue_depth=max(k, 1))
    if fusion is not None:
        srv.set_pull_fusion(fusion)
    srv.set_weights(w0)
    for j, gj in enumerate(grads):
        assert srv.push(j % 5, gj)
    srv.apply_pull([0, 1], dsts[:2])
    srv.pull(2, dsts[2])
    w = parity.np_bits(srv.weights_copy())
    v = srv.velocity_copy()
    reps = [parity.np_bits(d) for d in dsts]
    st = srv.last_staleness()
    srv.close()
    o = orc.OracleServer(parity.np_bits(w0), lr, momentum, depth=max(k, 1))
    for j, gj in enumerate(grads):
        o.push(j % 5, parity.np_bits(gj))
    o.apply_pending()
    for l in range(3):
        o.pull(l, l, pdt)
    assert parity.bitwise(w, o.w), (n, k, momentum, gdt, pdt, offset_g, offset_d)
    if momentum:
        assert parity.bitwise(parity.np_bits(v), o.v)
    for r in range(3):
        assert parity.bitwise(reps[r], o.replicas[r]), r
    assert st == o.staleness


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 8, 9, 63, 64, 65, 255, 256, 257, 4095, 4097,
                               4 * 256 * 7 + 3])
def test_edge_sizes(torch, n):
    for k in (1, 9):
        for momentum in (0.0, 0.9):
            for gdt, pdt in ((ps.PS_F32, ps.PS_F32), (ps.PS_BF16, ps.PS_BF16), (ps.PS_F32, ps.PS_BF16)):
                for fusion in (None, 2):
                    _run_edge(torch, n, k, momentum, gdt, pdt, seed=n, fusion=fusion)


@pytest.mark.parametrize("k", list(range(1, 18)) + [23, 31, 32, 33, 40, 47, 48, 63, 64])
def test_edge_queue_depths(torch, k):
    _run_edge(torch, 10007, k, 0.9, ps.PS_F32, ps.PS_F32, seed=k)
    _run_edge(torch, 10007, k, 0.0, ps.PS_F32, ps.PS_F32, seed=k + 100)
    _run_edge(torch, 10007, k, 0.0, ps.PS_BF16, ps.PS_BF16, seed=k, fusion=2)


@pytest.mark.parametrize("og,od", [(1, 0), (0, 1), (2, 3), (4, 4), (3, 0)])
def test_misaligned_buffers_scalar_path(torch, og, od):
    """Element offsets that break 16-byte (fp32) or 8-byte (bf16) alignment
    take the scalar kernels and must give the same bits."""
    for gdt, pdt in ((ps.PS_F32, ps.PS_F32), (ps.PS_BF16, ps.PS_BF16)):
        for momentum in (0.0, 0.9):
            for fusion in (None, 2):
                _run_edge(torch, 20011, 5, momentum, gdt, pdt, offset_g=og, offset_d=od,
                          seed=og * 7 + od, fusion=fusion)


@pytest.mark.parametrize("r", [2, 3, 16, 64])
def test_tiled_pull_many_tiles_ragged(torch, r):
    """The sliced fan-out over four full tiles (2 Mi coordinates each), a
    partial tile and a ragged tail: every replica equals w (fp32) or RNE(w)
    (bf16)."""
    n = 2 * (4 << 20) + 1234567 + 3
    gen = torch.Generator(device="cuda")
    gen.manual_seed(r)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=1)
    srv.set_weights(w0)
    w_host = parity.np_bits(w0)
    for dt, tdt in ((ps.PS_F32, torch.float32), (ps.PS_BF16, torch.bfloat16)):
        reps = wl.Rows(r, n, tdt, "cuda")
        reps.buf.fill_(7.0)
        srv.pull_many(list(range(r)), reps.rows)
        srv.sync()
        want = w_host if dt == ps.PS_F32 else orc.f32_to_bf16(w_host)
        for j in range(r):
            assert parity.bitwise(parity.np_bits(reps[j]), want), (dt, j)
        del reps
    srv.close()


@pytest.mark.parametrize("n,r", [
    (7 * (2 << 20) - 3, 2),      # 7 slice tiles, the last short
    (7 * (2 << 20) + 5, 5),      # 8 slice tiles, the last of one chunk plus a 1-value tail
    (9 * (2 << 20) + 4097 * 4 + 2, 3),   # 10 slice tiles, the last short
])
def test_pull_paths_every_element(torch, n, r):
    """The sliced 3-D fan-out writes every element of every replica exactly
    as w (fp32) or RNE(w) (bf16): replicas start as a NaN sentinel and are
    compared whole, bitwise, against the oracle's copy."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(n % 1000 + r)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=1)
    srv.set_weights(w0)
    w_host = parity.np_bits(w0)
    for dt, tdt in ((ps.PS_F32, torch.float32), (ps.PS_BF16, torch.bfloat16)):
        reps = [torch.full((n,), float("nan"), dtype=tdt, device="cuda") for _ in range(r)]
        srv.pull_many(list(range(r)), reps)
        srv.sync()
        want = w_host if dt == ps.PS_F32 else orc.f32_to_bf16(w_host)
        for j in range(r):
            assert parity.bitwise(parity.np_bits(reps[j]), want), (n, r, dt, j)
        del reps
    srv.close()


@pytest.mark.parametrize("n,r", [
    (8 * (4 << 20) + 5, 5),              # 8 full tiles, a tile of one chunk, a 1-value tail
    (9 * (4 << 20) + 4097 * 4 + 2, 3),   # 10 tiles, the last short
])
def test_one_d_tiled_pull_every_element(torch, n, r):
    """The 1-D tiled fan-out (fp32 replicas of 8 or more 4 Mi tiles): every
    element of every replica, NaN sentinels first, equals w bit for bit (an
    fp32 pull is a copy), compared on the device; bf16 replicas of the same
    vector (sliced fan-out) equal RNE(w) from the oracle."""
    say(f"[case] 1-D tiled pull n={n} R={r}")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(53 + r)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=1)
    srv.set_weights(w0)
    w_host = parity.np_bits(w0)
    for dt, tdt in ((ps.PS_F32, torch.float32), (ps.PS_BF16, torch.bfloat16)):
        want = w_host if dt == ps.PS_F32 else orc.f32_to_bf16(w_host)
        want = torch.from_numpy(want.view(np.int32 if dt == ps.PS_F32 else np.int16)).to("cuda")
        reps = [torch.full((n,), float("nan"), dtype=tdt, device="cuda") for _ in range(r)]
        srv.pull_many(list(range(r)), reps)
        srv.sync()
        for j in range(r):
            assert torch.equal(reps[j].view(torch.int32 if dt == ps.PS_F32 else torch.int16), want), (dt, j)
        del reps, want
    srv.close()
    free(torch)


@pytest.mark.parametrize("n", [5, 4096 * 256 + 3, 10_000_019])
def test_single_replica_pull_every_element(torch, n):
    """One replica per call takes the streaming copy (pull_vec) for both
    replica dtypes: every element equals w (fp32) or RNE(w) (bf16), tail
    included, against the oracle's copy."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(n % 997)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=1)
    srv.set_weights(w0)
    w_host = parity.np_bits(w0)
    for tdt, want in ((torch.float32, w_host), (torch.bfloat16, orc.f32_to_bf16(w_host))):
        dst = torch.full((n,), float("nan"), dtype=tdt, device="cuda")
        srv.pull_many([0], [dst])
        srv.sync()
        assert parity.bitwise(parity.np_bits(dst), want), (n, tdt)
    srv.close()


def _f32_rounding_probes(n_random, seed, nan=True):
    """fp32 bit patterns that probe rounding to bf16: ties that stay and ties
    that carry, just below and above one half, carries into the exponent and
    to infinity, subnormals, signed zeros, infinities and (with nan) NaNs of
    both kinds and signs; then random patterns over the whole 32-bit range."""
    hand = [0x00000000, 0x80000000, 0x00000001, 0x80000001, 0x00007FFF, 0x00008000,
            0x00008001, 0x00018000, 0x0000FFFF, 0x007F8000, 0x007FFFFF, 0x80FF8000,
            0x00800000, 0x3F808000, 0x3F818000, 0x3F807FFF, 0x3F808001, 0xBF818000,
            0x3FFF8000, 0x7F7F7FFF, 0x7F7F8000, 0x7F7EFFFF, 0x7F7FFFFF, 0xFF7FFFFF,
            0x7F800000, 0xFF800000]
    nans = [0x7F800001, 0x7F80FFFF, 0x7FBFFFFF, 0x7FC00000, 0x7FFFFFFF, 0xFFC00001,
            0xFF800001, 0xFFFFFFFF]
    bits = np.array(hand + (nans if nan else []), dtype=np.uint32)
    rnd = np.random.default_rng(seed).integers(0, 1 << 32, size=n_random, dtype=np.uint64)
    rnd = rnd.astype(np.uint32)
    if not nan:
        rnd = rnd[(rnd & 0x7FFFFFFF) <= 0x7F800000]
    return np.concatenate([bits, rnd])


def _device_f32(torch, bits):
    return torch.from_numpy(bits.view(np.int32).copy()).to("cuda").view(torch.float32)


@pytest.mark.parametrize("r,offset", [(1, 0), (3, 0), (3, 4), (3, 1), (1, 1)],
                         ids=["vec", "slices-8", "slices-4", "scalar", "vec-scalar"])
def test_bf16_replica_rounding_special_values(torch, r, offset):
    """Every pull kernel rounds to bf16 as the oracle does: one replica (the
    streaming copy), several (the sliced fan-out, 8 values per lane, or 4 for
    8-byte-aligned replicas) and replicas at an odd element offset (scalar),
    over ties, carries, subnormals, infinities, NaN payloads and random bit
    patterns. fp32 replicas carry w's bits unchanged, NaN payloads included."""
    bits = _f32_rounding_probes(70_000, seed=10 * r + offset)
    n = bits.size
    say(f"[bf16 specials] r={r} offset={offset} n={n}")
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=1)
    srv.set_weights(_device_f32(torch, bits))
    want = orc.f32_to_bf16(bits.view(np.float32))
    bufs = [torch.full((n + 8,), float("nan"), dtype=torch.bfloat16, device="cuda")
            for _ in range(r)]
    dsts = [b[offset:offset + n] for b in bufs]
    srv.pull_many(list(range(r)), dsts)
    f = torch.full((n + 8,), 7.0, device="cuda")
    srv.pull_many([r], [f[offset:offset + n]])
    srv.sync()
    for j in range(r):
        assert parity.bitwise(parity.np_bits(dsts[j]), want), (r, offset, j)
    assert parity.bitwise(parity.np_bits(f[offset:offset + n]), bits.view(np.float32))
    srv.close()


@pytest.mark.parametrize("gdt", [ps.PS_F32, ps.PS_BF16], ids=["f32-grad", "bf16-grad"])
@pytest.mark.parametrize("offset", [0, 4, 1])
def test_bf16_replicas_from_the_apply_special_values(torch, gdt, offset):
    """Replicas written by the apply pass itself (fusion) round as the oracle
    does, for every apply kernel (8 or 4 values per lane, scalar). w holds the
    probe patterns without NaN (NaN arithmetic is not bit-specified); zero
    gradients leave every finite w and infinity in place up to the sign of
    zero, the same on both sides."""
    bits = _f32_rounding_probes(50_000, seed=100 + offset + gdt, nan=False)
    n = bits.size
    say(f"[bf16 specials fused] gdt={gdt} offset={offset} n={n}")
    gtd = torch.bfloat16 if gdt == ps.PS_BF16 else torch.float32
    g = torch.zeros(n, dtype=gtd, device="cuda")
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=1)
    srv.set_pull_fusion(2)
    srv.set_weights(_device_f32(torch, bits))
    bufs = [torch.full((n + 8,), float("nan"), dtype=torch.bfloat16, device="cuda")
            for _ in range(2)]
    dsts = [b[offset:offset + n] for b in bufs]
    assert srv.push(0, g)
    srv.apply_pull([0, 1], dsts)
    srv.sync()
    o = orc.OracleServer(bits.view(np.float32).copy(), 0.01, 0.0, depth=1)
    o.push(0, parity.np_bits(g))
    o.apply_pending()
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w)
    for j in range(2):
        o.pull(j, j, orc.BF16)
        assert parity.bitwise(parity.np_bits(dsts[j]), o.replicas[j]), (gdt, offset, j)
    srv.close()


def test_bf16_rounding_exhaustive(torch):
    """All 2^32 fp32 bit patterns, in 16 chunks of 2^28, pulled into two bf16
    replicas (the sliced fan-out, 8 values per lane) and one more (the
    streaming copy): every replica equals the oracle's rounding, bit for
    bit."""
    chunk = 1 << 28
    srv = ps.ParameterServer(chunk, 0.01, 0.0, queue_depth=1)
    reps = [torch.empty(chunk, dtype=torch.bfloat16, device="cuda") for _ in range(3)]
    base = np.arange(chunk, dtype=np.uint32)
    for c in range(16):
        say(f"[bf16 exhaustive] chunk {c}")
        bits = base + np.uint32(c << 28)
        srv.set_weights(_device_f32(torch, bits))
        for t in reps:
            t.fill_(float("nan"))
        srv.pull_many([0, 1], reps[:2])
        srv.pull_many([2], reps[2:])
        srv.sync()
        want = orc.f32_to_bf16(bits.view(np.float32))
        for j, t in enumerate(reps):
            assert parity.bitwise(parity.np_bits(t), want), (c, j)
    del reps
    srv.close()
    free(torch)


def test_two_servers_on_their_own_streams(torch):
    """Two handles in one process, each on its own stream (different sizes,
    momentum, gradient and replica dtypes), with their calls interleaved:
    each matches its own oracle bitwise, so nothing is shared between
    handles."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(77)
    specs = [(70_001, 0.01, 0.9, torch.float32, ps.PS_F32), (123_457, 0.005, 0.0, torch.bfloat16, ps.PS_BF16)]
    servers, oracles, grads, reps = [], [], [], []
    for n, lr, m, gdt, pdt in specs:
        w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
        grads.append([(torch.randn(n, generator=gen, device="cuda") * 1e-2).to(gdt) for _ in range(5)])
        reps.append([torch.full((n,), float("nan"), device="cuda",
                                dtype=torch.bfloat16 if pdt == ps.PS_BF16 else torch.float32)
                     for _ in range(2)])
        torch.cuda.synchronize()
        srv = ps.ParameterServer(n, lr, m, queue_depth=4, stream=torch.cuda.Stream())
        srv.set_weights(w0)
        servers.append(srv)
        oracles.append(orc.OracleServer(parity.np_bits(w0), lr, m, depth=4))
    host = [[parity.np_bits(g) for g in gs] for gs in grads]
    for step in range(6):
        for j, (srv, o) in enumerate(zip(servers, oracles)):
            for q in range(3 - j):
                b = (step + q) % 5
                assert srv.push(q, grads[j][b])
                o.push(q, host[j][b])
        for j, (srv, o) in enumerate(zip(servers, oracles)):
            pdt = specs[j][4]
            if (step + j) % 2:
                srv.apply_pull([0, 1], reps[j])
                o.apply_pending()
            else:
                srv.apply_pending()
                srv.pull_many([0, 1], reps[j])
                o.apply_pending()
            for l in range(2):
                o.pull(l, l, pdt)
    for j, (srv, o) in enumerate(zip(servers, oracles)):
        srv.sync()
        assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w), j
        if specs[j][2]:
            assert parity.bitwise(parity.np_bits(srv.velocity_copy()), o.v), j
        for l in range(2):
            assert parity.bitwise(parity.np_bits(reps[j][l]), o.replicas[l]), (j, l)
        assert srv.timestamp == o.ts
        srv.close()


def test_lr_zero_and_zero_gradient(torch):
    n = 5000
    w0 = torch.linspace(-0.05, 0.05, n, device="cuda")
    w0[:2] = torch.tensor([0.0, -0.0])
    for lr, scale in ((0.0, 1.0), (0.01, 0.0)):
        srv = ps.ParameterServer(n, lr, 0.9, queue_depth=4)
        srv.set_weights(w0)
        g = torch.randn(n, device="cuda") * scale
        for _ in range(4):
            srv.push(0, g)
        srv.apply_pending()
        w = srv.weights_copy()
        o = orc.OracleServer(parity.np_bits(w0), lr, 0.9, depth=4)
        for _ in range(4):
            o.push(0, parity.np_bits(g))
        o.apply_pending()
        assert parity.bitwise(parity.np_bits(w), o.w)
        if scale == 0.0:
            assert parity.bitwise(parity.np_bits(w), parity.np_bits(w0))
        srv.close()


def test_mixed_dtype_queue(torch):
    """fp32 and bf16 gradients in one queue: applied as runs, in push order."""
    n = 30001
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    gs = [torch.randn(n, generator=gen, device="cuda") * 1e-2 for _ in range(7)]
    gs = [g.to(torch.bfloat16) if j in (1, 2, 5) else g for j, g in enumerate(gs)]
    for m in (0.0, 0.9):
        srv = ps.ParameterServer(n, 0.01, m, queue_depth=8)
        srv.set_weights(w0)
        dst = torch.empty(n, device="cuda")
        for j, g in enumerate(gs):
            srv.push(j, g)
        srv.apply_pull([0], [dst])
        o = orc.OracleServer(parity.np_bits(w0), 0.01, m, depth=8)
        for j, g in enumerate(gs):
            o.push(j, parity.np_bits(g))
        o.apply_pending()
        assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w)
        assert parity.bitwise(parity.np_bits(dst), o.w)
        assert srv.timestamp == 7
        srv.close()


def test_golden_staleness_script_through_abi(torch):
    """The hand-worked schedule of tests/golden/staleness_k2.txt, through the
    C ABI (timestamps, staleness, queue bound, pull skip)."""
    depth, ops, expect = golden_script.load("staleness_k2.txt")
    n = 4
    g = torch.full((n,), 0.5, device="cuda")
    dsts = {l: torch.empty(n, device="cuda") for l in range(3)}
    srv = ps.ParameterServer(n, 2.0 ** -4, 0.0, queue_depth=depth)
    srv.set_weights(torch.zeros(n, device="cuda"))
    stale = []
    for op, l, outcome in ops:
        if op == "push":
            assert srv.push(l, g) == (outcome == "ok")
        elif op == "apply":
            srv.apply_pending()
            stale += srv.last_staleness()
        else:
            before = srv.stats().pulls_skipped
            srv.pull(l, dsts[l])
            assert (srv.stats().pulls_skipped == before) == (outcome == "pulled")
        assert 0 <= srv.pending <= depth
    st = srv.stats()
    assert stale == expect["staleness"]
    assert srv.timestamp == expect["ts"][0]
    assert (st.pulls, st.pulls_skipped, st.pushes_rejected) == (
        expect["pulls"], expect["skipped"], expect["rejected"])
    assert st.staleness_max == 4 and st.staleness_sum == sum(expect["staleness"])
    assert torch.all(srv.weights_copy() == -7 / 32)
    srv.close()


def test_queue_full_and_errors(torch):
    n = 1000
    srv = ps.ParameterServer(n, 0.1, 0.0, queue_depth=3)
    g = torch.ones(n, device="cuda")
    assert all(srv.push(0, g) for _ in range(3))
    assert not srv.push(1, g) and srv.pending == 3          # refused, unchanged
    assert ps.ps_set_queue_depth(srv.h, 2) == ps.PS_ESTATE
    assert ps.ps_set_queue_depth(srv.h, 65) == ps.PS_EINVAL
    assert ps.ps_set_weights(srv.h, g.data_ptr()) == ps.PS_ESTATE
    assert ps.ps_push(srv.h, -1, g.data_ptr()) == ps.PS_EINVAL
    assert ps.ps_push(srv.h, ps.PS_MAX_LEARNERS, g.data_ptr()) == ps.PS_EINVAL
    assert ps.ps_push_dtype(srv.h, 0, g.data_ptr(), 7) == ps.PS_EINVAL
    d = torch.empty(n, device="cuda")
    assert ps.ps_pull_many(srv.h, [0, 1], [d.data_ptr(), d.data_ptr()], ps.PS_F32) == ps.PS_EINVAL
    assert ps.ps_pull_many(srv.h, [0] * 65, [d.data_ptr()] * 65, ps.PS_F32) == ps.PS_EINVAL
    srv.apply_pending()
    assert srv.timestamp == 3 and srv.pending == 0
    srv.apply_pending()                                       # empty: no-op
    assert srv.timestamp == 3
    st = srv.stats()
    assert (st.pushes_accepted, st.pushes_rejected, st.pushes_applied, st.applies) == (3, 1, 3, 1)
    srv.close()


def test_pull_skip_on_off_same_bits(torch):
    cfg = wl.CONFIGS["alexnet"].scaled(20000, pushes=200, pool=16)
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = [(0, cfg.n)]
    a = parity.gpu_replay(cfg, ev, pool, w0, ranges, pull_skip=True)
    b = parity.gpu_replay(cfg, ev, pool, w0, ranges, pull_skip=False)
    assert a["counts"][3] > 0 and b["counts"][3] == 0
    for x, y in zip(a["snaps"], b["snaps"]):
        for l in x:
            assert parity.bitwise(x[l][0], y[l][0])
    assert parity.bitwise(a["w"][0], b["w"][0])
    ps_, w0s = parity.host_inputs(cfg, pool, w0, ranges)
    o = parity.oracle_replay(cfg, ev, ps_, w0s, ranges, pull_skip=False)
    assert parity.compare(b, o, ranges) == []


def test_determinism_and_side_stream(torch):
    """Two runs are bitwise identical, also on a non-default stream."""
    cfg = wl.CONFIGS["vgg16"].scaled(100003, pushes=96, pool=40)
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = [(0, cfg.n)]
    a = parity.gpu_replay(cfg, ev, pool, w0, ranges, fused=True)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        b = parity.gpu_replay(cfg, ev, pool, w0, ranges, fused=True, stream=s)
    assert parity.bitwise(a["w"][0], b["w"][0]) and parity.bitwise(a["v"][0], b["v"][0])


def test_64bit_indexing_beyond_2_31_elements(torch):
    """n = 2^31 + 5 fp32 weights: element offsets past 2^31 (byte offsets past
    2^33) are indexed correctly; sampled against the oracle."""
    n = 2 ** 31 + 5
    k = 2
    gen = torch.Generator(device="cuda")
    gen.manual_seed(77)
    w0 = torch.empty(n, device="cuda").uniform_(-0.05, 0.05, generator=gen)
    grads = [torch.empty(n, device="cuda").normal_(0, 1e-2, generator=gen) for _ in range(k)]
    dst = torch.empty(n, device="cuda")
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=k)
    srv.set_weights(w0)
    for j, g in enumerate(grads):
        srv.push(j, g)
    srv.apply_pull([0], [dst])
    srv.sync()
    ranges = [(0, 1024), (2 ** 31 - 512, 2 ** 31 + 512), (n - 1029, n)]
    w = srv.weights_copy()
    for lo, hi in ranges:
        o = orc.OracleServer(parity.np_bits(w0[lo:hi]), 0.01, 0.9, depth=k)
        for j, g in enumerate(grads):
            o.push(j, parity.np_bits(g[lo:hi]))
        o.apply_pending()
        assert parity.bitwise(parity.np_bits(w[lo:hi]), o.w)
        assert parity.bitwise(parity.np_bits(dst[lo:hi]), o.w)
    srv.close()
    del w0, grads, dst, w
    free(torch)


# ---------------------------------------------------------------- SSGD

def _run_sync(torch, n, lam, steps, momentum, gdt, offset=0, seed=0, lr=0.01):
    """`steps` synchronous steps of `lam` learners (one gradient each), with a
    pull of every learner after each step, against the oracle."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3000 + seed)
    gtd = torch.bfloat16 if gdt == ps.PS_BF16 else torch.float32
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    big = (torch.randn(lam * steps, n + 8, generator=gen, device="cuda") * 1e-2).to(gtd)
    grads = [big[j, offset:offset + n] for j in range(lam * steps)]
    dst = torch.empty(n, device="cuda")
    srv = ps.ParameterServer(n, lr, momentum, queue_depth=lam)
    srv.set_weights(w0)
    o = orc.OracleServer(parity.np_bits(w0), lr, momentum, depth=lam)
    stale = []
    for s in range(steps):
        for l in range(lam):
            g = grads[s * lam + l]
            assert srv.push(l, g)
            assert o.push(l, parity.np_bits(g)) == orc.OK
        srv.apply_sync()
        stale += srv.last_staleness()
        assert o.apply_sync() == orc.OK
        for l in range(lam):
            srv.pull(l, dst)
            o.pull(l, "d", orc.F32)
    w = parity.np_bits(srv.weights_copy())
    assert parity.bitwise(w, o.w), (n, lam, momentum, gdt, offset)
    if momentum:
        assert parity.bitwise(parity.np_bits(srv.velocity_copy()), o.v)
    assert parity.bitwise(parity.np_bits(dst), o.w)
    assert srv.timestamp == o.ts == steps and stale == o.staleness
    srv.close()


@pytest.mark.parametrize("lam", [1, 2, 3, 7, 8, 9, 15, 16, 17, 24, 31, 32, 33, 64])
def test_sync_parity(torch, lam):
    for momentum in (0.0, 0.9):
        for gdt in (ps.PS_F32, ps.PS_BF16):
            _run_sync(torch, 30011, lam, 3, momentum, gdt, seed=lam)


@pytest.mark.parametrize("n", [1, 5, 8, 9, 4097, 2 * 1024 * 1024 + 3])
def test_sync_sizes_and_alignment(torch, n):
    for offset in (0, 1, 4):
        for gdt in (ps.PS_F32, ps.PS_BF16):
            _run_sync(torch, n, 16, 2, 0.9, gdt, offset=offset, seed=n + offset)


def test_sync_rejects_mixed_dtypes(torch):
    n = 1000
    srv = ps.ParameterServer(n, 0.1, 0.0, queue_depth=4)
    srv.push(0, torch.ones(n, device="cuda"))
    srv.push(1, torch.ones(n, dtype=torch.bfloat16, device="cuda"))
    assert ps.ps_apply_sync(srv.h) == ps.PS_EINVAL
    assert srv.pending == 2 and srv.timestamp == 0
    srv.apply_pending()
    assert srv.timestamp == 2
    srv.close()


def test_sync_vgg16_shaped_full_size_sampled(torch):
    """VGG-16 shape (138,357,544 parameters), 16 learners pushing one gradient
    each per synchronous step, 6 steps, all pulling after each step; sampled
    against the oracle."""
    cfg = wl.CONFIGS["vgg16"]
    pool = wl.make_pool(dataclasses.replace(cfg, pool=32), "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = _full_ranges(cfg)
    srv = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=16)
    srv.set_weights(w0)
    reps = wl.Rows(16, cfg.n, torch.float32, "cuda")
    steps = 6
    for s in range(steps):
        for l in range(16):
            srv.push(l, pool[(s * 16 + l) % 32])
        srv.apply_sync()
        srv.pull_many(list(range(16)), reps.rows)
    w = srv.weights_copy()
    got = [parity.np_bits(w[lo:hi]) for lo, hi in ranges]
    rep = [parity.np_bits(reps[7][lo:hi]) for lo, hi in ranges]
    srv.close()
    for r, (lo, hi) in enumerate(ranges):
        o = orc.OracleServer(parity.np_bits(w0[lo:hi]), cfg.lr, cfg.momentum, depth=16)
        for s in range(steps):
            for l in range(16):
                o.push(l, parity.np_bits(pool[(s * 16 + l) % 32][lo:hi]))
            o.apply_sync()
        assert parity.bitwise(got[r], o.w) and parity.bitwise(rep[r], o.w), (lo, hi)
    del pool, reps
    free(torch)


# ---------------------------------------------------------------- round robin

def test_golden_round_robin_through_abi(torch):
    """tests/golden/round_robin_k4.txt through the C ABI: service order, per-
    learner slot limit, staleness, counters."""
    depth, ops, expect, mode = golden_script.load("round_robin_k4.txt", with_mode=True)
    n = 4
    g = torch.full((n,), 0.5, device="cuda")
    dsts = {l: torch.empty(n, device="cuda") for l in range(3)}
    srv = ps.ParameterServer(n, 2.0 ** -4, 0.0, queue_depth=depth)
    srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, mode[1])
    srv.set_weights(torch.zeros(n, device="cuda"))
    order, stale = [], []
    for op, l, outcome in ops:
        if op == "push":
            assert srv.push(l, g) == (outcome == "ok")
        elif op == "apply":
            srv.apply_pending()
            order += srv.last_applied()
            stale += srv.last_staleness()
        else:
            srv.pull(l, dsts[l])
    st = srv.stats()
    assert order == expect["order"] and stale == expect["staleness"]
    assert srv.timestamp == expect["ts"][0]
    assert (st.pulls, st.pulls_skipped, st.pushes_rejected) == (
        expect["pulls"], expect["skipped"], expect["rejected"])
    srv.close()


@pytest.mark.parametrize("slots,depth", [(1, 1), (2, 4), (3, 5), (4, 16), (8, 64)])
def test_round_robin_random_vs_oracle(torch, slots, depth):
    """Random pushes (some refused), asynchronous applies, synchronous steps
    and pulls in round-robin mode with momentum: weights, velocity, service
    order, staleness and refusals equal the oracle's, bit for bit."""
    n = 50001
    lam = 6
    rng = np.random.default_rng(slots * 100 + depth)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(slots * 100 + depth)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    pool = [torch.randn(n, generator=gen, device="cuda") * 1e-2 for _ in range(24)]
    host = [parity.np_bits(p) for p in pool]
    dst = torch.empty(n, device="cuda")
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=depth)
    srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, slots)
    srv.set_weights(w0)
    o = orc.OracleServer(parity.np_bits(w0), 0.01, 0.9, depth=depth)
    assert o.set_queue_mode(orc.ROUND_ROBIN, slots) == orc.OK
    order, stale = [], []
    for step in range(400):
        r = rng.random()
        if r < 0.6:
            l, b = int(rng.integers(0, lam)), int(rng.integers(0, len(pool)))
            ok = srv.push(l, pool[b])
            assert ok == (o.push(l, host[b]) == orc.OK)
        elif r < 0.85:
            srv.apply_pending()
            o.apply_pending()
            order += srv.last_applied()
            stale += srv.last_staleness()
        elif r < 0.9:
            srv.apply_sync()
            assert o.apply_sync() == orc.OK
            order += srv.last_applied()
            stale += srv.last_staleness()
        else:
            l = int(rng.integers(0, lam))
            srv.pull(l, dst)
            o.pull(l, "d", orc.F32)
        assert srv.pending == o.pending()
    assert order == o.applied_order and stale == o.staleness
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w)
    assert parity.bitwise(parity.np_bits(srv.velocity_copy()), o.v)
    assert srv.stats().pushes_rejected > 0 or slots >= 4
    srv.close()


def test_queue_mode_rules(torch):
    n = 100
    srv = ps.ParameterServer(n, 0.1, 0.0, queue_depth=4)
    g = torch.ones(n, device="cuda")
    assert ps.ps_set_queue_mode(srv.h, 7, 1) == ps.PS_EINVAL
    assert ps.ps_set_queue_mode(srv.h, ps.PS_QUEUE_ROUND_ROBIN, 0) == ps.PS_EINVAL
    assert ps.ps_set_queue_mode(srv.h, ps.PS_QUEUE_ROUND_ROBIN, 65) == ps.PS_EINVAL
    srv.push(0, g)
    assert ps.ps_set_queue_mode(srv.h, ps.PS_QUEUE_ROUND_ROBIN, 2) == ps.PS_ESTATE
    srv.apply_pending()
    srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, 1)
    # 65 learners waiting is more than one synchronous step can average
    for l in range(65):
        srv.push(l, g)
    assert ps.ps_apply_sync(srv.h) == ps.PS_ESTATE
    while srv.pending:
        srv.apply_pending()
    assert srv.timestamp == 66
    srv.close()


# ---------------------------------------------------------------- fault tolerance

def _ft_schedule(cfg):
    ev = wl.schedule(cfg)
    applies = [i for i, e in enumerate(ev) if isinstance(e, wl.Apply)]
    return ev, applies


def _drive(srv, ev, pool, replicas, stale, learners_dead=(), start=0, stop=None):
    for e in ev[start:stop]:
        if isinstance(e, wl.Push):
            if e.learner not in learners_dead:
                assert srv.push(e.learner, pool[e.buf])
        elif isinstance(e, wl.Apply):
            srv.apply_pending()
            stale += srv.last_staleness()
        else:
            for rnd in parity.pull_rounds(e.learners):
                srv.pull_many(rnd, [replicas[l] for l in rnd])


@pytest.mark.parametrize("mode", [ps.PS_QUEUE_FIFO, ps.PS_QUEUE_ROUND_ROBIN])
def test_checkpoint_restart_is_bitwise_uninterrupted(torch, tmp_path, mode):
    """Sec. 4.3: run half the AlexNet-shaped schedule, checkpoint, destroy the
    server, create a new one, load, run the rest: weights, velocity, replicas
    and staleness equal the uninterrupted run bit for bit."""
    cfg = wl.CONFIGS["alexnet"].scaled(300007, pushes=320, pool=24)
    ev, applies = _ft_schedule(cfg)
    cut = applies[len(applies) // 2] + 1
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")

    def fresh():
        s = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=cfg.depth)
        if mode == ps.PS_QUEUE_ROUND_ROBIN:
            s.set_queue_mode(mode, cfg.depth)
        return s

    ra = wl.Rows(cfg.replicas, cfg.n, torch.float32, "cuda")
    a = fresh()
    a.set_weights(w0)
    sa = []
    _drive(a, ev, pool, ra, sa)
    wa, va = parity.np_bits(a.weights_copy()), parity.np_bits(a.velocity_copy())
    a.close()

    rb = wl.Rows(cfg.replicas, cfg.n, torch.float32, "cuda")
    b = fresh()
    b.set_weights(w0)
    sb = []
    _drive(b, ev, pool, rb, sb, stop=cut)
    path = str(tmp_path / "ps.ckpt")
    b.save(path)
    ts_cut = b.timestamp
    b.close()
    c = fresh()
    c.load(path)
    assert c.timestamp == ts_cut
    _drive(c, ev, pool, rb, sb, start=cut)
    assert parity.bitwise(parity.np_bits(c.weights_copy()), wa)
    assert parity.bitwise(parity.np_bits(c.velocity_copy()), va)
    assert sb == sa
    for l in range(cfg.replicas):
        assert parity.bitwise(parity.np_bits(rb[l]), parity.np_bits(ra[l]))
    c.close()


def test_checkpoint_errors_leave_server_unchanged(torch, tmp_path):
    n = 100003
    gen = torch.Generator(device="cuda")
    gen.manual_seed(9)
    w0 = torch.rand(n, generator=gen, device="cuda")
    a = ps.ParameterServer(n, 0.01, 0.9)
    a.set_weights(w0)
    a.push(0, torch.ones(n, device="cuda"))
    path = str(tmp_path / "a.ckpt")
    assert ps.ps_save(a.h, path) == ps.PS_ESTATE            # gradients pending
    a.apply_pending()
    a.save(path)
    w_saved = parity.np_bits(a.weights_copy())
    b = ps.ParameterServer(n, 0.01, 0.9)
    b.set_weights(torch.zeros(n, device="cuda"))
    raw = bytearray(open(path, "rb").read())
    bad = str(tmp_path / "bad.ckpt")
    raw[200] ^= 1
    open(bad, "wb").write(bytes(raw))
    assert ps.ps_load(b.h, bad) == ps.PS_EIO and "checksum" in ps.ps_last_error()
    # the header is checksummed too: a flipped timestamp bit (bytes 32..39)
    hdr = bytearray(open(path, "rb").read())
    hdr[32] ^= 1
    open(bad, "wb").write(bytes(hdr))
    assert ps.ps_load(b.h, bad) == ps.PS_EIO and "checksum" in ps.ps_last_error()
    hdr[32] ^= 1
    hdr[8] = 1                                               # format version field
    open(bad, "wb").write(bytes(hdr))
    assert ps.ps_load(b.h, bad) == ps.PS_EIO and "version" in ps.ps_last_error()
    open(bad, "wb").write(bytes(raw[:1000]))
    assert ps.ps_load(b.h, bad) == ps.PS_EIO
    assert ps.ps_load(b.h, str(tmp_path / "missing.ckpt")) == ps.PS_EIO
    assert torch.all(b.weights_copy() == 0) and b.timestamp == 0     # unchanged
    other = ps.ParameterServer(n + 1, 0.01, 0.9)
    assert ps.ps_load(other.h, path) == ps.PS_EINVAL
    other2 = ps.ParameterServer(n, 0.02, 0.9)
    assert ps.ps_load(other2.h, path) == ps.PS_EINVAL
    nomom = ps.ParameterServer(n, 0.01, 0.0)
    assert ps.ps_load(nomom.h, path) == ps.PS_EINVAL
    b.load(path)
    assert parity.bitwise(parity.np_bits(b.weights_copy()), w_saved) and b.timestamp == 1
    for s in (a, b, other, other2, nomom):
        s.close()


@pytest.mark.parametrize("mode", [ps.PS_QUEUE_FIFO, ps.PS_QUEUE_ROUND_ROBIN])
def test_dead_learner_isolated(torch, mode):
    """Sec. 4.3 / 6.4: learner 3 dies mid-run with gradients queued; they are
    dropped and it pushes no more; the server keeps applying the others'.
    The oracle does the same; weights, staleness and order agree bitwise."""
    cfg = wl.CONFIGS["vgg16"].scaled(200003, pushes=160, pool=20)
    ev = wl.schedule(cfg)
    die_at = len(ev) // 2
    while not isinstance(ev[die_at], wl.Push):
        die_at += 1
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    host = [parity.np_bits(pool[b]) for b in range(cfg.pool)]
    srv = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=cfg.depth)
    o = orc.OracleServer(parity.np_bits(w0), cfg.lr, cfg.momentum, depth=cfg.depth)
    if mode == ps.PS_QUEUE_ROUND_ROBIN:
        srv.set_queue_mode(mode, 8)
        o.set_queue_mode(orc.ROUND_ROBIN, 8)
    srv.set_weights(w0)
    dead, stale, order, dropped = set(), [], [], 0
    reps = wl.Rows(cfg.replicas, cfg.n, torch.float32, "cuda")
    for i, e in enumerate(ev):
        if i == die_at:
            dead.add(3)
            d = srv.drop_learner(3)
            assert d == o.drop_learner(3)
            dropped += d
        if isinstance(e, wl.Push):
            if e.learner in dead:
                continue
            ok = srv.push(e.learner, pool[e.buf])
            assert ok == (o.push(e.learner, host[e.buf]) == orc.OK)
            if not ok:   # round-robin slots full: apply, then push again
                srv.apply_pending(); o.apply_pending()
                order += srv.last_applied(); stale += srv.last_staleness()
                assert srv.push(e.learner, pool[e.buf]) and o.push(e.learner, host[e.buf]) == orc.OK
        elif isinstance(e, wl.Apply):
            srv.apply_pending(); o.apply_pending()
            order += srv.last_applied(); stale += srv.last_staleness()
        else:
            live = [l for l in e.learners if l not in dead]
            srv.pull_many(live, [reps[l] for l in live])
            for l in live:
                o.pull(l, l, orc.F32)
    while srv.pending:
        srv.apply_pending(); o.apply_pending()
        order += srv.last_applied(); stale += srv.last_staleness()
    assert order == o.applied_order and stale == o.staleness
    assert 3 not in order[-20:] and srv.stats().pushes_dropped == dropped
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w)
    srv.close()


# ---------------------------------------------------------------- concurrency

def test_push_async_waits_for_producer_stream(torch):
    """A learner writes its gradient on its own stream after a few ms of other
    work; it pushes with a ready event and the apply is enqueued at once, the
    host never waiting. The apply must see the finished gradient."""
    n = 4_000_003
    gen = torch.Generator(device="cuda")
    gen.manual_seed(50)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    truth = [torch.randn(n, generator=gen, device="cuda") * 1e-2 for _ in range(3)]
    grads = [torch.full((n,), float("nan"), device="cuda") for _ in range(3)]
    busy = torch.randn(1 << 24, generator=gen, device="cuda")
    producer = torch.cuda.Stream()
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=4)
    srv.set_stream(torch.cuda.current_stream())
    srv.set_weights(w0)
    torch.cuda.synchronize()
    events = []
    with torch.cuda.stream(producer):
        for j in range(3):
            for _ in range(100):
                busy.mul_(1.0000001)      # the learner's "training" before its push
            grads[j].copy_(truth[j])
            ev = torch.cuda.Event()
            ev.record(producer)
            events.append(ev)
    for j in range(3):
        assert srv.push_async(j, grads[j], events[j])
    srv.apply_pending()
    w = parity.np_bits(srv.weights_copy())
    o = orc.OracleServer(parity.np_bits(w0), 0.01, 0.9, depth=4)
    for j in range(3):
        o.push(j, parity.np_bits(truth[j]))
    o.apply_pending()
    assert parity.bitwise(w, o.w)
    srv.close()


def test_binding_freed_gradients_not_reused_before_apply(torch):
    """The binding marks pushed gradients as used on the server's stream: a
    caller that frees its gradient tensors right after apply_pending, while
    the apply still runs on a side stream, does not get their memory back
    from torch's allocator for a new tensor (whose writes would race the
    apply). The weights then match the oracle bitwise."""
    n, k = 1 << 24, 32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(51)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    grads = [torch.randn(n, generator=gen, device="cuda") * 1e-3 for _ in range(k)]
    host = [parity.np_bits(g) for g in grads]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        torch.cuda._sleep(50_000_000)     # ~20 ms: the apply is still queued when the host allocates
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=k, stream=side)
    srv.set_weights(w0)
    for j, g in enumerate(grads):
        assert srv.push(j % 8, g)
    srv.apply_pending()
    old = {g.data_ptr() for g in grads}
    del g
    grads.clear()
    fresh = [torch.empty(n, device="cuda") for _ in range(4)]
    for t in fresh:
        t.fill_(1e30)                     # on the current stream, at once
    assert not old & {t.data_ptr() for t in fresh}
    w = parity.np_bits(srv.weights_copy())
    o = orc.OracleServer(parity.np_bits(w0), 0.01, 0.9, depth=k)
    for j in range(k):
        o.push(j % 8, host[j])
    o.apply_pending()
    assert parity.bitwise(w, o.w)
    srv.close()


def test_binding_freed_weights_source_not_reused_before_copy(torch):
    """set_weights copies on the server's stream: a caller that frees the
    source tensor at once, while the copy is still queued behind other work
    on a side stream, does not get its memory back from torch's allocator for
    a new tensor (whose writes would race the copy). w then equals the source
    bitwise."""
    n = 1 << 24
    gen = torch.Generator(device="cuda")
    gen.manual_seed(52)
    src = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    want = parity.np_bits(src)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    srv = ps.ParameterServer(n, 0.01, 0.9, stream=side)
    with torch.cuda.stream(side):
        torch.cuda._sleep(50_000_000)     # ~20 ms: the copy is still queued when the host allocates
    srv.set_weights(src)
    old = src.data_ptr()
    del src
    fresh = [torch.empty(n, device="cuda") for _ in range(4)]
    for t in fresh:
        t.fill_(1e30)                     # on the current stream, at once
    assert old not in {t.data_ptr() for t in fresh}
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), want)
    assert not parity.np_bits(srv.velocity_copy()).view(np.uint32).any()
    srv.close()


def test_record_lets_producer_reuse_its_buffer(torch):
    """After ps_record, a producer stream that waits for the event may
    overwrite the gradient buffer; the apply already read the old values."""
    n = 8_000_001
    gen = torch.Generator(device="cuda")
    gen.manual_seed(51)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    g = torch.randn(n, generator=gen, device="cuda") * 1e-2
    g_host = parity.np_bits(g)
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=2)
    srv.set_stream(torch.cuda.current_stream())
    srv.set_weights(w0)
    torch.cuda.synchronize()
    srv.push(0, g)
    srv.apply_pending()
    done = torch.cuda.Event()
    srv.record(done)
    producer = torch.cuda.Stream()
    with torch.cuda.stream(producer):
        producer.wait_event(done)
        g.fill_(123.0)                    # the next gradient goes into the same buffer
    torch.cuda.synchronize()
    o = orc.OracleServer(parity.np_bits(w0), 0.01, 0.0, depth=2)
    o.push(0, g_host)
    o.apply_pending()
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w)
    srv.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_lock_free_pull_sees_before_or_after(torch, dtype):
    """HogWild! mode (Sec. 4.1): a pull on its own stream, concurrent with an
    apply, writes for every coordinate either the weights before the apply
    or after it (bitwise one of the two; which one may vary by coordinate).
    Nondeterministic by design, so checked by this bound, not by bits; the
    two candidates are the oracle's weights before and after that apply
    (and the server's equal them bitwise)."""
    n = 50_000_003
    gen = torch.Generator(device="cuda")
    gen.manual_seed(52)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    pool = wl.Rows(32, n, torch.float32, "cuda")
    for j in range(32):
        pool[j].normal_(0, 1e-2, generator=gen)
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=32)
    srv.set_stream(torch.cuda.current_stream())
    srv.set_weights(w0)
    for j in range(32):
        srv.push(j % 8, pool[j])
    srv.apply_pending()
    before = srv.weights_copy()
    # the weights before and after the raced apply, from the oracle
    o = orc.OracleServer(parity.np_bits(w0), 0.01, 0.9, depth=32)
    host = [parity.np_bits(pool[j]) for j in range(32)]
    for j in range(32):
        o.push(j % 8, host[j])
    o.apply_pending()
    o_before = o.w.copy()
    for j in range(32):
        o.push(j % 8, host[31 - j])
    o.apply_pending()
    o_after = o.w.copy()
    del host
    assert parity.bitwise(parity.np_bits(before), o_before)
    side = torch.cuda.Stream()
    srv.set_pull_stream(side)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dst = wl.Rows(1, n, tdt, "cuda")
    torch.cuda.synchronize()
    for j in range(32):
        srv.push(j % 8, pool[31 - j])
    srv.apply_pending()                   # long apply on the server's stream ...
    srv.pull_many([3], [dst[0]])          # ... and a pull racing it
    srv.sync()
    after = srv.weights_copy()
    assert parity.bitwise(parity.np_bits(after), o_after)
    d = parity.np_bits(dst[0])
    a, b = o_before, o_after
    if dtype == "bf16":
        a, b = orc.f32_to_bf16(a), orc.f32_to_bf16(b)
    else:
        a, b, d = a.view(np.uint32), b.view(np.uint32), d.view(np.uint32)
    assert np.all((d == a) | (d == b))
    say(f"[lock-free pull] {np.mean(d == b):.3f} of coordinates saw the new weights")
    # back to ordered pulls: a pull then sees exactly the latest weights
    srv.set_pull_stream(None)
    srv.pull_many([3], [dst[0]])
    srv.sync()
    want = o_after
    got = parity.np_bits(dst[0])
    assert parity.bitwise(got, want if dtype == "f32" else orc.f32_to_bf16(want))
    srv.close()


# ---------------------------------------------------------------- contraction-allowed build

@pytest.fixture
def fma_library(torch):
    """Swap the binding to libgadeips_fma.so (the same source built with
    -ffp-contract=fast) for one test."""
    from paper_1611_06213_amd import build as lib_build
    if not os.path.exists(lib_build.LIB_FMA):
        pytest.fail("libgadeips_fma.so is not built")
    saved = ps.load_library()
    ps._lib = ps.load_library(lib_build.LIB_FMA)
    yield
    ps._lib = saved


@pytest.mark.parametrize("name", list(wl.CONFIGS))
def test_fma_flavour_within_1e6_per_apply(torch, fma_library, name):
    """Built with contraction allowed, one apply of a full batch (K gradients,
    with momentum where the workload has it) from the same starting state
    stays within 1e-6 relative (R12: max|a-b| / max(|b|, RMS(w0))) of the
    oracle's sequential binary32 result, for the weights and the replicas."""
    cfg = wl.CONFIGS[name].scaled(SMALL_N, pool=min(wl.CONFIGS[name].pool, 64))
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    rdt = torch.bfloat16 if cfg.pull_dtype == wl.BF16 else torch.float32
    reps = wl.Rows(2, cfg.n, rdt, "cuda")
    srv = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=cfg.depth)
    srv.set_weights(w0)
    o = orc.OracleServer(parity.np_bits(w0), cfg.lr, cfg.momentum, depth=cfg.depth)
    for j in range(cfg.depth):
        srv.push(j % cfg.learners, pool[j])
        o.push(j % cfg.learners, parity.np_bits(pool[j]))
    srv.apply_pull([0, 1], reps.rows)
    o.apply_pending()
    tau = float(np.sqrt(np.mean(parity.np_bits(w0).astype(np.float64) ** 2)))
    a = parity.np_bits(srv.weights_copy()).astype(np.float64)
    b = o.w.astype(np.float64)
    err = float(np.max(np.abs(a - b) / np.maximum(np.abs(b), tau)))
    say(f"[fma] {name}: one apply of {cfg.depth}, R12 error {err:.2e}")
    assert err <= 1e-6
    if cfg.pull_dtype == wl.F32:
        r = parity.np_bits(reps[1]).astype(np.float64)
        assert np.max(np.abs(r - b) / np.maximum(np.abs(b), tau)) <= 1e-6
    srv.close()
    del pool, reps
    free(torch)


@pytest.mark.parametrize("name", list(wl.CONFIGS))
def test_fma_flavour_whole_schedule_drift_bounded(torch, fma_library, name):
    """Over a whole schedule the fused and the separately rounded runs drift
    apart like a random walk of per-step rounding differences: each step
    differs by at most about one ulp of the weight, so after T steps
    |a-b| <= 2*T*ulp(max|w|). Checked, and the R12 drift reported; with
    momentum the runs do differ (contraction really happened)."""
    cfg = wl.CONFIGS[name].scaled(SMALL_N, pool=min(wl.CONFIGS[name].pool, 64))
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ranges = [(0, cfg.n)]
    g = parity.gpu_replay(cfg, ev, pool, w0, ranges, fused=True)
    ps_, w0s = parity.host_inputs(cfg, pool, w0, ranges)
    o = parity.oracle_replay(cfg, ev, ps_, w0s, ranges)
    tau = float(np.sqrt(np.mean(w0s[0].astype(np.float64) ** 2)))
    a, b = g["w"][0].astype(np.float64), o["w"][0].astype(np.float64)
    T = o["ts"]
    ulp = float(np.spacing(np.float32(max(np.abs(b).max(), np.abs(w0s[0]).max()) * 1.5)))
    assert np.max(np.abs(a - b)) <= 2 * T * ulp
    err = float(np.max(np.abs(a - b) / np.maximum(np.abs(b), tau)))
    say(f"[fma] {name}: {T} sequential pushes, R12 drift {err:.2e}")
    if cfg.momentum:
        assert not parity.bitwise(g["w"][0], o["w"][0])
    assert g["staleness"] == o["staleness"] and g["ts"] == o["ts"]
    del pool
    free(torch)


# ---------------------------------------------------------------- layout

def _oracle_apply(torch, w0, grads, lr, m, k, pulls_bf16=False):
    o = orc.OracleServer(w0.cpu().numpy(), lr, m, depth=k)
    for j, g in enumerate(grads):
        h = g.cpu()
        h = h.view(torch.int16).numpy().view(np.uint16) if g.dtype == torch.bfloat16 else h.numpy()
        assert o.push(j % 7, h) == orc.OK
    o.apply_pending()
    return o


def test_alloc_rows_layout_and_parity(torch):
    """Server-owned rows: w at phase 0 within 2 MiB, v at 1.75 MiB, row i at
    ((i + 2) * 1.75 MiB) mod 2 MiB, no overlap, usable as fp32 and bf16
    gradients and replicas with results bitwise equal to the oracle; freeing
    refuses rows a pending gradient lies in."""
    n, k, lr, m = 3 * (1 << 20) + 5, 32, 0.01, 0.9
    say(f"[case] alloc_rows n={n} K={k}")
    two_mib = 2 << 20
    srv = ps.ParameterServer(n, lr, m, queue_depth=k)
    stagger = 7 << 18
    assert ps.ps_weights(srv.h) % two_mib == 0 and ps.ps_velocity(srv.h) % two_mib == stagger
    gen = torch.Generator(device="cuda")
    gen.manual_seed(31)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    srv.set_weights(w0)
    rows = srv.alloc_rows(k + 3)
    addrs = [r.data_ptr() for r in rows]
    assert [a % two_mib for a in addrs] == [((i + 2) * stagger) % two_mib for i in range(k + 3)]
    assert all(b - a >= 4 * n for a, b in zip(addrs, addrs[1:]))
    for r in rows[:k]:
        r.copy_(torch.randn(n, generator=gen, device="cuda") * 1e-3)
    for j in range(k):
        assert srv.push(j % 7, rows[j])
    with pytest.raises(ps.PSError) as e:
        srv.free_rows(rows)                       # pending gradients live there
    assert e.value.code == ps.PS_ESTATE
    reps16 = srv.alloc_rows(2, torch.bfloat16)
    assert [t.data_ptr() % two_mib for t in reps16] == [(2 * stagger) % two_mib, (3 * stagger) % two_mib]
    srv.apply_pull([0, 1, 2], rows[k:k + 3])
    srv.pull_many([3, 4], reps16)
    torch.cuda.synchronize()
    o = _oracle_apply(torch, w0, rows[:k], lr, m, k)
    wbits = parity.np_bits(srv.weights_copy())
    assert parity.bitwise(wbits, o.w.view(np.uint32))
    for r in rows[k:k + 3]:
        assert parity.bitwise(parity.np_bits(r), o.w.view(np.uint32))
    want16 = orc.f32_to_bf16(o.w)
    for r in reps16:
        assert np.array_equal(r.cpu().view(torch.int16).numpy().view(np.uint16), want16)
    # bf16 gradients in server rows
    g16 = srv.alloc_rows(4, torch.bfloat16)
    for r in g16:
        r.copy_((torch.randn(n, generator=gen, device="cuda") * 1e-3).to(torch.bfloat16))
    for j, r in enumerate(g16):
        assert srv.push(j, r)
    srv.apply_pending()
    for j, r in enumerate(g16):
        h = r.cpu().view(torch.int16).numpy().view(np.uint16)
        o.push(j, h)
    o.apply_pending()
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w.view(np.uint32))
    srv.free_rows(rows)
    with pytest.raises(ps.PSError):
        srv.free_rows(rows)                       # already freed
    assert ps.ps_free_rows(srv.h, g16[1].data_ptr()) == ps.PS_EINVAL   # not a first row
    srv.close()                                   # frees the remaining row sets
    free(torch)


def _host_grad(torch, g):
    h = g.cpu()
    return h.view(torch.int16).numpy().view(np.uint16) if g.dtype == torch.bfloat16 else h.numpy()


@pytest.mark.parametrize("gdt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["separate", "server_rows"])
def test_fronts_give_identical_bits(torch, layout, gdt):
    """Every front count (and the automatic choice) folds the same
    gradients into the same bits, for separately allocated buffers (one
    phase) and for server rows (distinct phases), fp32 gradients (4 per
    lane) and bf16 gradients (8 per lane); the synchronous step too."""
    n, k, lr, m = 5 * (1 << 20) + 3, 32, 0.01, 0.9
    say(f"[case] fronts layout={layout} gradients={gdt} n={n}")
    tdt = torch.bfloat16 if gdt == "bf16" else torch.float32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(37)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    holder = ps.ParameterServer(n, lr, m)
    if layout == "separate":
        grads = [torch.empty(n, dtype=tdt, device="cuda") for _ in range(k)]
    else:
        grads = holder.alloc_rows(k, tdt)
    for g in grads:
        g.copy_((torch.randn(n, generator=gen, device="cuda") * 1e-3).to(tdt))
    o = _oracle_apply(torch, w0, grads, lr, m, k)
    want = o.w.view(np.uint32).copy()
    so = orc.OracleServer(w0.cpu().numpy(), lr, m, depth=16)
    for j in range(16):
        so.push(j, _host_grad(torch, grads[j]))
    so.apply_sync()
    want_sync = so.w.view(np.uint32).copy()
    for f in (-1, 0, 1, 2, 3):
        srv = ps.ParameterServer(n, lr, m, queue_depth=k)
        srv.set_fronts(f)
        srv.set_weights(w0)
        for j, g in enumerate(grads):
            assert srv.push(j % 7, g)
        srv.apply_pending()
        assert parity.bitwise(parity.np_bits(srv.weights_copy()), want), f
        srv.set_weights(w0)
        for j in range(16):
            assert srv.push(j, grads[j])
        srv.apply_sync()
        assert parity.bitwise(parity.np_bits(srv.weights_copy()), want_sync), f
        srv.close()
    with pytest.raises(ps.PSError):
        holder.set_fronts(4)
    holder.close()
    free(torch)


@pytest.mark.parametrize("rdt", ["f32", "bf16"])
def test_argument_block_boundary(torch, rdt):
    """Launches of at most 8 gradients and 8 replicas run over the compact
    argument block, larger ones over the full one: at K = 7, 8, 9 and 16
    gradients and R = 7, 8, 9 and 16 replicas, ps_apply_pull with the
    replicas written from the apply pass, and the same apply followed by
    ps_pull_many, give the oracle's w, v and replica bits."""
    n, lr, m = 4 * 8192 + 3, 0.01, 0.9
    say(f"[case] argument block boundary replicas={rdt} n={n}")
    tdt = torch.bfloat16 if rdt == "bf16" else torch.float32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(43)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    grads = [torch.randn(n, generator=gen, device="cuda") * 1e-3 for _ in range(16)]
    host = [g.cpu().numpy() for g in grads]
    srv = ps.ParameterServer(n, lr, m, queue_depth=16)
    for k in (7, 8, 9, 16):
        o = orc.OracleServer(w0.cpu().numpy(), lr, m, depth=16)
        for j in range(k):
            assert o.push(j, host[j]) == orc.OK
        o.apply_pending()
        want_w, want_v = o.w.view(np.uint32).copy(), o.v.view(np.uint32).copy()
        want_r = want_w.view(np.float32) if rdt == "f32" else orc.f32_to_bf16(want_w.view(np.float32))
        for r in (7, 8, 9, 16):
            for fused in (True, False):
                reps = [torch.full((n,), float("nan"), dtype=tdt, device="cuda") for _ in range(r)]
                srv.set_weights(w0)
                for j in range(k):
                    assert srv.push(j, grads[j])
                if fused:
                    srv.set_pull_fusion(64)
                    srv.apply_pull(list(range(r)), reps)
                    srv.set_pull_fusion(-1)
                else:
                    srv.apply_pending()
                    srv.pull_many(list(range(r)), reps)
                assert parity.bitwise(parity.np_bits(srv.weights_copy()), want_w), (k, r, fused)
                assert parity.bitwise(parity.np_bits(srv.velocity_copy()), want_v), (k, r, fused)
                for rep in reps:
                    assert parity.bitwise(parity.np_bits(rep), want_r), (k, r, fused)
    srv.close()
    free(torch)


@pytest.mark.parametrize("m", [0.0, 0.9])
@pytest.mark.parametrize("gdt", ["f32", "bf16"])
def test_every_group_and_remainder(torch, gdt, m):
    """Every gradient group size the launcher takes (4, 8, 12, 16, 24, 32),
    forced with ps_set_launch_shape at every depth from 1 to two groups and 8
    more (at most 64), so that the first group, the loop over further groups,
    the groups of 16 and 8 and each exact remainder of 1..7 all run, under residency caps 0..4 in turn:
    w and v equal the oracle's bits after the same gradients (batched is
    sequential, so one oracle run gives every depth); the same applies writing
    two fp32 or bf16 replicas from their own pass give those bits and RNE of
    them; the synchronous step at every group size and depth too."""
    n, lr, kmax = 3 * 8192 + 5, 0.01, 64
    say(f"[case] groups x remainders gradients={gdt} m={m} n={n}")
    tdt = torch.bfloat16 if gdt == "bf16" else torch.float32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(41)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    grads = [(torch.randn(n, generator=gen, device="cuda") * 1e-3).to(tdt) for _ in range(kmax)]
    host = [_host_grad(torch, g) for g in grads]
    o = orc.OracleServer(w0.cpu().numpy(), lr, m, depth=1)
    want = {}
    for k in range(1, kmax + 1):
        assert o.push(0, host[k - 1]) == orc.OK
        o.apply_pending()
        want[k] = (o.w.view(np.uint32).copy(), None if m == 0 else o.v.view(np.uint32).copy())
    want_sync = {}
    for k in range(1, kmax + 1):
        so = orc.OracleServer(w0.cpu().numpy(), lr, m, depth=k)
        for j in range(k):
            assert so.push(j, host[j]) == orc.OK
        so.apply_sync()
        want_sync[k] = so.w.view(np.uint32).copy()
    srv = ps.ParameterServer(n, lr, m, queue_depth=kmax)
    case = 0
    for group in (4, 8, 12, 16, 24, 32):
        for k in range(1, min(2 * group + 8, kmax) + 1):
            srv.set_launch_shape(case % 5, group)
            case += 1
            srv.set_weights(w0)
            for j in range(k):
                assert srv.push(j % 7, grads[j])
            srv.apply_pending()
            ww, wv = want[k]
            assert parity.bitwise(parity.np_bits(srv.weights_copy()), ww), (group, k)
            if m != 0:
                assert parity.bitwise(parity.np_bits(srv.velocity_copy()), wv), (group, k)
            # the same apply writing two replicas from its own pass
            rdt = torch.float32 if case % 2 else torch.bfloat16
            reps = [torch.full((n,), float("nan"), dtype=rdt, device="cuda") for _ in range(2)]
            srv.set_pull_fusion(64)
            srv.set_weights(w0)
            for j in range(k):
                assert srv.push(j % 7, grads[j])
            srv.apply_pull([0, 1], reps)
            srv.set_pull_fusion(-1)
            assert parity.bitwise(parity.np_bits(srv.weights_copy()), ww), ("fused", group, k)
            rw = ww.view(np.float32) if rdt == torch.float32 else orc.f32_to_bf16(ww.view(np.float32))
            for rep in reps:
                assert parity.bitwise(parity.np_bits(rep), rw), ("replica", group, k, rdt)
            srv.set_weights(w0)
            for j in range(k):
                assert srv.push(j, grads[j])
            srv.apply_sync()
            assert parity.bitwise(parity.np_bits(srv.weights_copy()), want_sync[k]), ("sync", group, k)
    srv.set_launch_shape()
    for bad in ((-2, 0), (5, 0), (1, 3), (1, 20), (1, 40)):
        with pytest.raises(ps.PSError):
            srv.set_launch_shape(*bad)
    srv.close()
    free(torch)


# ---------------------------------------------------------------- host threads

def test_learner_threads_push_while_server_applies(torch):
    """Eight learner threads push concurrently (ctypes drops the GIL, so the C
    calls overlap) while the main thread applies and pulls, as in the paper's
    thread layout (Sec. 4.1). Every accepted push is applied exactly once,
    each learner's gradients in its own order (Theorem 2), and the weights
    equal the oracle replaying the order the server reports."""
    import threading
    n, learners, per, lr, m = (1 << 20) + 3, 8, 24, 0.01, 0.9
    say(f"[case] threads learners={learners} pushes={learners * per}")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(61)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    grads = [[torch.randn(n, generator=gen, device="cuda") * 1e-3 for _ in range(per)]
             for _ in range(learners)]
    srv = ps.ParameterServer(n, lr, m, queue_depth=32)
    srv.set_stream(torch.cuda.current_stream())
    srv.set_weights(w0)
    torch.cuda.synchronize()
    h = srv.h
    errors = []

    def learner(l):
        for j in range(per):
            while True:
                rc = ps.ps_push_dtype(h, l, grads[l][j].data_ptr(), ps.PS_F32)
                if rc == ps.PS_OK:
                    break
                if rc != ps.PS_EFULL:
                    errors.append((l, j, rc))
                    return

    threads = [threading.Thread(target=learner, args=(l,)) for l in range(learners)]
    for t in threads:
        t.start()
    order = []
    dst = torch.empty(n, device="cuda")
    while len(order) < learners * per:
        assert ps.ps_apply_pending(h) == ps.PS_OK
        order += ps.ps_last_applied(h)
        assert ps.ps_pull_many(h, [len(order) % learners], [dst.data_ptr()], ps.PS_F32) == 0
        if not any(t.is_alive() for t in threads) and ps.ps_pending(h) == 0:
            break
    for t in threads:
        t.join()
    assert ps.ps_apply_pending(h) == ps.PS_OK
    order += ps.ps_last_applied(h)
    assert errors == []
    assert len(order) == learners * per and all(order.count(l) == per for l in range(learners))
    st = srv.stats()
    assert st.pushes_accepted == st.pushes_applied == srv.timestamp == learners * per
    # replay: the j-th time learner l appears is its j-th gradient
    o = orc.OracleServer(w0.cpu().numpy(), lr, m, depth=1)
    seen = [0] * learners
    for l in order:
        assert o.push(l, grads[l][seen[l]].cpu().numpy()) == orc.OK
        o.apply_pending()
        seen[l] += 1
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), o.w.view(np.uint32))
    assert parity.bitwise(parity.np_bits(srv.velocity_copy()), o.v.view(np.uint32))
    srv.close()
    free(torch)


def test_buffers_overlapping_w_or_v_are_refused(torch):
    """A gradient, a replica or a set_weights source that shares bytes with
    the server's w or v is refused with PS_EINVAL before any state changes
    or device work: w, v, the queue and the other replicas stay as they
    were."""
    n = 4099
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=4)
    w0 = (torch.arange(n, device="cuda", dtype=torch.float32) - 2000.0) * 1e-3
    srv.set_weights(w0)
    g = torch.full((n,), 0.5, device="cuda")
    assert srv.push(0, g)
    srv.apply_pending()
    w_before = parity.np_bits(srv.weights_copy())
    v_before = parity.np_bits(srv.velocity_copy())
    h = srv.h
    wp, vp = ps.ps_weights(h), ps.ps_velocity(h)
    assert wp and vp
    ts = srv.timestamp
    # gradients: w itself, a bf16 view ending inside w, v shifted by 4 bytes
    assert ps.ps_push_dtype(h, 1, wp, ps.PS_F32) == ps.PS_EINVAL
    assert ps.ps_push_dtype(h, 1, wp - 2 * n + 2, ps.PS_BF16) == ps.PS_EINVAL
    assert ps.ps_push_dtype(h, 1, vp + 4, ps.PS_F32) == ps.PS_EINVAL
    assert "overlaps" in ps.ps_last_error()
    assert srv.pending == 0
    # replicas: one good buffer and one overlapping w or v, in either order
    good = torch.full((n,), 7.0, device="cuda")
    for bad, dt in ((wp, ps.PS_F32), (wp + 4 * n - 2, ps.PS_BF16), (vp, ps.PS_F32)):
        for ptrs in ([good.data_ptr(), bad], [bad, good.data_ptr()]):
            assert ps.ps_pull_many(h, [0, 1], ptrs, dt) == ps.PS_EINVAL
            assert ps.load_library().ps_apply_pull(h, 2, ps._ints([0, 1]), ps._ptrs(ptrs), dt) \
                == ps.PS_EINVAL
    assert ps.ps_set_weights(h, wp) == ps.PS_EINVAL
    assert ps.ps_set_weights(h, vp - 8) == ps.PS_EINVAL
    srv.sync()
    assert srv.timestamp == ts and srv.pending == 0
    assert bool((good == 7.0).all())
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), w_before)
    assert parity.bitwise(parity.np_bits(srv.velocity_copy()), v_before)
    # a buffer that ends where w starts, or starts where w ends, does not
    # overlap it (a push only records the pointer; both are dropped unapplied)
    assert ps.ps_push_dtype(h, 3, wp - 4 * n, ps.PS_F32) == ps.PS_OK
    assert ps.ps_push_dtype(h, 3, wp + 4 * n, ps.PS_F32) == ps.PS_OK
    assert ps.ps_drop_learner(h, 3) == 2 and srv.pending == 0
    srv.close()


def test_alloc_rows_argument_errors(torch):
    """ps_alloc_rows / ps_free_rows / ps_set_fronts / ps_set_pull_fusion
    refuse bad arguments with PS_EINVAL and change nothing."""
    srv = ps.ParameterServer(1000, 0.01, 0.0)
    assert ps.ps_alloc_rows(srv.h, 0, ps.PS_F32)[0] == ps.PS_EINVAL
    assert ps.ps_alloc_rows(srv.h, ps.PS_MAX_ROWS + 1, ps.PS_F32)[0] == ps.PS_EINVAL
    assert ps.ps_alloc_rows(srv.h, 2, 7)[0] == ps.PS_EINVAL
    assert ps.load_library().ps_alloc_rows(srv.h, 2, ps.PS_F32, None) == ps.PS_EINVAL
    assert ps.ps_free_rows(srv.h, 0) == ps.PS_EINVAL
    assert ps.ps_set_fronts(srv.h, -2) == ps.PS_EINVAL and ps.ps_set_fronts(srv.h, 4) == ps.PS_EINVAL
    assert ps.ps_set_pull_fusion(srv.h, -2) == ps.PS_EINVAL
    assert ps.ps_set_pull_fusion(srv.h, ps.PS_MAX_REPLICAS + 1) == ps.PS_EINVAL
    assert ps.ps_set_pull_fusion(srv.h, -1) == ps.PS_OK and ps.ps_set_pull_fusion(srv.h, 0) == ps.PS_OK
    rc, rows = ps.ps_alloc_rows(srv.h, ps.PS_MAX_ROWS, ps.PS_BF16)   # 4096 rows of 1000 values
    assert rc == ps.PS_OK and len(set(rows)) == ps.PS_MAX_ROWS
    assert ps.ps_free_rows(srv.h, rows[1]) == ps.PS_EINVAL           # not a first row
    assert ps.ps_free_rows(srv.h, rows[0]) == ps.PS_OK
    srv.close()
