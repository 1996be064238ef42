"""GPU tests of protocol rules added around the kernels: a dead learner's
gradients in the server's rows (retire), checkpoints that carry the queue
configuration, apply+pull after lock-free pulls, and the binding keeping
every gradient that is still queued alive."""
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


def test_golden_retire_through_abi(torch):
    """tests/golden/retire_rr.txt through the C ABI, every gradient in a
    server row (the paper's shared slots): service order, staleness,
    refused push and pull of the retired learner, counters, weights."""
    depth, ops, expect, mode = golden_script.load("retire_rr.txt", with_mode=True)
    n = 4
    srv = ps.ParameterServer(n, 2.0 ** -4, 0.0, queue_depth=depth)
    srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, mode[1])
    srv.set_weights(torch.zeros(n, device="cuda"))
    rows = srv.alloc_rows(len(ops))
    for r in rows:
        r.fill_(0.5)
    dsts = {l: torch.empty(n, device="cuda") for l in range(3)}
    order, stale = [], []
    for i, (op, l, outcome) in enumerate(ops):
        if op == "push":
            rc = ps.ps_push(srv.h, l, rows[i].data_ptr())
            assert rc == {"ok": ps.PS_OK, "full": ps.PS_EFULL, "refused": ps.PS_ESTATE}[outcome]
        elif op == "apply":
            srv.apply_pending()
            order += srv.last_applied()
            stale += srv.last_staleness()
        elif op == "retire":
            assert ps.ps_retire_learner(srv.h, l) == int(outcome)
        elif op == "drop":
            assert ps.ps_drop_learner(srv.h, l) == int(outcome)
        elif outcome == "refused":
            assert ps.ps_pull(srv.h, l, dsts[l].data_ptr()) == ps.PS_ESTATE
        else:
            before = srv.stats().pulls_skipped
            srv.pull(l, dsts[l])
            assert (srv.stats().pulls_skipped == before) == (outcome == "pulled")
    st = srv.stats()
    assert order == expect["order"] and stale == expect["staleness"]
    assert srv.timestamp == expect["ts"][0]
    assert (st.pulls, st.pulls_skipped, st.pushes_rejected) == (
        expect["pulls"], expect["skipped"], expect["rejected"])
    assert torch.all(srv.weights_copy() == -6 / 32)
    # a new run (set_weights) readmits the retired learner
    srv.set_weights(torch.zeros(n, device="cuda"))
    assert ps.ps_push(srv.h, 1, rows[0].data_ptr()) == ps.PS_OK
    srv.apply_pending()
    del rows
    srv.close()


def test_retire_refuses_borrowed_buffers(torch):
    """A queued gradient outside the server's rows may have died with its
    learner: retiring that learner is refused (nothing changes) and dropping
    is the way; a learner with only row gradients queued retires."""
    n = 100_003
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=8)
    srv.set_weights(torch.zeros(n, device="cuda"))
    rows = srv.alloc_rows(2)
    own = torch.ones(n, device="cuda")
    assert srv.push(0, rows[0]) and srv.push(1, own) and srv.push(0, rows[1])
    assert ps.ps_retire_learner(srv.h, 1) == ps.PS_ESTATE
    assert srv.pending == 3 and ps.ps_push(srv.h, 1, own.data_ptr()) == ps.PS_OK   # not retired
    assert ps.ps_retire_learner(srv.h, 0) == 2
    assert ps.ps_push(srv.h, 0, rows[0].data_ptr()) == ps.PS_ESTATE
    assert ps.ps_drop_learner(srv.h, 1) == 2
    srv.apply_pending()
    assert srv.last_applied() == [0, 0] and srv.timestamp == 2
    assert ps.ps_retire_learner(srv.h, -1) == ps.PS_EINVAL
    del rows
    srv.close()


def test_checkpoint_keeps_queue_configuration(torch, tmp_path):
    """A checkpoint records the queue mode, depth and slots per learner; a
    server set up otherwise refuses it (PS_EINVAL, unchanged), since the
    same gradients would then be served in another order."""
    n = 10_007
    a = ps.ParameterServer(n, 0.01, 0.9, queue_depth=4)
    a.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, 2)
    a.set_weights(torch.full((n,), 0.25, device="cuda"))
    g = torch.ones(n, device="cuda")
    a.push(0, g)
    a.apply_pending()
    path = str(tmp_path / "q.ckpt")
    a.save(path)
    for depth, mode, slots in ((4, ps.PS_QUEUE_FIFO, 1), (8, ps.PS_QUEUE_ROUND_ROBIN, 2),
                               (4, ps.PS_QUEUE_ROUND_ROBIN, 3)):
        b = ps.ParameterServer(n, 0.01, 0.9, queue_depth=depth)
        if mode == ps.PS_QUEUE_ROUND_ROBIN:
            b.set_queue_mode(mode, slots)
        b.set_weights(torch.zeros(n, device="cuda"))
        assert ps.ps_load(b.h, path) == ps.PS_EINVAL and "queue configuration" in ps.ps_last_error()
        assert torch.all(b.weights_copy() == 0) and b.timestamp == 0
        b.close()
    c = ps.ParameterServer(n, 0.01, 0.9, queue_depth=4)
    c.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, 2)
    c.load(path)
    assert c.timestamp == 1
    assert parity.bitwise(parity.np_bits(c.weights_copy()), parity.np_bits(a.weights_copy()))
    a.close()
    c.close()


def test_apply_pull_after_lock_free_pulls(torch):
    """Lock-free pulls of 64 replicas (slow) on their own stream, then at
    once an apply+pull into one of those replicas on the server's stream:
    the replica ends with the new weights (the apply+pull waits for the
    earlier lock-free pulls), and a repeat pull is skipped as current and
    leaves it so. Checked against the oracle."""
    n = 4_000_037
    gen = torch.Generator(device="cuda")
    gen.manual_seed(61)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    g = torch.randn(n, generator=gen, device="cuda") * 1e-2
    reps = wl.Rows(64, n, torch.float32, "cuda")
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=4)
    srv.set_stream(torch.cuda.current_stream())
    srv.set_weights(w0)
    side = torch.cuda.Stream()
    srv.set_pull_stream(side)
    torch.cuda.synchronize()
    srv.pull_many(list(range(64)), [reps[l] for l in range(64)])   # lock-free, old weights
    srv.push(5, g)
    srv.apply_pull([5], [reps[5]])                                  # ordered, new weights
    srv.apply_pull([5], [reps[5]])                                  # nothing pending: skipped
    srv.sync()
    assert srv.stats().pulls_skipped == 1
    o = orc.OracleServer(parity.np_bits(w0), 0.01, 0.0, depth=4)
    o.push(5, parity.np_bits(g))
    o.apply_pending()
    assert parity.bitwise(parity.np_bits(reps[5]), o.w)
    assert parity.bitwise(parity.np_bits(reps[6]), parity.np_bits(w0))
    srv.set_pull_stream(None)
    srv.close()


def test_binding_keeps_unapplied_gradients_referenced(torch):
    """Round-robin queues, 4 learners x 2 slots, depth 2: each apply takes
    two gradients and leaves the rest queued. The caller drops its own
    references right after the first apply and allocates and fills new
    tensors; the binding must keep the queued gradients alive (their memory
    not reused) until their applies are enqueued. Bitwise against the
    oracle."""
    n = 1_000_003
    gen = torch.Generator(device="cuda")
    gen.manual_seed(62)
    w0 = (torch.rand(n, generator=gen, device="cuda") - 0.5) * 0.1
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=2)
    srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, 2)
    srv.set_stream(torch.cuda.current_stream())
    srv.set_weights(w0)
    grads = [torch.randn(n, generator=gen, device="cuda") * 1e-2 for _ in range(8)]
    host = [parity.np_bits(t) for t in grads]
    for j, t in enumerate(grads):
        assert srv.push(j % 4, t)
    srv.apply_pending()
    del grads, t                        # the caller lets go of every gradient
    junk = [torch.full((n,), 1e6, device="cuda") for _ in range(8)]   # would reuse freed blocks
    while srv.pending:
        srv.apply_pending()
    w = parity.np_bits(srv.weights_copy())
    o = orc.OracleServer(parity.np_bits(w0), 0.01, 0.9, depth=2)
    o.set_queue_mode(orc.ROUND_ROBIN, 2)
    for j, hg in enumerate(host):
        o.push(j % 4, hg)
    while o.pending():
        o.apply_pending()
    assert parity.bitwise(w, o.w)
    assert srv._pending == {}
    del junk
    srv.close()


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_run_script_equals_calls(torch, fused):
    """ps_run over a prepared schedule (pushes, applies, pulls) gives the
    bits, staleness and counters of the same calls made one by one; it
    stops at the first call that fails (a full queue) and reports how many
    ran."""
    cfg = wl.CONFIGS["alexnet"].scaled(200_003, pushes=96, pool=16)
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    out = []
    for native in (False, True):
        srv = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=cfg.depth)
        srv.set_stream(torch.cuda.current_stream())
        srv.set_weights(w0)
        reps = wl.Rows(cfg.replicas, cfg.n, torch.float32, "cuda")
        sc = ps.OpScript()
        i = 0
        while i < len(ev):
            e = ev[i]
            if isinstance(e, wl.Push):
                if native:
                    sc.push(e.learner, pool[e.buf].data_ptr())
                else:
                    assert ps.ps_push(srv.h, e.learner, pool[e.buf].data_ptr()) == ps.PS_OK
            elif isinstance(e, wl.Apply):
                nxt = ev[i + 1] if i + 1 < len(ev) else None
                if fused and isinstance(nxt, wl.Pull):
                    ls = parity.pull_rounds(nxt.learners)
                    dl = [reps[l].data_ptr() for l in ls[0]]
                    if native:
                        sc.apply_pull(ls[0], dl)
                    else:
                        assert ps.ps_apply_pull(srv.h, ls[0], dl, ps.PS_F32) == ps.PS_OK
                    for rnd in ls[1:]:
                        dr = [reps[l].data_ptr() for l in rnd]
                        sc.pull(rnd, dr) if native else ps.ps_pull_many(srv.h, rnd, dr, ps.PS_F32)
                    i += 2
                    continue
                sc.apply() if native else ps.ps_apply_pending(srv.h)
            else:
                for rnd in parity.pull_rounds(e.learners):
                    dr = [reps[l].data_ptr() for l in rnd]
                    sc.pull(rnd, dr) if native else ps.ps_pull_many(srv.h, rnd, dr, ps.PS_F32)
            i += 1
        if native:
            assert ps.ps_run(srv.h, sc) == (ps.PS_OK, len(sc))
        st = srv.stats()
        out.append((parity.np_bits(srv.weights_copy()), parity.np_bits(srv.velocity_copy()),
                    [parity.np_bits(reps[l]) for l in range(cfg.replicas)], srv.last_staleness(),
                    (st.timestamp, st.pushes_applied, st.pulls, st.pulls_skipped, st.staleness_sum)))
        srv.close()
        del reps
    (wa, va, ra, sa, ca), (wb, vb, rb, sb, cb) = out
    assert parity.bitwise(wa, wb) and parity.bitwise(va, vb) and sa == sb and ca == cb
    assert all(parity.bitwise(x, y) for x, y in zip(ra, rb))
    # a script that overfills the queue stops at the refused push
    srv = ps.ParameterServer(cfg.n, cfg.lr, 0.0, queue_depth=2)
    sc = ps.OpScript()
    for j in range(3):
        sc.push(j, pool[j].data_ptr())
    sc.apply()
    assert ps.ps_run(srv.h, sc) == (ps.PS_EFULL, 2)
    assert srv.pending == 2
    assert ps.ps_run(srv.h, ps.OpScript()) == (ps.PS_OK, 0)
    srv.apply_pending()
    srv.close()
    del pool


def _schedule_script(cfg, ev, pool, reps, fused, sync=False):
    """An OpScript of a workload schedule in the workload's gradient and
    replica dtypes: pushes, applies (or apply+pull with the first pull
    round; with sync, synchronous steps) and pull rounds."""
    sc = ps.OpScript()
    gdt, pdt = cfg.grad_dtype, cfg.pull_dtype
    i = 0
    while i < len(ev):
        e = ev[i]
        if isinstance(e, wl.Push):
            sc.push(e.learner, pool[e.buf].data_ptr(), gdt)
        elif isinstance(e, wl.Apply):
            nxt = ev[i + 1] if i + 1 < len(ev) else None
            if sync:
                sc.apply_sync()
            elif fused and isinstance(nxt, wl.Pull):
                ls = parity.pull_rounds(nxt.learners)
                sc.apply_pull(ls[0], [reps[l].data_ptr() for l in ls[0]], pdt)
                for rnd in ls[1:]:
                    sc.pull(rnd, [reps[l].data_ptr() for l in rnd], pdt)
                i += 2
                continue
            else:
                sc.apply()
        else:
            for rnd in parity.pull_rounds(e.learners):
                sc.pull(rnd, [reps[l].data_ptr() for l in rnd], pdt)
        i += 1
    return sc


def _state(srv, reps, n_reps):
    st = srv.stats()
    return (parity.np_bits(srv.weights_copy()), parity.np_bits(srv.velocity_copy()),
            [parity.np_bits(reps[l]) for l in range(n_reps)], srv.last_staleness(),
            (st.timestamp, st.pushes_applied, st.pulls, st.pulls_skipped, st.staleness_sum))


@pytest.mark.parametrize("name,fused,sync", [("alexnet", False, False), ("alexnet", True, False),
                                             ("mixed", False, False), ("mixed", True, False),
                                             ("vgg16", False, True)],
                         ids=["alexnet-separate", "alexnet-fused", "mixed-bf16-separate",
                              "mixed-bf16-fused", "vgg16-ssgd"])
def test_graph_replays_equal_run(torch, name, fused, sync):
    """A schedule captured as a HIP graph (ps_graph_create) and replayed
    (ps_graph_launch) three times, each after resetting the weights and with
    other work enqueued and synchronized on the same stream in between,
    gives every time the bits, staleness and counters of ps_run of the same
    schedule (fp32, or bf16 gradients and replicas; asynchronous applies,
    apply+pull, or synchronous steps); capturing runs nothing and leaves the
    server's state as it was."""
    cfg = wl.CONFIGS[name].scaled(200_003, pushes=96, pool=16)
    ev = wl.schedule(cfg)
    pool = wl.make_pool(cfg, "cuda")
    w0 = wl.make_w0(cfg, "cuda")
    ref = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=cfg.depth)
    ref.set_stream(torch.cuda.current_stream())
    ref.set_weights(w0)
    rdt = torch.bfloat16 if cfg.pull_dtype == ps.PS_BF16 else torch.float32
    ref_reps = wl.Rows(cfg.replicas, cfg.n, rdt, "cuda")
    sc = _schedule_script(cfg, ev, pool, ref_reps, fused, sync)
    assert ps.ps_run(ref.h, sc) == (ps.PS_OK, len(sc))
    want = _state(ref, ref_reps, cfg.replicas)
    ref.close()

    stream = torch.cuda.Stream()
    srv = ps.ParameterServer(cfg.n, cfg.lr, cfg.momentum, queue_depth=cfg.depth, stream=stream)
    srv.set_weights(w0)
    srv.sync()
    reps = wl.Rows(cfg.replicas, cfg.n, rdt, "cuda")
    reps.buf.fill_(7.0)
    w_before = parity.np_bits(srv.weights_copy())
    rc, graph = ps.ps_graph_create(srv.h, _schedule_script(cfg, ev, pool, reps, fused, sync))
    assert rc == ps.PS_OK and graph
    srv.sync()
    assert srv.timestamp == 0 and ps.ps_pending(srv.h) == 0 and srv.stats().pulls == 0
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), w_before)
    assert float(reps.buf.max()) == 7.0 == float(reps.buf.min())
    side = torch.ones(1 << 20, device="cuda")
    for rep in range(3):
        srv.set_weights(w0)
        with torch.cuda.stream(stream):
            side.mul_(1.5)
        torch.cuda.synchronize()
        assert ps.ps_graph_launch(srv.h, graph) == ps.PS_OK, ps.ps_last_error()
        srv.sync()
        got = _state(srv, reps, cfg.replicas)
        assert parity.bitwise(got[0], want[0]) and parity.bitwise(got[1], want[1]), rep
        for a, b in zip(got[2], want[2]):
            assert parity.bitwise(a, b), rep
        assert got[3] == want[3] and got[4] == want[4], rep
    ps.ps_graph_destroy(graph)
    srv.close()


def test_graph_refuses_a_moved_round_robin_order(torch):
    """Round-robin queues: a cycle that leaves the service position on
    another learner makes the next cycle serve the learners in another
    order, so its kernels differ from the captured ones. The first replay
    runs (it starts where the capture started) and equals ps_run; the second
    is refused with PS_ESTATE and nothing changes; after ps_set_weights
    (which restarts the service order) it runs again."""
    n = 100_003
    stream = torch.cuda.Stream()
    srv = ps.ParameterServer(n, 0.01, 0.9, queue_depth=2, stream=stream)
    srv.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, 2)
    w0 = torch.rand(n, device="cuda")
    gs = [torch.full((n,), 0.25 * (j + 1), device="cuda") for j in range(4)]
    sc = ps.OpScript()
    for l, j in ((0, 0), (1, 1), (2, 2)):
        sc.push(l, gs[j].data_ptr())
    sc.apply()                       # serves learners 0 and 1
    sc.push(0, gs[3].data_ptr())
    sc.apply()                       # serves 2, then 0: the position ends on 0

    ref = ps.ParameterServer(n, 0.01, 0.9, queue_depth=2, stream=stream)
    ref.set_queue_mode(ps.PS_QUEUE_ROUND_ROBIN, 2)
    ref.set_weights(w0)
    assert ps.ps_run(ref.h, sc) == (ps.PS_OK, len(sc))
    ref.sync()
    want_w, want_v = parity.np_bits(ref.weights_copy()), parity.np_bits(ref.velocity_copy())
    want_order = ref.last_applied()
    ref.close()

    srv.set_weights(w0)
    rc, graph = ps.ps_graph_create(srv.h, sc)
    assert rc == ps.PS_OK
    assert ps.ps_graph_launch(srv.h, graph) == ps.PS_OK, ps.ps_last_error()
    srv.sync()
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), want_w)
    assert parity.bitwise(parity.np_bits(srv.velocity_copy()), want_v)
    assert srv.last_applied() == want_order
    ts, stats = srv.timestamp, srv.stats()
    assert ps.ps_graph_launch(srv.h, graph) == ps.PS_ESTATE
    assert srv.timestamp == ts == 4 and ps.ps_pending(srv.h) == 0
    assert srv.stats().pushes_applied == stats.pushes_applied
    srv.sync()
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), want_w)
    srv.set_weights(w0)
    assert ps.ps_graph_launch(srv.h, graph) == ps.PS_OK
    srv.sync()
    assert parity.bitwise(parity.np_bits(srv.weights_copy()), want_w)
    ps.ps_graph_destroy(graph)
    srv.close()


def test_graph_destroy_waits_for_its_launches(torch):
    """ps_graph_destroy right after 20 replays, with no synchronization in
    between, returns only once they have run: the stream is idle then, and
    the replica holds the 20th step's weights (20 sequential binary32 steps
    of Eq. gd, computed here in numpy)."""
    n = 1_000_003
    stream = torch.cuda.Stream()
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=2, stream=stream)
    w0 = torch.rand(n, device="cuda")
    srv.set_weights(w0)
    g = torch.full((n,), 0.25, device="cuda")
    rep = torch.empty(n, device="cuda")
    step = ps.OpScript()
    step.push(0, g.data_ptr())
    step.apply_pull([0], [rep.data_ptr()])
    rc, graph = ps.ps_graph_create(srv.h, step)
    assert rc == ps.PS_OK
    for _ in range(20):
        assert ps.ps_graph_launch(srv.h, graph) == ps.PS_OK
    ps.ps_graph_destroy(graph)
    assert stream.query()
    w = w0.cpu().numpy().astype(np.float32)
    p = np.float32(np.float32(0.01) * np.float32(0.25))
    for _ in range(20):
        w = (w - p).astype(np.float32)
    assert parity.bitwise(parity.np_bits(rep), w.view(np.uint32))
    assert srv.timestamp == 20
    srv.close()


def test_graph_binding(torch):
    """ParameterServer.capture and Graph: two replays of a push + apply_pull
    script give the two sequential binary32 steps; a replay whose pull would
    now be skipped raises PSError(PS_ESTATE) with nothing changed; close()
    is idempotent and a closed graph refuses to launch."""
    n = 50_003
    stream = torch.cuda.Stream()
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=2, stream=stream)
    w0 = torch.rand(n, device="cuda")
    srv.set_weights(w0)
    g = torch.full((n,), 0.5, device="cuda")
    rep = torch.empty(n, device="cuda")
    step = ps.OpScript()
    step.push(0, g.data_ptr())
    step.apply_pull([0], [rep.data_ptr()])
    pull_only = ps.OpScript()
    pull_only.pull([0], [rep.data_ptr()])
    pg = srv.capture(pull_only)              # captured while the pull writes
    with srv.capture(step) as graph:
        graph.launch()
        graph.launch()
        srv.sync()
        w = w0.cpu().numpy().astype(np.float32)
        p = np.float32(np.float32(0.01) * np.float32(0.5))
        for _ in range(2):
            w = (w - p).astype(np.float32)
        assert parity.bitwise(parity.np_bits(rep), w.view(np.uint32))
        pulls = srv.stats().pulls
        with pytest.raises(ps.PSError) as e:
            pg.launch()                      # the replica is current: skipped now
        assert e.value.code == ps.PS_ESTATE
        assert srv.timestamp == 2 and srv.stats().pulls == pulls
    pg.close()
    graph.close()
    with pytest.raises(ps.PSError):
        graph.launch()
    srv.close()


def test_graph_launch_checks_the_plan(torch):
    """A replay runs only if the calls would launch exactly the captured
    kernels: a pull written at capture that would now be skipped refuses the
    launch with PS_ESTATE and nothing changes; after a reset it runs again.
    Graphs need a stream other than the null stream, ordered pulls and an
    empty queue; a script that launches nothing, one that fails, and a graph
    of another server are refused."""
    n = 100_003
    stream = torch.cuda.Stream()
    srv = ps.ParameterServer(n, 0.01, 0.0, queue_depth=2, stream=stream)
    w0 = torch.rand(n, device="cuda")
    srv.set_weights(w0)
    g = torch.full((n,), 0.25, device="cuda")
    rep = torch.empty(n, device="cuda")

    pull_only = ps.OpScript()
    pull_only.pull([0], [rep.data_ptr()])
    rc, graph = ps.ps_graph_create(srv.h, pull_only)
    assert rc == ps.PS_OK
    assert ps.ps_graph_launch(srv.h, graph) == ps.PS_OK        # written, as at capture
    srv.sync()
    assert parity.bitwise(parity.np_bits(rep), parity.np_bits(w0))
    pulls = srv.stats().pulls
    assert ps.ps_graph_launch(srv.h, graph) == ps.PS_ESTATE    # would be skipped now
    assert srv.stats().pulls == pulls and srv.stats().pulls_skipped == 0
    srv.set_weights(w0)                                         # pull history cleared
    assert ps.ps_graph_launch(srv.h, graph) == ps.PS_OK

    step = ps.OpScript()
    step.push(0, g.data_ptr())
    step.apply_pull([0], [rep.data_ptr()])
    rc, g2 = ps.ps_graph_create(srv.h, step)
    assert rc == ps.PS_OK
    for k in range(1, 4):                                       # each replay one more step
        assert ps.ps_graph_launch(srv.h, g2) == ps.PS_OK
        assert srv.timestamp == k
    srv.sync()
    want = (w0.cpu().numpy().astype(np.float32) - np.float32(3 * np.float32(0.01) * np.float32(0.25)))
    assert np.allclose(parity.np_bits(rep), want, rtol=0, atol=1e-6)

    assert ps.ps_push(srv.h, 0, g.data_ptr()) == ps.PS_OK      # a pending gradient
    assert ps.ps_graph_launch(srv.h, g2) == ps.PS_ESTATE
    assert ps.ps_graph_create(srv.h, step)[0] == ps.PS_ESTATE
    srv.apply_pending()
    ts = srv.timestamp
    pushes_only = ps.OpScript()
    pushes_only.push(0, g.data_ptr())
    assert ps.ps_graph_create(srv.h, pushes_only)[0] == ps.PS_EINVAL   # launches nothing
    full = ps.OpScript()
    for _ in range(3):
        full.push(0, g.data_ptr())
    full.apply()
    assert ps.ps_graph_create(srv.h, full)[0] == ps.PS_EFULL          # the third push fails
    assert srv.timestamp == ts and ps.ps_pending(srv.h) == 0

    other = ps.ParameterServer(n, 0.01, 0.0, queue_depth=2, stream=stream)
    assert ps.ps_graph_launch(other.h, g2) == ps.PS_EINVAL
    null_stream = ps.ParameterServer(n, 0.01, 0.0, queue_depth=2)
    assert ps.ps_graph_create(null_stream.h, step)[0] == ps.PS_ESTATE
    side = torch.cuda.Stream()
    srv.set_pull_stream(side)
    assert ps.ps_graph_launch(srv.h, g2) == ps.PS_ESTATE
    assert ps.ps_graph_create(srv.h, step)[0] == ps.PS_ESTATE
    srv.sync()
    for gr in (graph, g2):
        ps.ps_graph_destroy(gr)
    for s_ in (other, null_stream, srv):
        s_.close()
