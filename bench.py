"""Benchmark: gradient pushes applied per second on one MI355X.

Workload: the VGG-16-shaped parameter server (138,357,544 fp32 parameters,
13 conv + 3 fc tensors flat; lr 0.001, heavy-ball momentum 0.9; 16 learners
pushing Laplace(0, 1e-3) gradients in seeded random order; K = 32 gradients
folded per apply; after each apply all 16 learners pull fp32 replicas).
One step = 32 pushes + one apply + one 16-replica pull, i.e. one pass of the
whole hot path over one batch. Inputs (64 distinct gradient buffers, 35 GB)
are resident in HBM before timing starts. By default they and the replicas
are the server's own rows (ps_alloc_rows: the queue slots learners fill);
--layout torch puts every buffer in its own torch allocation instead.

Timing. After W warm-up steps, `runs` (default 5) timed runs of exactly K
steps each, w and v reset to w0 and 0 before every run (ps_set_weights);
each run is one ps_run call (the library's native executor walks the
prepared schedule of pushes, applies and pulls), bracketed by device
synchronisation, and `value` is the median run's pushes/s. The same runs are
timed again replaying the schedule captured once as a HIP graph
(ps_graph_create / ps_graph_launch: the host protocol still runs per call,
the kernels go out as one graph); with --graph `value` is the median of
those (launch-bound workloads gain, HBM-bound ones do not). One more run
drives the same calls one by one from Python (`python_driven_pushes_per_s`),
and a last one records HIP events around every kernel on the stream it runs
on, for the per-kernel durations behind `roofline` (events between kernels
cost a few microseconds each, which only the launch-bound workloads notice,
so they stay out of the runs that give `value`).

Prints one JSON line (rank 0, N = 1). Extra keys: the dominant kernel's
roofline (algorithmic bytes per launch / mean launch time), HBM traffic from
recorded rocprofv3 counters when the code they were taken on is unchanged,
reference rates of other implementations on this machine (torch's sum, the HIP
runtime's device copy, the library's own one-replica copy), and the oracle
timed on the host's cores on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_GBPS = 8000.0          # MI355X HBM3E, published
METRIC = "gradient pushes applied/sec + achieved HBM GB/s (% of peak), 1 MI355X"
CSRC = os.path.join(ROOT, "paper_1611_06213_amd", "csrc")
# the kernels and the host code that decides their launch shapes and the
# buffers' placement: recorded counters stay valid only while all are unchanged
KERNEL_SRC = [os.path.join(CSRC, f) for f in ("ps_kernels.hip", "ps_kernels.h", "ps_server.cpp",
                                              "ps_layout.cpp", "ps_layout.h")]
# counter summaries, one per measured kernel, workload and mode (the mode line names them)
COUNTERS = os.path.join(ROOT, "profiles", "traffic_*.txt")


def algorithmic_bytes(cfg, mode: str, r: int):
    """Bytes the method must move per step (one apply of K gradients + R
    replica writes): K gradient reads, w read+write, v read+write (momentum),
    R replica writes, plus one more read of w when the pull is its own
    kernel. Returns (per step, per dominant-kernel launch)."""
    from paper_1611_06213_amd import accounting as acc
    gb = 2 if cfg.grad_dtype == 1 else 4
    rb = 2 if cfg.pull_dtype == 1 else 4
    apply_b = acc.apply_bytes(cfg.n, cfg.depth, gb, cfg.momentum != 0)
    if mode == "fused":
        # one ps_apply_pull call: a single pass up to the fusion limit (one
        # replica), otherwise the apply kernel and the tiled pull; the events
        # bracket the whole call
        step = apply_b + acc.pull_bytes(cfg.n, r, rb, separate=r > 1)
        return step, step
    return apply_b + acc.pull_bytes(cfg.n, r, rb), apply_b


def batches(cfg, wl):
    """The schedule's full batches: (pushes [(learner, pool buffer)], learners
    that pull after that apply, deduplicated). A pull issued between two
    applies sees the weights of the earlier apply whatever its position, so
    it is attached to that apply. The final partial batch is left out."""
    out, pushes, last = [], [], None
    for ev in wl.schedule(cfg):
        if isinstance(ev, wl.Push):
            pushes.append((ev.learner, ev.buf))
        elif isinstance(ev, wl.Apply):
            last = (pushes, [])
            if len(pushes) == cfg.depth:
                out.append(last)
            pushes = []
        elif last is not None:
            for l in ev.learners:
                if l not in last[1]:
                    last[1].append(l)
    return out


def kernel_source_digest(paths=KERNEL_SRC) -> str:
    """sha256 over the kernel source and the host files that shape its
    launches and buffer placement, with comments and blank space removed, so
    that a comment-only edit keeps recorded counters valid and any code
    change invalidates them."""
    import re
    if isinstance(paths, str):
        paths = [paths]
    h = hashlib.sha256()
    for path in paths:
        text = open(path).read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode() + b"\0")
    return h.hexdigest()


def read_summary(path: str) -> dict:
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    return vals


def recorded_traffic(kernel_label: str, pattern: str = COUNTERS):
    """HBM bytes per launch of the apply from the committed counter summary
    of this workload and mode, or None when there is none or it was taken
    on different kernel code."""
    import glob
    digest = kernel_source_digest()
    for path in sorted(glob.glob(pattern)):
        vals = read_summary(path)
        if vals.get("mode") == kernel_label and vals.get("kernel_code_digest") == digest:
            try:
                return float(vals["hbm_bytes_per_launch"])
            except (KeyError, ValueError):
                return None
    return None


def cpu_baseline(cfg, pool, w0, pulls_per_step: int, seconds: float, distinct: int = 16):
    """The oracle, as it stands, on a bounded sample of the same workload:
    whole steps (K pushes, one apply, the step's pulls) over the full vector,
    single-threaded, repeated until `seconds` of CPU work have accumulated.
    The pushes cycle over `distinct` pool buffers copied to host memory (the
    values do not change the work)."""
    from oracle import server as orc

    import numpy as np
    import torch

    def host(t):
        t = t.cpu()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()

    distinct = min(distinct, cfg.pool)
    host_g = [host(pool[j]) for j in range(distinct)]
    s = orc.OracleServer(w0.cpu().numpy(), cfg.lr, cfg.momentum, depth=cfg.depth)
    j = steps = 0
    t0 = time.perf_counter()
    while True:
        for _ in range(cfg.depth):
            s.push(j % cfg.learners, host_g[j % distinct])
            j += 1
        s.apply_pending()
        for r in range(pulls_per_step):
            s.pull(r, r, cfg.pull_dtype)
        steps += 1
        t1 = time.perf_counter()
        if t1 - t0 >= seconds:
            break
    oracle_rate = steps * cfg.depth / (t1 - t0)
    from paper_1611_06213_amd import accounting as acc
    step_bytes = (acc.apply_bytes(cfg.n, cfg.depth, 2 if cfg.grad_dtype == 1 else 4, cfg.momentum != 0)
                  + acc.pull_bytes(cfg.n, pulls_per_step, 2 if cfg.pull_dtype == 1 else 4))
    oracle_sample = (f"{steps} whole steps ({cfg.depth} pushes + apply + {pulls_per_step} pulls) "
                     f"over the full {cfg.n:,}-parameter vector, 1 thread, pushes cycling over "
                     f"{distinct} host copies of pool buffers; {t1 - t0:.1f} s of CPU work on "
                     f"{cpu_model()} ({os.cpu_count()} logical CPUs visible)")
    paper = paper_style_ps(cfg, host_g, s.w, pulls_per_step, seconds / 2)
    del host_g
    return {
        "value": round(oracle_rate, 4), "unit": "pushes/s", "cores": 1, "kind": "oracle",
        # the same algorithmic bytes per step as the GPU line, over the oracle's time
        "gbps_algorithmic": round(steps * step_bytes / (t1 - t0) / 1e9, 3),
        "sample": oracle_sample,
        "paper_style_ps": paper,
    }


def paper_style_ps(cfg, host_g, w_start, pulls_per_step: int, seconds: float):
    """The paper's own CPU server design (oracle/cpu_ps.c: one OpenMP pass
    over the weights per gradient, loop unrolled 8x, Sec. 4.1 and 4.4) on all
    the host cores this process may use, over the same whole steps: context
    for what that design does on this host. Bitwise equal to the oracle."""
    import numpy as np
    from oracle import cpu_ps

    threads = len(os.sched_getaffinity(0))
    w = np.array(w_start, dtype=np.float32, copy=True)
    v = np.zeros_like(w) if cfg.momentum != 0 else None
    dst = [np.empty_like(w) for _ in range(2)]
    j = steps = 0
    t0 = time.perf_counter()
    while True:
        for _ in range(cfg.depth):
            cpu_ps.step(w, v, host_g[j % len(host_g)], cfg.lr, cfg.momentum, threads)
            j += 1
        for r in range(pulls_per_step):
            cpu_ps.pull(dst[r % 2], w, threads)
        steps += 1
        t1 = time.perf_counter()
        if t1 - t0 >= seconds:
            break
    return {
        "value": round(steps * cfg.depth / (t1 - t0), 4), "unit": "pushes/s", "cores": threads,
        "kind": "paper-style CPU parameter server (OpenMP, one pass per gradient)",
        "sample": (f"{steps} whole steps over the full vector, {threads} threads, "
                   f"{t1 - t0:.1f} s"),
    }


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def reference_rates(torch, ps, lib, n: int = 1 << 28, reps: int = 10):
    """GB/s of plain device streams over 1 GiB on this machine, for context: a
    read by torch's sum reduction, a copy by the HIP runtime
    (hipMemcpyAsync device to device), and the library's own one-replica pull
    (a 1-read/1-write copy)."""
    import ctypes
    stream = torch.cuda.current_stream()
    x = torch.empty(n, dtype=torch.float32, device="cuda").normal_()
    y = torch.empty_like(x)
    hip = ps._hip()

    def hip_copy():
        if hip(ctypes.c_void_p(y.data_ptr()), ctypes.c_void_p(x.data_ptr()),
               ctypes.c_size_t(4 * n), 3, ctypes.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipMemcpyAsync failed")

    def rate(fn, byt):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return byt / (e0.elapsed_time(e1) / reps * 1e-3) / 1e9

    out = {"torch_sum_read_gbps": round(rate(lambda: x.sum(), 4 * n), 1),
           "hip_memcpy_d2d_gbps": round(rate(hip_copy, 8 * n), 1),
           "library_copy_gbps": round(copy_ceiling(torch, ps, lib, n, reps), 1),
           "bytes": 4 * n}
    del x, y
    return out


def copy_ceiling(torch, ps, lib, n: int = 1 << 28, reps: int = 10):
    """The library's pull kernel with a single fp32 replica is a plain
    1-read/1-write device copy."""
    h = ps.ps_create(n, 0.0, 0.0)
    stream = torch.cuda.current_stream()
    ps.ps_set_stream(h, stream.cuda_stream)
    ps.ps_set_pull_skip(h, False)
    dst = torch.empty(n, dtype=torch.float32, device="cuda")
    ids, dp = ps._ints([0]), ps._ptrs([dst.data_ptr()])
    lib.ps_pull_many(h, 1, ids, dp, 0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        lib.ps_pull_many(h, 1, ids, dp, 0)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    ps.ps_destroy(h)
    del dst
    return 8 * n / (ms * 1e-3) / 1e9


class HipEvents:
    """Timing events recorded with the HIP runtime the library is bound to.

    The same HIP events torch.cuda.Event wraps, recorded through ctypes: a
    record costs about a microsecond of host time instead of several, which
    matters for the launch-bound workloads (Tiny), where the host loop
    otherwise sets the pace."""

    def __init__(self, lib, count: int):
        import ctypes
        self._c = ctypes
        self._rec = lib.hipEventRecord
        self._rec.restype = ctypes.c_int
        self._rec.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self._elapsed = lib.hipEventElapsedTime
        self._elapsed.restype = ctypes.c_int
        self._elapsed.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self._destroy = lib.hipEventDestroy
        self._destroy.restype = ctypes.c_int
        self._destroy.argtypes = [ctypes.c_void_p]
        create = lib.hipEventCreate
        create.restype = ctypes.c_int
        create.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.ev = []
        for _ in range(count):
            e = ctypes.c_void_p()
            if create(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.ev.append(e.value)

    def record(self, i: int, stream_ptr: int) -> None:
        if self._rec(self.ev[i], stream_ptr) != 0:
            raise RuntimeError("hipEventRecord failed")

    def ms(self, i: int, j: int) -> float:
        out = self._c.c_float()
        if self._elapsed(self._c.byref(out), self.ev[i], self.ev[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return out.value

    def close(self) -> None:
        for e in self.ev:
            self._destroy(e)
        self.ev = []


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--runs", type=int, default=5,
                    help="timed runs of --steps steps each, w and v reset before each; "
                         "value is the median run")
    ap.add_argument("--graph", action="store_true",
                    help="value from runs that replay the prepared steps captured once as a HIP "
                         "graph (ps_graph_launch) instead of one ps_run call; both rates are "
                         "reported either way")
    ap.add_argument("--config", default="vgg16")
    ap.add_argument("--mode", choices=["fused", "separate", "hogwild"], default="separate",
                    help="separate: ps_apply_pending + ps_pull_many (one kernel each, timed "
                         "apart); fused: ps_apply_pull (the same kernels above one replica); "
                         "hogwild: pulls lock-free on a second stream, overlapping the next "
                         "apply (Sec. 4.1)")
    ap.add_argument("--apply", choices=["asgd", "sync"], default="asgd",
                    help="asgd: the workload's K-gradient asynchronous applies; sync: one "
                         "synchronous step (Eq. ssgd) per step over one gradient per learner")
    ap.add_argument("--layout", choices=["server", "torch"], default="server",
                    help="server: gradient pool and replicas in the server's own rows "
                         "(ps_alloc_rows, distinct offsets within 2 MiB); torch: each "
                         "buffer its own torch allocation, as plain user code would make them")
    ap.add_argument("--queue", choices=["fifo", "rr"], default="fifo",
                    help="fifo: one queue of K slots; rr: a queue per learner served "
                         "round-robin, one gradient per visit (Sec. 4.1), K slots each")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a plain 1 GiB copy (known bytes) for counter calibration")
    args = ap.parse_args()

    if args.apply == "sync" and args.mode != "separate":
        ap.error("--apply sync runs apply and pull as separate calls (--mode separate)")
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the parameter server here runs on a single "
              "MI355X; multi-GPU sharding is a design note, not built.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1611_06213_amd import ps
    from paper_1611_06213_amd import workloads as wl
    from paper_1611_06213_amd.accounting import learner_ps_bytes_per_push
    from paper_1611_06213_amd.accounting import pull_bytes as pull_bytes_of

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    lib = ps.load_library()
    cfg = wl.CONFIGS[args.config]
    if args.apply == "sync":
        # one gradient per learner per step; every learner pulls after it
        cfg = wl.dataclasses.replace(cfg, depth=cfg.learners)
    n, K, R = cfg.n, cfg.depth, cfg.replicas
    # a stream of its own (default priority), current for torch's work too:
    # the legacy null stream cannot be captured into a graph
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)

    h = ps.ps_create(n, cfg.lr, cfg.momentum)
    if not h:
        raise RuntimeError(ps.ps_last_error())
    gdt_t = torch.bfloat16 if cfg.grad_dtype == wl.BF16 else torch.float32
    rdt = torch.bfloat16 if cfg.pull_dtype == wl.BF16 else torch.float32
    if args.layout == "server":
        rc, gp = ps.ps_alloc_rows(h, cfg.pool, cfg.grad_dtype)
        rc2, rp = ps.ps_alloc_rows(h, R, cfg.pull_dtype)
        if rc or rc2:
            raise RuntimeError(ps.ps_last_error())
        pool = ps.rows_as_tensors(gp, n, gdt_t)
        replicas = ps.rows_as_tensors(rp, n, rdt)
    else:
        pool = [torch.empty(n, dtype=gdt_t, device="cuda") for _ in range(cfg.pool)]
        replicas = [torch.empty(n, dtype=rdt, device="cuda") for _ in range(R)]
    for j in range(cfg.pool):
        pool[j].copy_(wl.make_grad(cfg, j, "cuda"))
    w0 = wl.make_w0(cfg, "cuda")
    if args.apply == "sync":
        plan = [([(l, (s * cfg.learners + l) % cfg.pool) for l in range(cfg.learners)],
                 list(range(cfg.replicas))) for s in range(cfg.pool)]
    else:
        plan = batches(cfg, wl)
    torch.cuda.synchronize()

    assert ps.ps_set_queue_depth(h, K) == 0
    if args.queue == "rr":
        assert ps.ps_set_queue_mode(h, ps.PS_QUEUE_ROUND_ROBIN, K) == 0
    assert ps.ps_set_stream(h, stream.cuda_stream) == 0
    assert ps.ps_set_weights(h, w0.data_ptr()) == 0

    pstream = None
    if args.mode == "hogwild":
        pstream = torch.cuda.Stream(device=stream.device)     # default priority
        assert ps.ps_set_pull_stream(h, pstream.cuda_stream) == 0

    gptr = [pool[j].data_ptr() for j in range(cfg.pool)]
    calls = []
    for pushes_b, pulls_b in plan:
        dl = [replicas[l].data_ptr() for l in pulls_b]
        calls.append(([(l, gptr[b]) for l, b in pushes_b], len(pulls_b), ps._ints(pulls_b or [0]),
                      ps._ptrs(dl or [0]), list(pulls_b), dl))
    pdt = cfg.pull_dtype
    gdt = cfg.grad_dtype
    push = lib.ps_push_dtype
    it = 0

    sptr = stream.cuda_stream
    pptr = pstream.cuda_stream if pstream is not None else sptr

    def script(steps: int):
        """The calls of `steps` steps from the start of the plan, for ps_run."""
        sc = ps.OpScript()
        for i in range(steps):
            pushes_b, r, _, _, ids, dl = calls[i % len(calls)]
            for l, g in pushes_b:
                sc.push(l, g, gdt)
            if args.mode == "fused":
                sc.apply_pull(ids, dl, pdt)
            else:
                sc.apply_sync() if args.apply == "sync" else sc.apply()
                sc.pull(ids, dl, pdt)
        return sc.build()

    # events of step s: 4s = before the apply, 4s+1 = after it (both on the
    # library's stream), 4s+2 / 4s+3 = around the pull on the stream it runs
    # on (with ordered pulls the same point as 4s+1, so 4s+1 serves as both)
    def step(s_=None):
        nonlocal it
        pushes_b, r, ids, dptr, _, _ = calls[it % len(calls)]
        it += 1
        for l, g in pushes_b:
            if push(h, l, g, gdt) != 0:
                raise RuntimeError(ps.ps_last_error())
        if s_ is not None:
            evs.record(4 * s_, sptr)
        if args.mode == "fused":
            rc = lib.ps_apply_pull(h, r, ids, dptr, pdt)
            if s_ is not None:
                evs.record(4 * s_ + 1, sptr)
        else:
            rc = lib.ps_apply_sync(h) if args.apply == "sync" else lib.ps_apply_pending(h)
            if s_ is not None:
                evs.record(4 * s_ + 1, sptr)
                if pstream is not None:
                    evs.record(4 * s_ + 2, pptr)
            rc = rc or lib.ps_pull_many(h, r, ids, dptr, pdt)
            if s_ is not None:
                evs.record(4 * s_ + 3, pptr)
        if rc != 0:
            raise RuntimeError(ps.ps_last_error())
        return r

    def reset():
        """w := w0, v := 0, timestamp and learner history cleared; the plan
        restarts at its first step."""
        nonlocal it
        if ps.ps_set_weights(h, w0.data_ptr()) != 0:
            raise RuntimeError(ps.ps_last_error())
        it = 0
        torch.cuda.synchronize()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # value: median of `runs` runs of exactly K steps, each one native call
    timed = script(args.steps)
    rs = [calls[i % len(calls)][1] for i in range(args.steps)]
    run_s = []
    for _ in range(args.runs):
        reset()
        t0 = time.perf_counter()
        rc, done = ps.ps_run(h, timed)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        if rc != 0 or done != len(timed):
            raise RuntimeError(f"ps_run stopped at call {done}: {ps.ps_last_error()}")
        run_s.append(t1 - t0)

    # the same steps as HIP graph replays (ordered pulls only): one cycle of
    # the plan captured once and enqueued back to back (the host plans replay
    # i + 1 while the device runs replay i), the steps left over as a second
    # graph
    graph_s = []
    graph_note = None
    if pstream is None:
        cycle = len(calls)
        q, rem = divmod(args.steps, cycle)
        graphs = []
        for steps_, count in ((cycle, q), (rem, 1 if rem else 0)):
            if count == 0:
                continue
            reset()
            rc, g_ = ps.ps_graph_create(h, script(steps_))
            if rc != 0:
                raise RuntimeError(f"ps_graph_create: {ps.ps_last_error()}")
            graphs.append((g_, count))
        for _ in range(args.runs):
            reset()
            t0 = time.perf_counter()
            rc = 0
            for g_, count in graphs:
                for _ in range(count):
                    rc = rc or ps.ps_graph_launch(h, g_)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            if rc == ps.PS_ESTATE and not args.graph:
                # the plan changes from cycle to cycle (round-robin service
                # order): the replay refuses, and there is no graph rate
                graph_note = ps.ps_last_error()
                graph_s = []
                break
            if rc != 0:
                raise RuntimeError(f"ps_graph_launch: {ps.ps_last_error()}")
            graph_s.append(t1 - t0)
        for g_, _ in graphs:
            ps.ps_graph_destroy(g_)
    elif args.graph:
        raise SystemExit("--graph needs ordered pulls (not --mode hogwild)")
    value_s = graph_s if args.graph else run_s
    elapsed = sorted(value_s)[len(value_s) // 2]

    # the same steps driven call by call from Python
    reset()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    py_elapsed = time.perf_counter() - t0

    # per-kernel durations: events around every kernel, on its stream
    reset()
    evs = HipEvents(lib, 4 * args.steps)
    for s_ in range(args.steps):
        step(s_)
    torch.cuda.synchronize()

    pushes = K * args.steps
    step_bytes = sum(algorithmic_bytes(cfg, args.mode, r)[0] for r in rs)
    launch_bytes = sum(algorithmic_bytes(cfg, args.mode, r)[1] for r in rs) / args.steps
    k_each = sorted(evs.ms(4 * s_, 4 * s_ + 1) for s_ in range(args.steps))
    k_ms = sum(k_each) / args.steps
    p0 = 2 if pstream is not None else 1
    p_each = (sorted(evs.ms(4 * s_ + p0, 4 * s_ + 3) for s_ in range(args.steps))
              if args.mode != "fused" else [0.0])
    p_ms = sum(p_each) / len(p_each)
    evs.close()
    gbps = step_bytes / elapsed / 1e9
    achieved = launch_bytes / (k_ms * 1e-3) / 1e9
    label = (f"{args.config}-{args.mode}" + ("-sync" if args.apply == "sync" else "")
             + ("-torch-buffers" if args.layout == "torch" else "")
             + ("-rr" if args.queue == "rr" else ""))
    traffic = recorded_traffic(label)

    if args.calib_copy:
        a = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(2.0)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    ts = ps.ps_timestamp(h)
    refs = reference_rates(torch, ps, lib)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, pool, w0, round(sum(rs) / len(rs)), args.cpu_seconds)
    del pool, replicas            # views of the server's rows (server layout)
    ps.ps_destroy(h)

    kern = ("ps_apply_pull (apply + pull kernels)" if args.mode == "fused"
            else "sync_vec (synchronous step)" if args.apply == "sync"
            else "apply_vec (fused K-gradient apply)")
    pull_bytes = sum(pull_bytes_of(n, r, 2 if pdt == wl.BF16 else 4) for r in rs) / args.steps
    out = {
        "metric": METRIC,
        "value": round(pushes / elapsed, 2),
        "unit": "pushes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "timing": {
            "runs": args.runs,
            "pushes_per_s_each_run": [round(pushes / t, 2) for t in value_s],
            "value_is": ("median run; each run " + ("the prepared steps as HIP graph replays "
                         "(one cycle of the plan captured once, replayed back to back with "
                         "ps_graph_launch)" if args.graph else "one ps_run call over the "
                         "prepared steps") + ", after ps_set_weights(w0) reset w, v and the "
                         "timestamp"),
            "ps_run_pushes_per_s": round(pushes / sorted(run_s)[len(run_s) // 2], 2),
            "graph_pushes_per_s": (round(pushes / sorted(graph_s)[len(graph_s) // 2], 2)
                                   if graph_s else None),
            "graph_not_replayable": graph_note,
            "python_driven_pushes_per_s": round(pushes / py_elapsed, 2),
        },
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if cfg.grad_dtype == wl.F32 else "bf16-grad/f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{cfg.name}: {n:,} fp32 params, K={K} pushes per apply, "
                         f"R={max(rs)} {'fp32' if pdt == wl.F32 else 'bf16'} replicas per apply, "
                         f"lr={cfg.lr}, momentum={cfg.momentum}, {cfg.learners} learners, "
                         f"{args.mode} apply+pull"),
            "params": n, "queue_depth": K, "replicas_per_apply": round(sum(rs) / len(rs), 2),
            "mode": args.mode, "apply": args.apply, "queue": args.queue,
            "layout": ("server rows (ps_alloc_rows)" if args.layout == "server"
                       else "separate torch allocations"),
        },
        "gbps": round(gbps, 1),
        "pct_peak": round(100 * gbps / PEAK_GBPS, 2),
        # the paper's accounting (2 x fp32 model per push, Sec. 3), comparable to
        # its Table "bandwidth_utilized"; not an HBM figure
        "learner_ps_gbps_paper_accounting": round(
            pushes / elapsed * learner_ps_bytes_per_push(n) / 1e9, 1),
        "bytes_per_step": round(step_bytes / args.steps),
        # kernel time summed over both streams (with hogwild the two overlap)
        "pushes_per_s_device": round(pushes / ((k_ms + p_ms) * args.steps * 1e-3), 2),
        "kernel_ms": {"apply": round(k_ms, 4), **({"pull": round(p_ms, 4)} if p_ms else {})},
        "kernel_ms_median": {"apply": round(k_each[len(k_each) // 2], 4),
                             **({"pull": round(p_each[len(p_each) // 2], 4)} if p_ms else {})},
        **({"pull_kernel_gbps": round(pull_bytes / (p_ms * 1e-3) / 1e9, 1)} if p_ms else {}),
        "roofline": {
            "bound": "hbm", "kernel": kern,
            "achieved": round(achieved, 1), "peak": PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / PEAK_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": round(launch_bytes),
        },
        "reference_rates": refs,
        "apply_vs_reference": {
            "of_8tbps_peak": round(achieved / PEAK_GBPS, 4),
            "of_torch_sum_read": round(achieved / refs["torch_sum_read_gbps"], 4),
            "of_hip_memcpy_d2d": round(achieved / refs["hip_memcpy_d2d_gbps"], 4),
            "of_library_copy": round(achieved / refs["library_copy_gbps"], 4),
        },
        "cpu_baseline": cpu,
        "timestamp_after": ts,
    }
    state_mb = n * (8 if cfg.momentum != 0 else 4) / 1e6
    if state_mb <= 256:
        # small workloads: the weights stay in the memory-side cache between
        # steps, and tiny steps are paced by launches, not by bandwidth
        out["roofline"]["note"] = (
            f"w{' and v' if cfg.momentum != 0 else ''} ({state_mb:.0f} MB) fit the 256 MB "
            "memory-side cache, so part of the traffic is served from it: GB/s is effective, "
            "not HBM-only" + ("; steps this small are launch-latency bound"
                              if step_bytes / args.steps < 64e6 else ""))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
