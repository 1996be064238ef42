"""A parameter server and its learners as separate processes on one GPU.

The layout of Sec. 4.1 and 4.3: every learner and the server has its own
address space; they share one region holding the gradient queues (lambda
single-producer single-consumer queues, a fixed number of slots each) and
the weights the learners read. Here the region is the server's own device
rows (ps_alloc_rows), shared with HIP IPC (ps_export_rows / ps_import_rows):
each learner gets `slots` gradient rows and one replica row. A Unix socket
per learner stands in for the paper's shared counters and condition
variables: a learner says which slot it filled (after its device write has
completed), the server says which slots it has consumed and the timestamp of
the weights it then wrote into the learner's replica. The server learns of a
learner's death when that socket closes without a goodbye, and then retires
it (its queued gradients still apply, Theorem 2) or drops it (they are
discarded), as the run's configuration says.

Usage: python tests/mp_ps.py server CONF.json
       python tests/mp_ps.py learner CONF.json L
CONF holds: sock, out (a directory), n, lr, momentum, learners, slots,
depth, pool, pushes (per learner), die ({learner: pushes before dying}),
dead_mode ("retire" | "drop"), and optionally workload ("alexnet": fp32
gradients, or "mixed": bf16), queue ("rr": per-learner queues of `slots`,
or "fifo": one queue of `depth`; the learners still own `slots` rows each),
push_offset (learner l's k-th push uses pool buffer (5 l + push_offset + k)
mod pool), and the restart of Sec. 4.3 in two runs: stop_after (after that
many applies the server stops taking pushes, tells the learners to stop and
waits until they have detached, applies what is queued, writes the
checkpoint `checkpoint` and exits -- the watchdog's restart point) and
resume (a checkpoint the server loads instead of starting from w0; the
learners are new processes).

The server writes out/server.json (every protocol call it made, in order:
push, apply with the learners served and their staleness, pull, retire or
drop with the count still queued) and out/w.npy, out/v.npy; each learner
that finishes writes out/learner<L>.json (the timestamp and sha256 of its
final replica). Test infrastructure: tests/test_gpu_multiprocess.py replays
the server's log through the oracle and compares.
"""
import collections
import hashlib
import json
import os
import selectors
import socket
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def say(*a):
    print(f"[mp_ps {os.getpid()}]", *a, flush=True)


def workload(conf):
    from paper_1611_06213_amd import workloads as wl
    return wl.CONFIGS[conf.get("workload", "alexnet")].scaled(conf["n"], pushes=sum(conf["pushes"]),
                                                             pool=conf["pool"])


def buffer_of(conf, learner, k):
    """Pool buffer of learner's k-th push."""
    return (5 * learner + conf.get("push_offset", 0) + k) % conf["pool"]


class Lines:
    """Newline-delimited JSON over a stream socket."""

    def __init__(self, sock):
        self.sock = sock
        self.buf = b""
        self.eof = False

    def send(self, obj):
        self.sock.sendall((json.dumps(obj) + "\n").encode())

    def feed(self):
        """Read what is there (the socket is readable); False at EOF."""
        try:
            data = self.sock.recv(1 << 16)
        except ConnectionResetError:
            data = b""
        if not data:
            self.eof = True
            return False
        self.buf += data
        return True

    def pop(self):
        if b"\n" not in self.buf:
            return None
        line, self.buf = self.buf.split(b"\n", 1)
        return json.loads(line)

    def pop_ready(self):
        """Whether a complete message is there, reading what the socket
        holds without blocking."""
        if b"\n" in self.buf:
            return True
        if not self.eof:
            import select
            while select.select([self.sock], [], [], 0)[0]:
                if not self.feed():
                    break
                if b"\n" in self.buf:
                    break
        return b"\n" in self.buf

    def recv(self):
        """Block for the next message; None at EOF."""
        while True:
            m = self.pop()
            if m is not None:
                return m
            if self.eof or not self.feed():
                return None


def check(rc, what):
    from paper_1611_06213_amd import ps
    if rc < 0:
        raise RuntimeError(f"{what}: [{rc}] {ps.ps_last_error()}")
    return rc


def server(conf):
    import numpy as np
    import torch

    from paper_1611_06213_amd import ps
    from paper_1611_06213_amd import workloads as wl

    torch.cuda.set_device(0)
    cfg = workload(conf)
    n, L, S, D = conf["n"], conf["learners"], conf["slots"], conf["depth"]
    stream = torch.cuda.current_stream()
    h = ps.ps_create(n, conf["lr"], conf["momentum"])
    check(ps.ps_set_stream(h, stream.cuda_stream), "set_stream")
    check(ps.ps_set_queue_depth(h, D), "set_queue_depth")
    if conf.get("queue", "rr") == "rr":
        check(ps.ps_set_queue_mode(h, ps.PS_QUEUE_ROUND_ROBIN, S), "set_queue_mode")
    gdt = cfg.grad_dtype
    fifo = conf.get("queue", "rr") == "fifo"
    log = []
    if conf.get("resume"):
        check(ps.ps_load(h, conf["resume"]), "load")
        log.append(["resume", ps.ps_timestamp(h)])
    else:
        w0 = wl.make_w0(cfg, "cuda")
        check(ps.ps_set_weights(h, w0.data_ptr()), "set_weights")
    slots, reps, offer = {}, {}, {}
    for l in range(L):
        rc, g = ps.ps_alloc_rows(h, S, gdt)
        check(rc, "alloc_rows")
        rc, r = ps.ps_alloc_rows(h, 1, ps.PS_F32)
        check(rc, "alloc_rows")
        rc, gh, goff = ps.ps_export_rows(h, g[0])
        check(rc, "export_rows")
        rc, rh, roff = ps.ps_export_rows(h, r[0])
        check(rc, "export_rows")
        slots[l], reps[l] = g, r[0]
        offer[l] = {"grad": gh.hex(), "goff": goff, "stride": (g[1] - g[0]) if S > 1 else 0,
                    "rep": rh.hex(), "roff": roff}
    torch.cuda.synchronize()

    lsock = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    lsock.bind(conf["sock"])
    lsock.listen(L)
    lsock.settimeout(60)
    conns = {}
    while len(conns) < L:
        c, _ = lsock.accept()
        ch = Lines(c)
        hello = ch.recv()
        l = hello["hello"]
        ch.send(offer[l])
        conns[l] = ch
    say(f"server: {L} learners attached")

    sel = selectors.DefaultSelector()
    for l, ch in conns.items():
        sel.register(ch.sock, selectors.EVENT_READ, l)
    queued = {l: collections.deque() for l in range(L)}   # slots waiting, oldest first
    live, done = set(range(L)), set()

    stopping = False

    def on_message(l, m):
        if "push" in m and stopping:
            return                         # after the stop decision: lost, as in a crash
        if "push" in m:
            s = m["push"]
            if fifo and check(ps.ps_pending(h), "pending") >= D:
                apply_and_pull()           # one queue of D: make room first
            check(ps.ps_push_dtype(h, l, slots[l][s], gdt), "push")
            queued[l].append(s)
            log.append(["push", l, s, m["buf"]])
        elif "done" in m:
            done.add(l)

    def on_eof(l):
        sel.unregister(conns[l].sock)
        if l in live and l not in done and not stopping:
            if conf["dead_mode"] == "retire":
                cnt = check(ps.ps_retire_learner(h, l), "retire_learner")
            else:
                cnt = check(ps.ps_drop_learner(h, l), "drop_learner")
                queued[l].clear()
            log.append([conf["dead_mode"], l, cnt])
            say(f"server: learner {l} died with {cnt} gradients queued ({conf['dead_mode']})")
        live.discard(l)

    def drain(timeout):
        got = False
        for key, _ in sel.select(timeout):
            l, ch = key.data, conns[key.data]
            if ch.feed():
                while (m := ch.pop()) is not None:
                    on_message(l, m)
                got = True
            else:
                while (m := ch.pop()) is not None:
                    on_message(l, m)
                on_eof(l)
                got = True
        return got

    def apply_and_pull():
        check(ps.ps_apply_pending(h), "apply_pending")
        ids, st = ps.ps_last_applied(h), ps.ps_last_staleness(h)
        log.append(["apply", ids, st])
        freed = collections.defaultdict(list)
        for l in ids:
            freed[l].append(queued[l].popleft())
        pull = [l for l in sorted(freed) if l in live]
        if pull:
            check(ps.ps_pull_many(h, pull, [reps[l] for l in pull], ps.PS_F32), "pull_many")
            log.append(["pull", pull])
        check(ps.ps_sync(h), "sync")          # slots consumed, replicas written
        ts = ps.ps_timestamp(h)
        for l in pull:
            try:
                conns[l].send({"free": freed[l], "ts": ts})
            except (BrokenPipeError, ConnectionResetError):
                pass                          # it died; its EOF is read next

    def stop_and_checkpoint():
        """The watchdog's restart point: no more pushes are taken, the
        learners are told to stop and detach (they release the shared rows
        before this process frees them), the queued gradients are applied
        and the checkpoint is written."""
        nonlocal stopping
        stopping = True
        for l in sorted(live):
            try:
                conns[l].send({"stop": 1})
            except (BrokenPipeError, ConnectionResetError):
                pass
        t_stop = time.monotonic() + 60
        while live:
            drain(0.5)
            if time.monotonic() > t_stop:
                raise RuntimeError("server: learners did not stop")
        while check(ps.ps_pending(h), "pending"):
            apply_and_pull()
        check(ps.ps_save(h, conf["checkpoint"]), "save")
        log.append(["checkpoint", ps.ps_timestamp(h)])
        with open(os.path.join(conf["out"], "server.json"), "w") as f:
            json.dump({"log": log, "ts": ps.ps_timestamp(h)}, f)
        ps.ps_destroy(h)
        lsock.close()
        say(f"server: checkpoint at ts {log[-1][1]}, stopping")
        return 0

    applies = 0
    t_end = time.monotonic() + conf.get("limit", 120)
    while time.monotonic() < t_end:
        if conf.get("stop_after") and applies >= conf["stop_after"]:
            return stop_and_checkpoint()
        got = drain(0.05)
        # everything already there or arriving within 2 ms (a learner that
        # stops right after a push closes its socket just after it), EOFs included
        while drain(0.002):
            got = True
        pending = check(ps.ps_pending(h), "pending")
        active = live - done
        if not active and pending == 0:
            break
        if pending >= D or (pending > 0 and (not got or not active)):
            apply_and_pull()
            applies += 1
    else:
        raise RuntimeError("server: run did not finish in time")

    final = sorted(live)
    if final:
        check(ps.ps_pull_many(h, final, [reps[l] for l in final], ps.PS_F32), "pull_many")
        log.append(["pull", final])
    check(ps.ps_sync(h), "sync")
    ts = ps.ps_timestamp(h)
    for l in final:
        try:
            conns[l].send({"bye": ts})
        except (BrokenPipeError, ConnectionResetError):
            pass
    while live:                      # wait for the finished learners to detach
        if not drain(1.0) and time.monotonic() > t_end:
            raise RuntimeError("server: learners did not detach")

    def host(ptr):
        t = torch.empty(n, dtype=torch.float32, device="cuda")
        import ctypes
        rc = ps._hip()(ctypes.c_void_p(t.data_ptr()), ctypes.c_void_p(ptr), ctypes.c_size_t(4 * n),
                       3, ctypes.c_void_p(stream.cuda_stream))
        assert rc == 0
        torch.cuda.synchronize()
        return t.cpu().numpy()

    out = conf["out"]
    np.save(os.path.join(out, "w.npy"), host(ps.ps_weights(h)))
    if ps.ps_velocity(h):
        np.save(os.path.join(out, "v.npy"), host(ps.ps_velocity(h)))
    with open(os.path.join(out, "server.json"), "w") as f:
        json.dump({"log": log, "ts": ts}, f)
    ps.ps_destroy(h)
    lsock.close()
    say(f"server: done at ts {ts}")
    return 0


def learner(conf, l):
    import torch

    from paper_1611_06213_amd import ps
    from paper_1611_06213_amd import workloads as wl

    torch.cuda.set_device(0)
    cfg = workload(conf)
    n, S = conf["n"], conf["slots"]
    c = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    t0 = time.monotonic()
    while True:
        try:
            c.connect(conf["sock"])
            break
        except (FileNotFoundError, ConnectionRefusedError):
            if time.monotonic() - t0 > 90:
                raise
            time.sleep(0.05)
    ch = Lines(c)
    ch.send({"hello": l})
    offer = ch.recv()
    if l == 0:   # the import refuses an offset outside the allocation, leaving nothing mapped
        bad, _ = ps.ps_import_rows(bytes.fromhex(offer["grad"]), 1 << 50)
        assert bad == ps.PS_EINVAL, bad
    rc, g0 = ps.ps_import_rows(bytes.fromhex(offer["grad"]), offer["goff"])
    check(rc, "import_rows")
    if l == 0:   # ... and a second import of a mapped row set; release wants a first row
        again, _ = ps.ps_import_rows(bytes.fromhex(offer["grad"]), offer["goff"])
        assert again == ps.PS_EINVAL, again
        assert ps.ps_release_rows(g0 + 16) == ps.PS_EINVAL
    rc, r0 = ps.ps_import_rows(bytes.fromhex(offer["rep"]), offer["roff"])
    check(rc, "import_rows")
    gtd = torch.bfloat16 if cfg.grad_dtype == wl.BF16 else torch.float32
    slot = ps.rows_as_tensors([g0 + i * offer["stride"] for i in range(S)], n, gtd)
    replica = ps.rows_as_tensors([r0], n, torch.float32)[0]
    free = collections.deque(range(S))
    die = conf["die"].get(str(l))
    grads = {}
    bye = None

    stop = False

    def handle(m):
        nonlocal bye, stop
        if m is None:
            raise RuntimeError(f"learner {l}: server went away")
        if "free" in m:
            free.extend(m["free"])
        elif "bye" in m:
            bye = m["bye"]
        elif "stop" in m:
            stop = True

    def detach(why):
        c.close()
        check(ps.ps_release_rows(g0), "release_rows")
        check(ps.ps_release_rows(r0), "release_rows")
        say(f"learner {l}: {why}")
        return 0

    for k in range(conf["pushes"][l]):
        while not free and not stop:
            handle(ch.recv())
        while ch.pop_ready():             # messages already there (a stop among them)
            handle(ch.pop())
        if stop:
            del slot, replica
            return detach(f"stopped by the server after {k} pushes")
        s = free.popleft()
        j = buffer_of(conf, l, k)
        if j not in grads:
            grads[j] = wl.make_grad(cfg, j, "cuda")
        slot[s].copy_(grads[j])
        torch.cuda.synchronize()           # the write is complete before the push
        ch.send({"push": s, "buf": j})
        if die is not None and k + 1 == die:
            del slot, replica              # dies here, gradients still queued
            return detach(f"stopping after {k + 1} pushes")
    ch.send({"done": 1})
    while bye is None and not stop:
        handle(ch.recv())
    if stop:
        del slot, replica
        return detach("stopped by the server after its last push")
    digest = hashlib.sha256(replica.cpu().numpy().tobytes()).hexdigest()
    with open(os.path.join(conf["out"], f"learner{l}.json"), "w") as f:
        json.dump({"ts": bye, "replica_sha256": digest}, f)
    del slot, replica
    check(ps.ps_release_rows(g0), "release_rows")
    check(ps.ps_release_rows(r0), "release_rows")
    c.close()
    say(f"learner {l}: finished at ts {bye}")
    return 0


def main(argv):
    with open(argv[2]) as f:
        conf = json.load(f)
    if argv[1] == "server":
        return server(conf)
    return learner(conf, int(argv[3]))


if __name__ == "__main__":
    sys.exit(main(sys.argv))
