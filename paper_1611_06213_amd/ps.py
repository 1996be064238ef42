"""ctypes binding of libgadeips.so (the C ABI in include/ps.h).

Module-level functions carry the C names and return the C status codes;
they only marshal arguments. `ParameterServer` wraps a handle for torch
device tensors and raises `PSError` on failure. Every computation runs in the
library's HIP kernels; if the library is not built, loading raises.
"""
from __future__ import annotations

import ctypes
import os
import threading
from collections import deque
from typing import Optional, Sequence

PS_OK = 0
PS_EINVAL = -1
PS_EFULL = -2
PS_ENOMEM = -3
PS_EHIP = -4
PS_ESTATE = -5
PS_EIO = -6

PS_F32 = 0
PS_BF16 = 1

PS_QUEUE_FIFO = 0
PS_QUEUE_ROUND_ROBIN = 1

PS_MAX_QUEUE_DEPTH = 64
PS_MAX_REPLICAS = 64
PS_MAX_LEARNERS = 65536
PS_STALENESS_BINS = 64
PS_MAX_ROWS = 4096
PS_IPC_HANDLE_BYTES = 64

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgadeips.so")

_u64 = ctypes.c_uint64


class ps_stats(ctypes.Structure):
    _fields_ = [
        ("timestamp", _u64), ("pushes_accepted", _u64), ("pushes_rejected", _u64),
        ("pushes_applied", _u64), ("pushes_dropped", _u64), ("applies", _u64), ("pulls", _u64),
        ("pulls_skipped", _u64),
        ("staleness_max", _u64), ("staleness_sum", _u64),
        ("staleness_hist", _u64 * PS_STALENESS_BINS),
    ]


PS_OP_PUSH = 0
PS_OP_APPLY = 1
PS_OP_APPLY_SYNC = 2
PS_OP_PULL = 3
PS_OP_APPLY_PULL = 4


class ps_op(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int), ("learner_id", ctypes.c_int), ("dtype", ctypes.c_int),
        ("count", ctypes.c_int), ("grad", ctypes.c_void_p),
        ("learner_ids", ctypes.POINTER(ctypes.c_int)), ("dsts", ctypes.POINTER(ctypes.c_void_p)),
    ]


# name -> (restype, argtypes); the same list the header declares
_VP = ctypes.c_void_p
_SIGS = {
    "ps_create": (_VP, [ctypes.c_size_t, ctypes.c_float, ctypes.c_float]),
    "ps_destroy": (None, [_VP]),
    "ps_push": (ctypes.c_int, [_VP, ctypes.c_int, _VP]),
    "ps_push_dtype": (ctypes.c_int, [_VP, ctypes.c_int, _VP, ctypes.c_int]),
    "ps_push_async": (ctypes.c_int, [_VP, ctypes.c_int, _VP, ctypes.c_int, _VP]),
    "ps_record": (ctypes.c_int, [_VP, _VP]),
    "ps_set_pull_stream": (ctypes.c_int, [_VP, _VP]),
    "ps_apply_pending": (ctypes.c_int, [_VP]),
    "ps_apply_sync": (ctypes.c_int, [_VP]),
    "ps_pull": (ctypes.c_int, [_VP, ctypes.c_int, _VP]),
    "ps_pull_many": (ctypes.c_int, [_VP, ctypes.c_int, ctypes.POINTER(ctypes.c_int),
                                    ctypes.POINTER(_VP), ctypes.c_int]),
    "ps_apply_pull": (ctypes.c_int, [_VP, ctypes.c_int, ctypes.POINTER(ctypes.c_int),
                                     ctypes.POINTER(_VP), ctypes.c_int]),
    "ps_set_stream": (ctypes.c_int, [_VP, _VP]),
    "ps_set_queue_depth": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ps_set_pull_skip": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ps_set_fronts": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ps_set_launch_shape": (ctypes.c_int, [_VP, ctypes.c_int, ctypes.c_int]),
    "ps_set_queue_mode": (ctypes.c_int, [_VP, ctypes.c_int, ctypes.c_int]),
    "ps_last_applied": (ctypes.c_int, [_VP, ctypes.POINTER(ctypes.c_int), ctypes.c_int]),
    "ps_set_pull_fusion": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ps_set_weights": (ctypes.c_int, [_VP, _VP]),
    "ps_weights": (_VP, [_VP]),
    "ps_velocity": (_VP, [_VP]),
    "ps_num_params": (ctypes.c_size_t, [_VP]),
    "ps_timestamp": (_u64, [_VP]),
    "ps_pending": (ctypes.c_int, [_VP]),
    "ps_last_staleness": (ctypes.c_int, [_VP, ctypes.POINTER(ctypes.c_int64), ctypes.c_int]),
    "ps_drop_learner": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ps_retire_learner": (ctypes.c_int, [_VP, ctypes.c_int]),
    "ps_export_rows": (ctypes.c_int, [_VP, _VP, _VP, ctypes.POINTER(ctypes.c_size_t)]),
    "ps_import_rows": (ctypes.c_int, [_VP, ctypes.c_size_t, ctypes.POINTER(_VP)]),
    "ps_release_rows": (ctypes.c_int, [_VP]),
    "ps_save": (ctypes.c_int, [_VP, ctypes.c_char_p]),
    "ps_load": (ctypes.c_int, [_VP, ctypes.c_char_p]),
    "ps_sync": (ctypes.c_int, [_VP]),
    "ps_run": (ctypes.c_int, [_VP, ctypes.POINTER(ps_op), ctypes.c_int,
                              ctypes.POINTER(ctypes.c_int)]),
    "ps_graph_create": (ctypes.c_int, [_VP, ctypes.POINTER(ps_op), ctypes.c_int,
                                       ctypes.POINTER(_VP)]),
    "ps_graph_launch": (ctypes.c_int, [_VP, _VP]),
    "ps_graph_destroy": (None, [_VP]),
    "ps_get_stats": (ctypes.c_int, [_VP, ctypes.POINTER(ps_stats)]),
    "ps_alloc_rows": (ctypes.c_int, [_VP, ctypes.c_int, ctypes.c_int, ctypes.POINTER(_VP)]),
    "ps_free_rows": (ctypes.c_int, [_VP, _VP]),
    "ps_last_error": (ctypes.c_char_p, []),
}

_lib = None


def load_library(path: Optional[str] = None):
    """Load the built library (once). Raises if it is missing."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(
            f"{p} is not built: run `python -c 'import __graft_entry__ as g; g.build()'` "
            "(the parameter server has no CPU fallback)")
    # torch bundles its own HIP runtime. Loading torch first makes the
    # library bind to that one (same soname); loading the library first would
    # put a second HIP runtime in the process, and torch's streams and
    # allocations would not be valid in it.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    L = ctypes.CDLL(p)
    for name, (res, args) in _SIGS.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    if path is None:
        _lib = L
    return L


class PSError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


def _ints(xs: Sequence[int]):
    return (ctypes.c_int * max(1, len(xs)))(*xs)


def _ptrs(xs: Sequence[int]):
    return (_VP * max(1, len(xs)))(*xs)


# ------------------------------------------------------------ C-named calls

def ps_last_error() -> str:
    return load_library().ps_last_error().decode()


def ps_create(n_params: int, lr: float, momentum: float) -> int:
    h = load_library().ps_create(n_params, lr, momentum)
    if not h:
        raise PSError(PS_EINVAL, ps_last_error())
    return h


def ps_destroy(h: int) -> None:
    load_library().ps_destroy(h)


def ps_push(h: int, learner_id: int, grad_ptr: int) -> int:
    return load_library().ps_push(h, learner_id, grad_ptr)


def ps_push_dtype(h: int, learner_id: int, grad_ptr: int, dtype: int) -> int:
    return load_library().ps_push_dtype(h, learner_id, grad_ptr, dtype)


def ps_push_async(h: int, learner_id: int, grad_ptr: int, dtype: int, ready_event: int) -> int:
    return load_library().ps_push_async(h, learner_id, grad_ptr, dtype, ready_event)


def ps_record(h: int, event: int) -> int:
    return load_library().ps_record(h, event)


def ps_set_pull_stream(h: int, stream_ptr: int) -> int:
    return load_library().ps_set_pull_stream(h, stream_ptr)


def ps_apply_pending(h: int) -> int:
    return load_library().ps_apply_pending(h)


def ps_apply_sync(h: int) -> int:
    return load_library().ps_apply_sync(h)


def ps_pull(h: int, learner_id: int, dst_ptr: int) -> int:
    return load_library().ps_pull(h, learner_id, dst_ptr)


def ps_pull_many(h: int, learner_ids: Sequence[int], dst_ptrs: Sequence[int], dst_dtype: int) -> int:
    return load_library().ps_pull_many(h, len(learner_ids), _ints(learner_ids), _ptrs(dst_ptrs),
                                       dst_dtype)


def ps_apply_pull(h: int, learner_ids: Sequence[int], dst_ptrs: Sequence[int], dst_dtype: int) -> int:
    return load_library().ps_apply_pull(h, len(learner_ids), _ints(learner_ids), _ptrs(dst_ptrs),
                                        dst_dtype)


def ps_set_stream(h: int, stream_ptr: int) -> int:
    return load_library().ps_set_stream(h, stream_ptr)


def ps_set_queue_depth(h: int, depth: int) -> int:
    return load_library().ps_set_queue_depth(h, depth)


def ps_set_pull_skip(h: int, enabled: bool) -> int:
    return load_library().ps_set_pull_skip(h, 1 if enabled else 0)


def ps_set_queue_mode(h: int, mode: int, slots_per_learner: int = 1) -> int:
    return load_library().ps_set_queue_mode(h, mode, slots_per_learner)


def ps_last_applied(h: int, cap: int = PS_MAX_QUEUE_DEPTH):
    out = (ctypes.c_int * cap)()
    n = load_library().ps_last_applied(h, out, cap)
    if n < 0:
        return n
    return [int(out[i]) for i in range(min(n, cap))]


def ps_set_pull_fusion(h: int, max_replicas: int) -> int:
    return load_library().ps_set_pull_fusion(h, max_replicas)


def ps_set_weights(h: int, src_ptr: int) -> int:
    return load_library().ps_set_weights(h, src_ptr)


def ps_weights(h: int) -> int:
    return load_library().ps_weights(h) or 0


def ps_velocity(h: int) -> int:
    return load_library().ps_velocity(h) or 0


def ps_num_params(h: int) -> int:
    return load_library().ps_num_params(h)


def ps_timestamp(h: int) -> int:
    return load_library().ps_timestamp(h)


def ps_pending(h: int) -> int:
    return load_library().ps_pending(h)


def ps_last_staleness(h: int, cap: int = PS_MAX_QUEUE_DEPTH):
    out = (ctypes.c_int64 * cap)()
    n = load_library().ps_last_staleness(h, out, cap)
    if n < 0:
        return n
    return [int(out[i]) for i in range(min(n, cap))]


def ps_drop_learner(h: int, learner_id: int) -> int:
    return load_library().ps_drop_learner(h, learner_id)


def ps_retire_learner(h: int, learner_id: int) -> int:
    return load_library().ps_retire_learner(h, learner_id)


def ps_export_rows(h: int, first_row: int):
    """(status, handle bytes, offset of the first row in the allocation)."""
    buf = ctypes.create_string_buffer(PS_IPC_HANDLE_BYTES)
    off = ctypes.c_size_t()
    rc = load_library().ps_export_rows(h, first_row, buf, ctypes.byref(off))
    return rc, (buf.raw if rc == PS_OK else b""), off.value


def ps_import_rows(handle: bytes, offset: int):
    """(status, address of the first row mapped into this process)."""
    if len(handle) != PS_IPC_HANDLE_BYTES:
        return PS_EINVAL, 0
    out = _VP()
    rc = load_library().ps_import_rows(handle, offset, ctypes.byref(out))
    return rc, (out.value or 0)


def ps_release_rows(first_row: int) -> int:
    return load_library().ps_release_rows(first_row)


def ps_save(h: int, path: str) -> int:
    return load_library().ps_save(h, os.fsencode(path))


def ps_load(h: int, path: str) -> int:
    return load_library().ps_load(h, os.fsencode(path))


def ps_sync(h: int) -> int:
    return load_library().ps_sync(h)


class OpScript:
    """A prepared ps_run script: a ctypes ps_op array plus the id and
    pointer arrays its pull ops point into (kept alive here)."""

    def __init__(self):
        self._ops = []
        self._keep = []
        self.array = None

    def push(self, learner_id: int, grad_ptr: int, dtype: int = PS_F32):
        self._ops.append(ps_op(PS_OP_PUSH, learner_id, dtype, 0, grad_ptr, None, None))

    def apply(self):
        self._ops.append(ps_op(PS_OP_APPLY, 0, 0, 0, None, None, None))

    def apply_sync(self):
        self._ops.append(ps_op(PS_OP_APPLY_SYNC, 0, 0, 0, None, None, None))

    def _pulls(self, kind, learner_ids, dst_ptrs, dtype):
        ids, dp = _ints(learner_ids), _ptrs(dst_ptrs)
        self._keep += [ids, dp]
        self._ops.append(ps_op(kind, 0, dtype, len(learner_ids), None,
                               ctypes.cast(ids, ctypes.POINTER(ctypes.c_int)),
                               ctypes.cast(dp, ctypes.POINTER(_VP))))

    def pull(self, learner_ids, dst_ptrs, dtype: int = PS_F32):
        self._pulls(PS_OP_PULL, learner_ids, dst_ptrs, dtype)

    def apply_pull(self, learner_ids, dst_ptrs, dtype: int = PS_F32):
        self._pulls(PS_OP_APPLY_PULL, learner_ids, dst_ptrs, dtype)

    def __len__(self):
        return len(self._ops)

    def build(self):
        self.array = (ps_op * max(1, len(self._ops)))(*self._ops)
        return self


def ps_run(h: int, script: "OpScript"):
    """(status, calls completed)."""
    if script.array is None:
        script.build()
    done = ctypes.c_int()
    rc = load_library().ps_run(h, script.array, len(script), ctypes.byref(done))
    return rc, done.value


def ps_graph_create(h: int, script: "OpScript"):
    """(status, graph handle): the script captured as a HIP graph (nothing
    runs; ps_graph_launch replays it). The script's buffers must outlive the
    graph."""
    if script.array is None:
        script.build()
    out = _VP()
    rc = load_library().ps_graph_create(h, script.array, len(script), ctypes.byref(out))
    return rc, (out.value or 0)


def ps_graph_launch(h: int, graph: int) -> int:
    return load_library().ps_graph_launch(h, graph)


def ps_graph_destroy(graph: int) -> None:
    load_library().ps_graph_destroy(graph)


def ps_set_fronts(h: int, fronts_log2: int) -> int:
    return load_library().ps_set_fronts(h, fronts_log2)


def ps_set_launch_shape(h: int, blocks_per_cu: int, group: int) -> int:
    return load_library().ps_set_launch_shape(h, blocks_per_cu, group)


def ps_alloc_rows(h: int, count: int, dtype: int):
    """(status, [row addresses])."""
    out = (_VP * max(1, count))()
    rc = load_library().ps_alloc_rows(h, count, dtype, out)
    return rc, ([int(out[i]) for i in range(count)] if rc == PS_OK else [])


def ps_free_rows(h: int, first_row: int) -> int:
    return load_library().ps_free_rows(h, first_row)


def ps_get_stats(h: int):
    s = ps_stats()
    rc = load_library().ps_get_stats(h, ctypes.byref(s))
    return rc if rc < 0 else s


# ------------------------------------------------------------ tensor wrapper

def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return PS_F32
    if t.dtype == torch.bfloat16:
        return PS_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


class ParameterServer:
    """A server handle for torch device tensors.

    Pushed gradients are borrowed: the tensor is kept referenced until the
    apply that consumes it has been enqueued, and the caller must not write it
    before that apply has run on the server's stream. An apply may leave
    gradients queued (round-robin mode takes at most `depth`, a synchronous
    step one per waiting learner); those stay referenced. Gradients and
    replicas are marked as used on the torch streams given to set_stream and
    set_pull_stream (Tensor.record_stream), so a tensor the caller frees is not
    reused by torch's allocator before the server's kernels on it have run.
    One lock covers each library call together with this bookkeeping, so
    learner threads may push while another thread applies."""

    def __init__(self, n_params: int, lr: float, momentum: float = 0.0,
                 queue_depth: Optional[int] = None, stream=None):
        self.h = ps_create(n_params, lr, momentum)
        self.n = n_params
        self._lock = threading.RLock()
        self._pending = {}   # learner id -> deque of pushed tensors, oldest first
        self._streams = []   # torch streams the device work may run on (set_stream, set_pull_stream)
        if queue_depth is not None:
            self._check(ps_set_queue_depth(self.h, queue_depth), "set_queue_depth")
        if stream is not None:
            self.set_stream(stream)

    def _check(self, rc: int, what: str) -> int:
        if rc < 0:
            raise PSError(rc, f"{what}: {ps_last_error()}")
        return rc

    def _tensor(self, t, what: str):
        if not t.is_cuda or not t.is_contiguous() or t.numel() != self.n:
            raise ValueError(f"{what}: need a contiguous device tensor of {self.n} elements")
        return t.data_ptr()

    def close(self):
        with self._lock:
            if self.h:
                ps_destroy(self.h)
                self.h = 0
                self._pending = {}

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _track(self, stream) -> None:
        if stream is not None and not isinstance(stream, int) and stream not in self._streams:
            self._streams.append(stream)

    def _uses(self, t) -> None:
        """Tell torch's caching allocator that the server's streams use `t`,
        so that freeing the tensor does not hand its memory to a new tensor
        before the kernels enqueued there have run."""
        for st in self._streams:
            t.record_stream(st)

    def set_stream(self, stream) -> None:
        ptr = stream if isinstance(stream, int) else stream.cuda_stream
        self._check(ps_set_stream(self.h, ptr), "set_stream")
        self._track(stream)

    def set_weights(self, w0) -> None:
        """Copy w0 (fp32, n values, on the device) into w on the server's
        stream; v restarts at zero."""
        if _dtype_code(w0) != PS_F32:
            raise TypeError(f"set_weights: need float32 weights, got {w0.dtype}")
        self._check(ps_set_weights(self.h, self._tensor(w0, "set_weights")), "set_weights")
        self._uses(w0)

    def set_fronts(self, fronts_log2: int) -> None:
        self._check(ps_set_fronts(self.h, fronts_log2), "set_fronts")

    def set_launch_shape(self, blocks_per_cu: int = -1, group: int = 0) -> None:
        self._check(ps_set_launch_shape(self.h, blocks_per_cu, group), "set_launch_shape")

    def set_pull_skip(self, enabled: bool) -> None:
        self._check(ps_set_pull_skip(self.h, enabled), "set_pull_skip")

    def set_queue_mode(self, mode: int, slots_per_learner: int = 1) -> None:
        self._check(ps_set_queue_mode(self.h, mode, slots_per_learner), "set_queue_mode")

    def last_applied(self):
        return ps_last_applied(self.h)

    def set_pull_fusion(self, max_replicas: int) -> None:
        self._check(ps_set_pull_fusion(self.h, max_replicas), "set_pull_fusion")

    def set_queue_depth(self, depth: int) -> None:
        self._check(ps_set_queue_depth(self.h, depth), "set_queue_depth")

    def push(self, learner: int, grad) -> bool:
        """Enqueue; False when the queue is full (nothing enqueued)."""
        ptr, code = self._tensor(grad, "push"), _dtype_code(grad)
        with self._lock:
            rc = ps_push_dtype(self.h, learner, ptr, code)
            if rc == PS_EFULL:
                return False
            self._check(rc, "push")
            self._uses(grad)
            self._pending.setdefault(learner, deque()).append(grad)
        return True

    def push_async(self, learner: int, grad, ready_event) -> bool:
        """Push a gradient still being written on another stream; the apply
        waits for `ready_event` (a recorded torch.cuda.Event) on the device."""
        ptr, code = self._tensor(grad, "push_async"), _dtype_code(grad)
        with self._lock:
            rc = ps_push_async(self.h, learner, ptr, code, ready_event.cuda_event)
            if rc == PS_EFULL:
                return False
            self._check(rc, "push_async")
            self._uses(grad)
            self._pending.setdefault(learner, deque()).append((grad, ready_event))
        return True

    def _release_applied(self) -> None:
        """Drop the references of the gradients the last apply consumed: per
        learner the oldest ones (every queue mode keeps each learner's pushes
        in order), as many as ps_last_applied names. Caller holds the lock."""
        ids = ps_last_applied(self.h)
        if isinstance(ids, int):
            self._check(ids, "last_applied")
        for l in ids:
            q = self._pending.get(l)
            if q:
                q.popleft()
                if not q:
                    del self._pending[l]

    def record(self, event) -> None:
        """Record a torch.cuda.Event on the server's stream."""
        if not event.cuda_event:
            # torch creates the HIP event on first record; make it exist
            import torch
            event.record(torch.cuda.current_stream())
        self._check(ps_record(self.h, event.cuda_event), "record")

    def set_pull_stream(self, stream) -> None:
        ptr = 0 if stream is None else (stream if isinstance(stream, int) else stream.cuda_stream)
        self._check(ps_set_pull_stream(self.h, ptr), "set_pull_stream")
        self._track(stream)

    def apply_pending(self) -> None:
        with self._lock:
            self._check(ps_apply_pending(self.h), "apply_pending")
            self._release_applied()

    def apply_sync(self) -> None:
        with self._lock:
            self._check(ps_apply_sync(self.h), "apply_sync")
            self._release_applied()

    def pull(self, learner: int, dst) -> None:
        self.pull_many([learner], [dst])

    def _replicas(self, learners: Sequence[int], dsts, what: str):
        """Pointers and the one dtype of a pull's replica tensors."""
        if len(dsts) != len(learners):
            raise ValueError(f"{what}: one destination per learner")
        codes = {_dtype_code(d) for d in dsts}
        if len(codes) > 1:
            raise ValueError(f"{what}: all replicas of one call must share a dtype")
        ptrs = [self._tensor(d, what) for d in dsts]
        for d in dsts:
            self._uses(d)
        return ptrs, (codes.pop() if codes else PS_F32)

    def pull_many(self, learners: Sequence[int], dsts) -> None:
        ptrs, dt = self._replicas(learners, dsts, "pull_many")
        self._check(ps_pull_many(self.h, list(learners), ptrs, dt), "pull_many")

    def apply_pull(self, learners: Sequence[int], dsts) -> None:
        ptrs, dt = self._replicas(learners, dsts, "apply_pull")
        with self._lock:
            self._check(ps_apply_pull(self.h, list(learners), ptrs, dt), "apply_pull")
            self._release_applied()

    def retire_learner(self, learner: int) -> int:
        """A dead learner whose gradients in server rows still apply (the
        references stay until their apply is enqueued)."""
        with self._lock:
            return self._check(ps_retire_learner(self.h, learner), "retire_learner")

    def drop_learner(self, learner: int) -> int:
        with self._lock:
            n = self._check(ps_drop_learner(self.h, learner), "drop_learner")
            # dropped gradients are never read by a kernel
            self._pending.pop(learner, None)
        return n

    def save(self, path: str) -> None:
        self._check(ps_save(self.h, path), "save")

    def load(self, path: str) -> None:
        self._check(ps_load(self.h, path), "load")

    def sync(self) -> None:
        self._check(ps_sync(self.h), "sync")

    @property
    def timestamp(self) -> int:
        return ps_timestamp(self.h)

    @property
    def pending(self) -> int:
        return ps_pending(self.h)

    def last_staleness(self):
        return ps_last_staleness(self.h)

    def stats(self) -> ps_stats:
        s = ps_get_stats(self.h)
        if isinstance(s, int):
            self._check(s, "get_stats")
        return s

    def alloc_rows(self, count: int, dtype=None):
        """`count` server-owned device buffers of n elements (ps_alloc_rows)
        as torch tensors viewing that memory. They stay valid until
        free_rows(rows) or close(); the server does not keep them alive."""
        import torch
        dtype = torch.float32 if dtype is None else dtype
        if dtype not in (torch.float32, torch.bfloat16):
            raise TypeError(f"alloc_rows: rows hold float32 or bfloat16, not {dtype}")
        code = PS_BF16 if dtype == torch.bfloat16 else PS_F32
        rc, ptrs = ps_alloc_rows(self.h, count, code)
        self._check(rc, "alloc_rows")
        return rows_as_tensors(ptrs, self.n, dtype)

    def free_rows(self, rows) -> None:
        self._check(ps_free_rows(self.h, rows[0].data_ptr()), "free_rows")

    def capture(self, script: "OpScript") -> "Graph":
        """The prepared script captured as a HIP graph (ps_graph_create):
        nothing runs and the server's state is unchanged; Graph.launch()
        replays it. The script's gradient and replica buffers must outlive
        the graph (the script itself is kept by the Graph)."""
        with self._lock:
            rc, g = ps_graph_create(self.h, script)
            self._check(rc, "graph_create")
        return Graph(self, g, script)

    def weights_copy(self):
        """A new device tensor holding w (waits for the server's stream)."""
        return self._copy(ps_weights(self.h))

    def velocity_copy(self):
        p = ps_velocity(self.h)
        return self._copy(p) if p else None

    def _copy(self, ptr: int):
        import torch
        self.sync()
        out = torch.empty(self.n, dtype=torch.float32, device="cuda")
        stream = torch.cuda.current_stream().cuda_stream
        rc = _hip()(ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ptr),
                    ctypes.c_size_t(4 * self.n), 3,   # device to device
                    ctypes.c_void_p(stream))
        if rc != 0:
            raise PSError(PS_EHIP, f"hipMemcpyAsync failed ({rc})")
        return out


class Graph:
    """A script captured by ParameterServer.capture. launch() replays it on
    the server's stream with the effect of ps_run of the script
    (ps_graph_launch); it raises PSError with PS_ESTATE, changing nothing,
    when the server's state would now launch other kernels than were
    captured. close() frees the graph after its last replay has run
    (ps_graph_destroy); close it before the server."""

    def __init__(self, server: "ParameterServer", handle: int, script: "OpScript"):
        self.server = server
        self.h = handle
        self.script = script

    def launch(self) -> None:
        if not self.h:
            raise PSError(PS_EINVAL, "graph_launch: the graph is closed")
        with self.server._lock:
            self.server._check(ps_graph_launch(self.server.h, self.h), "graph_launch")

    def close(self) -> None:
        if self.h:
            ps_graph_destroy(self.h)
            self.h = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


_hip_rt = None


def rows_as_tensors(ptrs: Sequence[int], n: int, dtype):
    """Torch tensors of n elements viewing device memory at `ptrs` (rows from
    ps_alloc_rows); no copy, no ownership."""
    import torch
    bf16 = dtype == torch.bfloat16
    out = []
    for p in ptrs:
        iface = {"shape": (n,), "typestr": "<i2" if bf16 else "<f4", "data": (p, False),
                 "version": 2}
        t = torch.as_tensor(_DeviceArray(iface), device="cuda")
        out.append(t.view(torch.bfloat16) if bf16 else t)
    return out


class _DeviceArray:
    """Device memory described by the CUDA array interface (torch imports it
    without copying)."""

    def __init__(self, iface):
        self.__cuda_array_interface__ = iface


def _hip():
    """hipMemcpyAsync of the HIP runtime the library itself is bound to
    (looked up through the library's handle, which searches its
    dependencies), for the plain copy above."""
    global _hip_rt
    if _hip_rt is None:
        f = load_library().hipMemcpyAsync
        f.restype = ctypes.c_int
        f.argtypes = [_VP, _VP, ctypes.c_size_t, ctypes.c_int, _VP]
        _hip_rt = f
    return _hip_rt
