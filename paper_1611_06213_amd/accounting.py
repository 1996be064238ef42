"""Byte accounting of the parameter server.

Two views, kept apart:
  * algorithmic HBM bytes of this implementation (what the kernels must
    move: K gradient reads, w and v read and write, replica writes);
  * the paper's learner<->PS accounting (Sec. 3): every push moves the
    gradient to the server and the weights back, so 2 x ModelSize per push,
    and the minimum bandwidth for any ASGD speedup is
    RB = 2 * ModelSize / (TPE / (N / mu))   (Table "bandwidth_requirement"),
    with TPE the training time per epoch, N the training samples and mu the
    mini-batch size. Table "bandwidth_utilized" reports the same accounting
    measured ("data transferred between learners and PS / runtime").
"""


def learner_ps_bytes_per_push(n_params: int, bytes_per_param: int = 4) -> int:
    """Gradient in + weights out, one model each (Sec. 3)."""
    return 2 * n_params * bytes_per_param


def required_bandwidth(model_bytes: float, samples: float, mu: float, tpe_seconds: float) -> float:
    """RB in bytes/s: 2 x model per mini-batch over the time per mini-batch."""
    return 2.0 * model_bytes * (samples / mu) / tpe_seconds


def apply_bytes(n: int, k: int, grad_bytes: int, momentum: bool) -> int:
    """HBM bytes of one apply of k gradients: k gradient reads, w read and
    write, v read and write with momentum."""
    return k * n * grad_bytes + 8 * n + (8 * n if momentum else 0)


def pull_bytes(n: int, r: int, replica_bytes: int, separate: bool = True) -> int:
    """HBM bytes of writing r replicas: r writes, plus one read of w when the
    pull is its own kernel (a fused pull reuses the apply's registers). No
    replica, no kernel: 0."""
    if r <= 0:
        return 0
    return r * n * replica_bytes + (4 * n if separate else 0)
