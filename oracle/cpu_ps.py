"""The paper-style CPU parameter server (cpu_ps.c), for context beside the
oracle: one OpenMP pass over the weights per gradient, eight coordinates per
loop iteration (Sec. 4.1, 4.4). Test infrastructure, like the rest of
oracle/; bitwise equal to the oracle (tests/test_cpu_ps.py)."""
import ctypes
import os

import numpy as np

from oracle import build as _build

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.CPS_LIB):
            _build.build()
        L = ctypes.CDLL(_build.CPS_LIB)
        L.cps_step.restype = None
        L.cps_step.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                               ctypes.c_size_t, ctypes.c_float, ctypes.c_float, ctypes.c_int]
        L.cps_pull.restype = None
        L.cps_pull.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _lib = L
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def step(w: np.ndarray, v, g: np.ndarray, lr: float, m: float, threads: int) -> None:
    """One gradient (float32, or uint16 bf16 bits) folded into w (and v) in place."""
    assert w.dtype == np.float32 and w.flags.c_contiguous and g.size == w.size
    assert g.dtype in (np.float32, np.uint16) and g.flags.c_contiguous
    lib().cps_step(_p(w), _p(v) if v is not None else None, _p(g), int(g.dtype == np.uint16),
                   w.size, lr, m if v is not None else 0.0, threads)


def pull(dst: np.ndarray, w: np.ndarray, threads: int) -> None:
    assert dst.dtype == np.float32 and dst.size == w.size
    lib().cps_pull(_p(dst), _p(w), w.size, threads)
