"""The paper-style CPU server (oracle/cpu_ps.c) gives the oracle's bits:
fp32 and bf16 gradients, with and without momentum, at several thread
counts and a ragged length; pulls copy exactly."""
import numpy as np
import pytest

from oracle import cpu_ps
from oracle import server as orc


@pytest.mark.parametrize("threads", [1, 3, 8])
@pytest.mark.parametrize("m", [0.0, 0.9])
def test_cpu_ps_bitwise_equal_to_oracle(threads, m):
    rng = np.random.default_rng(7 + threads)
    n, k, lr = 100_003, 6, 0.01
    w0 = rng.uniform(-0.05, 0.05, n).astype(np.float32)
    grads = []
    for j in range(k):
        g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
        grads.append(orc.f32_to_bf16(g) if j % 3 == 2 else g)
    o = orc.OracleServer(w0, lr, m, depth=k)
    for j, g in enumerate(grads):
        o.push(j, g)
    o.apply_pending()
    w = w0.copy()
    v = np.zeros_like(w) if m else None
    for g in grads:
        cpu_ps.step(w, v, g, np.float32(lr), np.float32(m), threads)
    assert np.array_equal(w.view(np.uint32), o.w.view(np.uint32))
    if m:
        assert np.array_equal(v.view(np.uint32), o.v.view(np.uint32))
    dst = np.empty_like(w)
    cpu_ps.pull(dst, w, threads)
    assert np.array_equal(dst.view(np.uint32), w.view(np.uint32))
