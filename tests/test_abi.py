"""The C ABI library loads on a machine without a GPU and exports every
function include/ps.h declares; argument validation that needs no device
answers with the documented status codes."""
import ctypes
import os
import re

import pytest

from paper_1611_06213_amd import ps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "ps.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ps_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ps.LIB_PATH):
        pytest.fail("libgadeips.so is not built (run __graft_entry__.build())")
    return ps.load_library()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert "ps_create" in names and "ps_apply_pending" in names and len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    # and the binding covers the same list, under the same names
    assert set(names) == set(ps._SIGS)
    for n in names:
        assert callable(getattr(ps, n)), n


def test_header_constants_match_binding():
    text = open(os.path.join(ROOT, "include", "ps.h")).read()
    for name in ("PS_OK", "PS_EINVAL", "PS_EFULL", "PS_ENOMEM", "PS_EHIP", "PS_ESTATE",
                 "PS_EIO", "PS_F32", "PS_BF16", "PS_QUEUE_FIFO", "PS_QUEUE_ROUND_ROBIN"):
        m = re.search(rf"\b{name}\s*=\s*(-?\d+)", text)
        assert m and int(m.group(1)) == getattr(ps, name), name
    for name in ("PS_OP_PUSH", "PS_OP_APPLY", "PS_OP_APPLY_SYNC", "PS_OP_PULL",
                 "PS_OP_APPLY_PULL"):
        m = re.search(rf"\b{name}\s*=\s*(-?\d+)", text)
        assert m and int(m.group(1)) == getattr(ps, name), name
    for name in ("PS_MAX_QUEUE_DEPTH", "PS_MAX_REPLICAS", "PS_MAX_LEARNERS", "PS_STALENESS_BINS",
                 "PS_MAX_ROWS", "PS_IPC_HANDLE_BYTES"):
        m = re.search(rf"#define {name} (\d+)", text)
        assert m and int(m.group(1)) == getattr(ps, name), name
    assert ctypes.sizeof(ps.ps_stats) == 8 * (10 + ps.PS_STALENESS_BINS)
    # ps_op: four ints, then three pointers (x86-64)
    assert ctypes.sizeof(ps.ps_op) == 40 and ps.ps_op.grad.offset == 16


def test_validation_without_device(lib):
    assert lib.ps_create(0, 0.1, 0.0) is None
    assert "n_params" in ps.ps_last_error()
    assert lib.ps_create((1 << 48) + 1, 0.1, 0.0) is None     # sizes could overflow
    assert lib.ps_create(1 << 62, 0.1, 0.0) is None
    assert lib.ps_create(10, float("nan"), 0.0) is None
    assert lib.ps_create(10, 0.1, float("inf")) is None
    assert lib.ps_push(None, 0, None) == ps.PS_EINVAL
    assert lib.ps_run(None, None, 0, None) == ps.PS_EINVAL
    assert lib.ps_retire_learner(None, 0) == ps.PS_EINVAL
    assert lib.ps_export_rows(None, None, None, None) == ps.PS_EINVAL
    assert lib.ps_import_rows(None, 0, None) == ps.PS_EINVAL
    assert lib.ps_release_rows(ctypes.c_void_p(4096)) == ps.PS_EINVAL
    assert ps.ps_import_rows(b"short", 0) == (ps.PS_EINVAL, 0)
    assert lib.ps_apply_pending(None) == ps.PS_EINVAL
    assert lib.ps_pull(None, 0, None) == ps.PS_EINVAL
    assert ps.ps_pull_many(None, [0], [1], ps.PS_F32) == ps.PS_EINVAL
    assert lib.ps_set_queue_depth(None, 4) == ps.PS_EINVAL
    assert lib.ps_sync(None) == ps.PS_EINVAL
    assert lib.ps_pending(None) == ps.PS_EINVAL
    assert lib.ps_save(None, b"/tmp/x") == ps.PS_EINVAL and lib.ps_load(None, b"/tmp/x") == ps.PS_EINVAL
    assert lib.ps_drop_learner(None, 0) == ps.PS_EINVAL
    assert ps.ps_alloc_rows(None, 2, ps.PS_F32)[0] == ps.PS_EINVAL
    assert lib.ps_free_rows(None, None) == ps.PS_EINVAL
    assert lib.ps_set_fronts(None, 0) == ps.PS_EINVAL
    assert lib.ps_set_launch_shape(None, 1, 16) == ps.PS_EINVAL
    assert lib.ps_set_pull_fusion(None, -1) == ps.PS_EINVAL
    assert lib.ps_graph_launch(None, None) == ps.PS_EINVAL
    assert ps.ps_graph_create(None, ps.OpScript())[0] == ps.PS_EINVAL
    lib.ps_graph_destroy(None)   # no-op
    assert lib.ps_timestamp(None) == 0 and lib.ps_num_params(None) == 0
    assert not lib.ps_weights(None)
    lib.ps_destroy(None)   # no-op


def test_binding_refuses_missing_library(tmp_path):
    with pytest.raises(RuntimeError, match="not built"):
        ps.load_library(str(tmp_path / "missing.so"))


def test_one_hip_runtime_whatever_the_import_order():
    """Loading the library through the binding before anything else imports
    torch must still leave a single HIP runtime in the process (torch's), so
    torch streams and allocations are valid in the library."""
    import ast
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_1611_06213_amd import ps\n"
            "ps.load_library()\n"
            "import torch\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "print(sorted({l.split()[-1] for l in maps if 'libamdhip64' in l}))\n") % ROOT
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    libs = ast.literal_eval(out.stdout.strip().splitlines()[-1])
    assert len(libs) == 1, libs


def test_binding_refuses_mixed_replica_dtypes():
    """The binding passes one dtype per pull call, so it must refuse replica
    lists that mix dtypes (a bf16 buffer written as fp32 would overflow)."""
    import torch
    srv = ps.ParameterServer.__new__(ps.ParameterServer)
    srv.n = 4
    srv.h = 0
    srv._streams = []

    class FakeDev:
        def __init__(self, dtype):
            self.dtype = dtype
            self.is_cuda = True

        def is_contiguous(self):
            return True

        def numel(self):
            return 4

        def data_ptr(self):
            return 4096

    with pytest.raises(ValueError, match="share a dtype"):
        srv._replicas([0, 1], [FakeDev(torch.float32), FakeDev(torch.bfloat16)], "pull_many")
    ptrs, dt = srv._replicas([0, 1], [FakeDev(torch.bfloat16)] * 2, "pull_many")
    assert dt == ps.PS_BF16 and ptrs == [4096, 4096]


def test_binding_refuses_non_fp32_weights():
    """ps_set_weights copies n fp32 values: a bf16 tensor of n elements holds
    half as many bytes, so the binding must refuse it before the call."""
    import torch
    srv = ps.ParameterServer.__new__(ps.ParameterServer)
    srv.n = 4
    srv.h = 0
    srv._streams = []

    class FakeDev:
        dtype = torch.bfloat16
        is_cuda = True

        def is_contiguous(self):
            return True

        def numel(self):
            return 4

        def data_ptr(self):
            return 4096

    with pytest.raises(TypeError, match="float32"):
        srv.set_weights(FakeDev())


def test_binding_refuses_other_row_dtypes():
    """Server rows hold fp32 or bf16; any other dtype is refused before the
    library is called (a float16 request must not come back as fp32 rows)."""
    import torch
    srv = ps.ParameterServer.__new__(ps.ParameterServer)
    srv.n = 4
    srv.h = 0
    srv._streams = []
    for dt in (torch.float16, torch.float64, torch.int32):
        with pytest.raises(TypeError, match="float32 or bfloat16"):
            srv.alloc_rows(2, dt)
