"""bench.py's host-side pieces on the CPU: the kernel-code digest that keys
recorded counters, and the multi-GPU refusal."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_kernel_digest_ignores_comments_not_code(tmp_path):
    a = tmp_path / "a.hip"
    a.write_text("// header\n__global__ void k(float *p) { p[0] = 1.0f; /* one */ }\n")
    b = tmp_path / "b.hip"
    b.write_text("/* another\n header */\n__global__ void k(float *p) {\n  p[0] = 1.0f; // one\n}\n")
    c = tmp_path / "c.hip"
    c.write_text("__global__ void k(float *p) { p[0] = 2.0f; }\n")
    da, db, dc = (bench.kernel_source_digest(str(x)) for x in (a, b, c))
    assert da == db != dc
    # over several files: any code change in any of them counts
    assert bench.kernel_source_digest([str(a), str(c)]) == bench.kernel_source_digest([str(b), str(c)])
    assert bench.kernel_source_digest([str(a), str(c)]) != bench.kernel_source_digest([str(a), str(a)])


def test_kernel_digest_covers_launch_shaping_host_code():
    """The counters bench.py reports are keyed to the kernels and to the host
    code that picks their launch shapes and buffer placement."""
    names = {os.path.basename(p) for p in bench.KERNEL_SRC}
    assert names == {"ps_kernels.hip", "ps_kernels.h", "ps_server.cpp", "ps_layout.cpp",
                     "ps_layout.h"}


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_cpu_baseline_reports_rate_and_bytes():
    """The oracle leg on a small workload: pushes/s, the algorithmic GB/s of
    the same steps (bytes per step x steps / time), one core, and the
    paper-style server beside it."""
    from paper_1611_06213_amd import accounting as acc
    from paper_1611_06213_amd import workloads as wl
    cfg = wl.CONFIGS["alexnet"].scaled(50_000, pool=8)
    pool = [wl.make_grad(cfg, j, "cpu") for j in range(cfg.pool)]
    r = bench.cpu_baseline(cfg, pool, wl.make_w0(cfg, "cpu"), 4, 0.2)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["unit"] == "pushes/s"
    step = acc.apply_bytes(cfg.n, cfg.depth, 4, True) + acc.pull_bytes(cfg.n, 4, 4)
    assert abs(r["gbps_algorithmic"] / (r["value"] / cfg.depth * step / 1e9) - 1) < 0.01
    assert r["paper_style_ps"]["value"] > 0


def test_algorithmic_bytes_per_step_and_launch():
    """The bytes bench.py divides by: a VGG-16 step moves the apply's
    19,923,486,336 bytes plus the 16-replica pull's 9,408,312,992 (29.33 GB,
    the figure the roofline is quoted on); the dominant launch is the apply.
    ps_apply_pull with one replica writes it from the apply pass (no second
    read of w); above one replica the pull is its own kernel again."""
    from paper_1611_06213_amd import workloads as wl
    cfg = wl.CONFIGS["vgg16"]
    n = cfg.n
    assert bench.algorithmic_bytes(cfg, "separate", 16) == (29_331_799_328, 19_923_486_336)
    assert bench.algorithmic_bytes(cfg, "fused", 16) == (29_331_799_328, 29_331_799_328)
    one = 19_923_486_336 + 4 * n
    assert bench.algorithmic_bytes(cfg, "fused", 1) == (one, one)
    assert bench.algorithmic_bytes(cfg, "separate", 0) == (19_923_486_336, 19_923_486_336)
    mixed = wl.CONFIGS["mixed"]
    assert bench.algorithmic_bytes(mixed, "separate", 32)[0] == 29_600_000_000


def test_recorded_traffic_matches_mode_and_digest(tmp_path):
    """Counter bytes are reported for the workload and mode they were taken
    on, and only while the kernel code digest still matches."""
    d = bench.kernel_source_digest()
    (tmp_path / "traffic_apply_vec_a.txt").write_text(
        f"# header\nmode: vgg16-separate\nkernel_code_digest: {d}\nhbm_bytes_per_launch: 123\n")
    (tmp_path / "traffic_apply_vec_b.txt").write_text(
        f"mode: mixed-separate\nkernel_code_digest: {d}\nhbm_bytes_per_launch: 456\n")
    (tmp_path / "traffic_apply_vec_c.txt").write_text(
        "mode: alexnet-separate\nkernel_code_digest: 0000\nhbm_bytes_per_launch: 789\n")
    pat = str(tmp_path / "traffic_apply_vec_*.txt")
    assert bench.recorded_traffic("vgg16-separate", pat) == 123.0
    assert bench.recorded_traffic("mixed-separate", pat) == 456.0
    assert bench.recorded_traffic("alexnet-separate", pat) is None     # other kernel code
    assert bench.recorded_traffic("vgg16-fused", pat) is None          # not measured
