"""bench.py's command line without a GPU: the one-GPU refusal and the modes it
offers."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)
    assert not r.stdout.strip().startswith("{")


def test_help_lists_every_mode():
    r = _run("--help")
    assert r.returncode == 0
    for flag in ("--steps", "--warmup", "--workload", "--decoder", "--grid", "--frontend",
                 "--no-cpu-baseline", "--cpu-seconds", "--row-tiles"):
        assert flag in r.stdout, flag



def test_roofline_work_is_the_projection_count():
    # the roofline's work is the least-squares projection of every block on every
    # seed's basis: 2 C P flops per candidate (48 at P = 3), not the kernel's own
    # quadratic form (72) or what it issues (96), which are reported separately
    sys.path.insert(0, ROOT)
    import bench
    assert bench.projection_flops(16, 3) == 65535 * 2 * 8 * 3
    assert bench.projection_flops(12, 2) == 4095 * 32
    assert bench.projection_flops(20, 4) == ((1 << 20) - 1) * 64
    assert bench.QUADFORM_FLOPS_PER_CANDIDATE == 72.0
    assert bench.ISSUED_FLOPS_PER_CANDIDATE == 96.0
