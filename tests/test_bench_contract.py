"""bench.py's command-line contract on the host: it measures one GPU and
refuses more, before anything touches a device."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          env=env, capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_multi_rank_launch_is_refused():
    r = _run([], {"WORLD_SIZE": "2"})
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_percentile_helper_is_nearest_rank():
    sys.path.insert(0, ROOT)
    import bench

    ts = [1.0, 2.0, 3.0, 4.0, 5.0, 6.0, 7.0, 8.0, 9.0, 10.0, 11.0]
    assert bench.pct(ts, 0) == 1.0e-3
    assert bench.pct(ts, 50) == 6.0e-3
    assert bench.pct(ts, 90) == 10.0e-3
    assert bench.pct(ts, 100) == 11.0e-3
    assert bench.pct([4.0], 10) == 4.0e-3
