"""bench.py's contract: on the host it refuses more than one GPU before
anything touches a device; on the GPU a short run prints the one JSON line."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env_extra=None, timeout=120):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          env=env, capture_output=True, text=True, timeout=timeout)


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


@pytest.mark.gpu
def test_bench_line_on_the_gpu():
    """One short run of the decode-step benchmark: one JSON line with the
    contract's keys, and per-call spreads that bracket their medians."""
    import json

    r = _run(["--steps", "3", "--warmup", "1", "--no-secondary", "--no-cpu-baseline",
              "--roofline-reps", "4"], timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "breakdown"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["value"] > 0
    assert d["config"]["workload"]
    rl = d["roofline"]
    assert rl["bound"] in ("hbm", "mfma")
    assert 0 < rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], abs=1e-3)
    assert len(d["breakdown"]) == 40
    for c in d["breakdown"]:
        assert 0 < c["us_p10"] <= c["us"] <= c["us_p90"], c


@pytest.mark.gpu
def test_ceiling_probes_on_the_gpu():
    """bench.py --ceilings: the probe kernels run, and what they measure is
    positive and within the published peaks (HBM 8 TB/s, FP16 2.5 and FP8
    5.0 PFLOP/s dense); the LDS fill grows with the issuing waves on
    L2-resident data."""
    import json

    r = _run(["--ceilings"], timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    c = json.loads(r.stdout.strip().splitlines()[-1])["ceilings"]
    assert 0 < c["hbm_read_GBs_plain"] <= 8000 and 0 < c["hbm_read_GBs_nontemporal"] <= 8000
    assert 0 < c["mfma_f16_TFLOPs"] <= 2500 and 0 < c["mfma_fp8_TFLOPs"] <= 5000
    fill = c["lds_fill_GBs_per_CU"]
    assert len(fill) == 6 and all(v > 0 for v in fill.values())
    assert fill["l2_1MiB_16waves"] > fill["l2_1MiB_4waves"]
    loop = c["mfma_lds_loop_TFLOPs"]
    assert len(loop) == 4 and all(0 < v <= 2500 for v in loop.values())
