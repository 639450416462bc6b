"""bench.py's overlapped step (the training RMSE of step k on a second stream beside step k+1, X
and Theta double-buffered, step k+2 waiting for it) computes what the serial step computes: the
same training RMSE after the last step, to the last bit (every kernel is deterministic and the
RMSE does not depend on how many waves run it)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(config, *extra):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--config", config, "--steps", "3",
           "--warmup", "1", "--no-cpu", "--no-peaks", *extra]
    print("[bench]", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    return json.loads(r.stdout.strip().splitlines()[-1])


@pytest.mark.gpu
@pytest.mark.parametrize("config", ["tiny", "movie"])
def test_overlapped_step_matches_serial(config):
    ov = _bench(config)
    se = _bench(config, "--serial-rmse")
    assert ov["nonspd_rows"] == 0 and se["nonspd_rows"] == 0
    assert ov["train_rmse"] == se["train_rmse"]
    assert 0.0 < ov["train_rmse"] < 10.0


@pytest.mark.gpu
def test_bench_line_contract():
    """One JSON line with the contract's fields: the metric, whole-job value and step time,
    the roofline of the dominant kernel (frac = achieved / peak; no traffic figure for a workload
    the counters were not taken on) and the oracle's CPU baseline."""
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--config", "tiny", "--steps", "2",
           "--warmup", "1", "--no-peaks"]
    print("[bench]", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    out = json.loads(r.stdout.strip().splitlines()[-1])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in out, key
    assert out["n_gpus"] == 1 and out["steps"] == 2 and out["warmup"] == 1
    assert out["value"] > 0 and out["unit"] == "half-sweeps/s" and out["higher_is_better"]
    assert abs(out["value"] - 2000.0 / out["ms_per_step"]) <= 0.01 * out["value"]
    assert out["config"]["workload"].startswith("tiny:")
    rl = out["roofline"]
    assert rl["bound"] == "mfma" and rl["unit"] == "TFLOP/s" and rl["peak"] == 157.3
    assert abs(rl["frac"] - rl["achieved"] / rl["peak"]) < 1e-3
    assert rl["traffic"] is None
    cb = out["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["sample"]
