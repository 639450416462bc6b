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
