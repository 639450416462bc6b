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
           "--warmup", "1", "--no-cpu", "--no-peaks", "--no-others", *extra]
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
    the counters were not taken on), the oracle's CPU baseline and the peak microbenchmarks
    measured in the same run."""
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--config", "tiny", "--steps", "2",
           "--warmup", "1"]
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
    pk = out["peaks_measured"]
    assert 0 < pk["mfma_f32_tflops"] and 0 < pk["valu_f32_fma_tflops"] and 0 < pk["hbm_copy_gbs"]
    pair = pk["mfma_valu_same_simd"]
    assert min(pair["mfma_only_ms"], pair["valu_only_ms"]) > 0
    assert pair["both_ms"] >= max(pair["mfma_only_ms"], pair["valu_only_ms"]) * 0.95
    assert abs(pair["both_over_sum"] - pair["both_ms"] /
               (pair["mfma_only_ms"] + pair["valu_only_ms"])) < 2e-3
    assert abs(rl["frac_of_measured_mfma"] - rl["achieved"] / pk["mfma_f32_tflops"]) < 1e-3
    _check_share(out["share"], out["config"]["nnz"])


def _check_share(sh, nnz):
    """GPU 0's share of an 8-GPU node: about nnz / 8 ratings per side, timed like the rest."""
    assert sh["gpus"] == 8
    for side in ("user", "item"):
        s = sh[side]
        assert s["share_rows"] >= 1 and 0 < s["herm_ms"] <= s["half_sweep_ms"]
        # the first rows (columns) that reach nnz / 8; one row or column overshoots it
        assert nnz / 8 <= s["share_nnz"] <= nnz / 8 + 0.05 * nnz
        # (a tiny share is launch-bound: its fraction of the peak can round to 0)
        assert 0 <= s["herm_frac_fp32_peak"] < 1 and s["full_over_gpus_ms"] > 0


@pytest.mark.gpu
def test_bench_workloads_block():
    """The bench line's block of other workloads (here the rank sweep and the music shape; the
    default run adds the wiki shape): per workload and side, the half-sweep and k_herm_solve
    times from the library's HIP events, the fraction of the FP32 peak, the roofline bound with
    its AI and where the bytes came from, and the algorithmic Gram / solve flop split."""
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--config", "movie", "--steps", "2",
           "--warmup", "1", "--no-cpu", "--no-peaks", "--other-steps", "1",
           "--others", "movie_f32,movie_f64,movie_f128,music"]
    print("[bench]", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    out = json.loads(r.stdout.strip().splitlines()[-1])
    assert "workloads_error" not in out, out.get("workloads_error")
    w = out["workloads"]
    assert set(w) == {"movie_f32", "movie_f64", "movie_f128", "music"}
    for name, blk in w.items():
        f = int(blk["workload"].split(" f=")[1].split()[0])
        assert blk["half_sweeps_per_s"] > 0 and 0 < blk["herm_pair_frac_fp32_peak"] < 1
        for side in ("user", "item"):
            s = blk[side]
            assert 0 < s["herm_ms"] <= s["half_sweep_ms"]
            assert abs(s["herm_frac_fp32_peak"] - s["herm_tflops"] / 157.3) < 1e-3
            rl = s["roofline"]
            assert rl["bound"] in ("hbm", "mfma")
            herm_fl = s["flops"]["gram"] + (s["rows"] - s["split_rows"]) * (
                f ** 3 / 3 + 2.5 * f * f + f / 6)
            assert abs(rl["ai_flop_per_byte"] - herm_fl / rl["bytes"]) <= 0.006
            peak = min(157.3, 8.0 * herm_fl / rl["bytes"])
            assert abs(rl["peak_tflops"] - peak) < 0.006
            assert (rl["bound"] == "hbm") == (peak < 157.3)
            assert abs(rl["frac"] - s["herm_tflops"] / rl["peak_tflops"]) < 1e-3
            assert 0 < s["flops"]["gram_share"] < 1
        # the user side carries the solves: its Gram share is the smaller one
        assert blk["user"]["flops"]["gram_share"] < blk["item"]["flops"]["gram_share"]
        if name == "music":
            nnz = int(blk["workload"].split(" nnz=")[1].split()[0])
            _check_share(blk["share"], nnz)
