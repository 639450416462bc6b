#!/usr/bin/env python3
"""Benchmark: ALS half-sweeps/s and get_hermitian+solve GFLOP/s on one MI355X.

One step = one ALS iteration on the movie-shaped workload (480,000 x 17,770, 100M synthetic
ratings, f = 100, lambda = 0.05): update-X (half-sweep on the CSR), update-Theta (half-sweep
on the CSC) and the training RMSE, all through the C ABI of include/als.h.  Inputs are
resident in HBM before the timed region.  `value` = half-sweeps per second over the K timed
steps (2 per step).  Step k's RMSE (it reads X_k and Theta_k) runs on a second stream, one wave
per SIMD, beside step k+1 (which only reads Theta_k; X and Theta are double-buffered), and
step k+2, which overwrites X_k and Theta_k, waits for it; --serial-rmse runs it after
update-Theta instead.

After the timed region: peak microbenchmarks (FP32 MFMA and VALU FMA rates, an HBM copy) for
measured denominators, then the fp64 CPU oracle on a bounded row sample (all host threads, plus
one thread on the first 10,000 user rows).

Prints one JSON line.  Flop accounting (algorithmic, symmetric-half):
  per stored entry  F_h = f^2 + 3 f          (lower-triangle Gram f(f+1) + right-hand side 2f)
  per non-empty row F_s = f^3/3 + 5 f^2/2 + f/6  (Cholesky + two triangular solves)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_PEAK_TFLOPS = 157.3      # MI355X dense FP32 (matrix and packed vector), datasheet
HBM_PEAK_GBS = 8000.0
METRIC = "ALS half-sweeps/sec and get_hermitian+solve GFLOP/s (% of FP32 peak), 1 GPU"


def F_h(f):
    return f * f + 3 * f


def F_s(f):
    return f ** 3 / 3.0 + 2.5 * f * f + f / 6.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="movie", help="synth config name (movie, tiny, music)")
    ap.add_argument("--f", type=int, default=None, help="rank override (rank sweep)")
    ap.add_argument("--cpu-flops", type=float, default=1.2e12,
                    help="algorithmic flops of the oracle baseline's sample (every k-th row of "
                         "each side, k chosen to match)")
    ap.add_argument("--cpu-stride", type=int, default=0, help="fixed sampling stride instead")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-peaks", action="store_true", help="skip the peak microbenchmarks")
    ap.add_argument("--driver", action="store_true",
                    help="instead of the step benchmark: the ALS driver on a seeded 99/1 "
                         "train/test split, test RMSE per iteration, with and without async "
                         "checkpoints (one JSON line)")
    ap.add_argument("--test-frac", type=float, default=0.01)
    ap.add_argument("--stream", action="store_true",
                    help="instead of the step benchmark: half-sweeps with R streamed from pinned "
                         "host memory in row batches (PCIe-inclusive; one JSON line)")
    ap.add_argument("--batch-entries", type=int, default=16_000_000)
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the step benchmark: the half-sweeps under each design "
                         "alternative (gather form x last-block form), one JSON line")
    ap.add_argument("--checkpoint-every", type=int, default=5)
    ap.add_argument("--serial-rmse", action="store_true",
                    help="run each step's RMSE after its update-Theta on the same stream (default: "
                         "on a second stream and context, one wave per SIMD, beside the next "
                         "step's update-X, with X double-buffered)")
    ap.add_argument("--other-steps", type=int, default=3,
                    help="timed steps per other workload (rank sweep, music, wiki)")
    ap.add_argument("--no-share", action="store_true",
                    help="skip the one-GPU-share timing (GPU 0's nnz-balanced 1/8 of each side)")
    ap.add_argument("--no-others", action="store_true",
                    help="time the headline workload only (no rank sweep, music or wiki block)")
    ap.add_argument("--others", default="movie_f32,movie_f64,movie_f128,music,wiki",
                    help="comma list of the other workloads to time after the headline")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="for hardware-counter runs: a 1 GiB device copy (the bytes-per-KiB "
                         "calibration), then one user and one item half-sweep, one "
                         "full-width training RMSE and one device CSR->CSC build; no JSON")
    return ap.parse_args()


KERNEL_SRC = os.path.join(ROOT, "paper_1603_03820_amd", "csrc", "als.hip")


def traffic_file(tag: str) -> str:
    """The committed counter summary of k_herm_solve's HBM traffic on one workload."""
    return os.path.join(ROOT, "profiles", f"k_herm_solve_{tag}_traffic.txt")


def measured_traffic(workload: str, tag: str = "movie_f100", key: str = "bytes_per_launch"):
    """HBM bytes per k_herm_solve launch (or per user / item launch with key bytes_user_launch,
    bytes_item_launch) from the committed counter summary, if it was taken on this workload
    and on the kernel source as it is now (else None)."""
    import hashlib
    path = traffic_file(tag)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    src = hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()
    if kv.get("source_sha256") != src or kv.get("workload") != workload or key not in kv:
        return None
    return float(kv[key])


def roofline_bound(flops: float, nbytes: float):
    """The roofline that bounds a kernel doing `flops` with `nbytes` of HBM traffic:
    min(FP32 peak, HBM peak x AI) in TFLOP/s, and which side binds."""
    ai = flops / nbytes
    hbm_tflops = HBM_PEAK_GBS * ai / 1e3
    if hbm_tflops < FP32_PEAK_TFLOPS:
        return "hbm", hbm_tflops, ai
    return "mfma", FP32_PEAK_TFLOPS, ai


def algorithmic_bytes(nnz: int, m: int, n: int, f: int) -> float:
    """Compulsory HBM bytes of one half-sweep: indices + ratings, row pointers, the gathered
    factor once, the written factor once (A_u never leaves the chip)."""
    return 8.0 * nnz + 8.0 * (m + 1) + 4.0 * n * f + 4.0 * m * f


def split_rows(bounds: np.ndarray, rowptr: np.ndarray) -> int:
    """Rows cut by a chunk boundary (finished by the reduce kernel, not by herm_solve)."""
    m = len(rowptr) - 1
    cut = set()
    for u, k in bounds[1:-1]:
        if u < m and 0 < k < rowptr[u + 1] - rowptr[u]:
            cut.add(int(u))
    return len(cut)


def measure_peaks(dev):
    """Measured FP32 MFMA and VALU FMA rates and an HBM copy rate on this GPU (the kernels in
    csrc/peaks.hip), each the best of 3 event-timed launches on the current stream."""
    import ctypes
    import torch
    from paper_1603_03820_amd import build as B
    if not os.path.exists(B.PEAKS_LIB):
        raise RuntimeError(f"{B.PEAKS_LIB} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(B.PEAKS_LIB)
    V, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.peaks_mfma.argtypes = [V, V, i32, i32, V]
    lib.peaks_fma.argtypes = [V, V, i32, i32, V]
    lib.peaks_copy.argtypes = [V, V, i64, i32, V]
    lib.peaks_pair.argtypes = [V, V, i32, i32, i32, i32, V]
    chains = lib.peaks_chains()
    per_iter = lib.peaks_fma_per_iter()
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    st = torch.cuda.current_stream()
    sp = V(st.cuda_stream)
    inp = torch.rand(128, device=dev)

    def best_ms(launch):
        assert launch() == 0
        times = []
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            assert launch() == 0
            e1.record(st)
            e1.synchronize()
            times.append(e0.elapsed_time(e1))
        return min(times)

    def best(launch, work):
        return work / (best_ms(launch) * 1e-3)

    blocks, iters = cus * 8, 20000                      # 2 waves per SIMD
    out = torch.empty(blocks * 256, device=dev)
    mfma = best(lambda: lib.peaks_mfma(V(inp.data_ptr()), V(out.data_ptr()), blocks, iters, sp),
                blocks * iters * chains * 2048.0)
    fblocks, fiters = cus * 8, 5000                     # 8 waves per SIMD
    fout = torch.empty(fblocks * 256, device=dev)
    fma = best(lambda: lib.peaks_fma(V(inp.data_ptr()), V(fout.data_ptr()), fblocks, fiters, sp),
               fblocks * 256.0 * fiters * per_iter * 2)
    # one MFMA wave and one VALU wave on every SIMD: alone, then together
    pout = torch.empty(cus * 512, device=dev)
    pair = [best_ms(lambda: lib.peaks_pair(V(inp.data_ptr()), V(pout.data_ptr()), cus, 20000,
                                           20000, mode, sp)) for mode in (1, 2, 3)]
    n4 = (1 << 30) // 16                                # 1 GiB each way
    src = torch.ones(n4 * 4, device=dev)
    dst = torch.empty_like(src)
    copy = best(lambda: lib.peaks_copy(V(src.data_ptr()), V(dst.data_ptr()), n4, cus * 16, sp),
                32.0 * n4)
    del src, dst
    return {"mfma_f32_tflops": round(mfma / 1e12, 2), "valu_f32_fma_tflops": round(fma / 1e12, 2),
            "hbm_copy_gbs": round(copy / 1e9, 1),
            "mfma_clock_ghz": round(mfma / (cus * 256.0) / 1e9, 3),
            "mfma_valu_same_simd": {"mfma_only_ms": round(pair[0], 3),
                                    "valu_only_ms": round(pair[1], 3),
                                    "both_ms": round(pair[2], 3),
                                    "both_over_sum": round(pair[2] / (pair[0] + pair[1]), 3)},
            "note": "unpacked FP32 FMA (packed FP32 is not used); copy = read + write bytes; "
                    "mfma_valu_same_simd: one MFMA-stream wave and one VALU-stream wave per SIMD, "
                    "both_over_sum near 1 = the two kinds of work do not overlap"}


def csc_build(ctx, dp, p, reps=3):
    """The item side's input, R^T as CSC, built on the device by als_csr_to_csc from the resident
    CSR (outside the timed steps): median HIP-event time, and whether it equals, bit for bit, the
    CSC the host-side input generator produced (which the timed steps read)."""
    import torch
    from paper_1603_03820_amd import als
    out = (torch.empty_like(dp.colptr), torch.empty_like(dp.rowidx), torch.empty_like(dp.vals_t))
    ts = []
    for _ in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        als.als_csr_to_csc(ctx, dp.rowptr, dp.colidx, dp.vals, p.m, p.n, nnz=p.nnz, out=out)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    same = (torch.equal(out[0], dp.colptr) and torch.equal(out[1], dp.rowidx)
            and torch.equal(out[2].view(torch.int32), dp.vals_t.view(torch.int32)))
    return {"ms": round(float(np.median(ts[1:])), 3), "matches_generator_csc": bool(same),
            "note": "R^T on the device (als_csr_to_csc), not part of a step"}


def cpu_baseline(p, csc, budget, stride=0):
    """The fp64 oracle as it stands, on every k-th row of each side (k chosen so the sample has
    about `budget` algorithmic flops, or `stride`), extrapolated to a full half-sweep pair by
    the algorithmic flop count."""
    import oracle
    orc = oracle.get()
    f = p.f
    if stride <= 0:
        full = 0.0
        for rp in (p.rowptr, csc[0]):
            cnt = np.diff(rp)
            full += float(cnt.sum() * F_h(f) + (cnt > 0).sum() * F_s(f))
        stride = max(1, int(round(full / budget)))
    colptr, rowidx, vt = csc
    theta = p.theta0.astype(np.float64)
    xin = np.zeros((p.m, f))  # the item side's input factor: any fixed values time the same
    xin[:] = 0.01
    total_t, total_frac_t, full_pair = 0.0, 0.0, 0.0
    sides = [(p.rowptr, p.colidx, p.vals, p.m, p.n, theta), (colptr, rowidx, vt, p.n, p.m, xin)]
    for rp, ci, v, m, n, th in sides:
        rows = np.arange(0, m, stride, dtype=np.int64)
        cnt = np.diff(rp)
        flops_sample = float((cnt[rows] * F_h(f)).sum() + (cnt[rows] > 0).sum() * F_s(f))
        flops_full = float(cnt.sum() * F_h(f) + (cnt > 0).sum() * F_s(f))
        t0 = time.perf_counter()
        orc.half_sweep(rp, ci, v, m, n, f, p.lam, th, rows=rows)
        dt = time.perf_counter() - t0
        total_frac_t += dt
        total_t += dt * flops_full / flops_sample
        full_pair += flops_full
    threads = orc.threads()
    # one core: the first 10,000 user rows on a single thread
    k1 = min(10000, p.m)
    rows1 = np.arange(k1, dtype=np.int64)
    cnt = np.diff(p.rowptr)
    fl1 = float((cnt[:k1] * F_h(f)).sum() + (cnt[:k1] > 0).sum() * F_s(f))
    orc.set_threads(1)
    try:
        t0 = time.perf_counter()
        orc.half_sweep(p.rowptr, p.colidx, p.vals, p.m, p.n, f, p.lam, theta, rows=rows1)
        dt1 = time.perf_counter() - t0
    finally:
        orc.set_threads(threads)
    return {
        "value": 2.0 / total_t, "unit": "half-sweeps/s", "cores": threads, "kind": "oracle",
        "sample": f"fp64 oracle on every {stride}-th row of each side ({total_frac_t:.1f} s measured),"
                  f" extrapolated by algorithmic flops to one user + one item half-sweep",
        "gflops": round(full_pair / total_t / 1e9, 2),
        "one_core": {"rows": k1, "seconds": round(dt1, 2), "gflops": round(fl1 / dt1 / 1e9, 3),
                     "sample": f"first {k1} user rows on 1 thread"},
    }


def driver_bench(args):
    """The driver (test RMSE per iteration, async checkpoints) on the workload's training split."""
    import shutil
    import tempfile
    import torch
    import synth
    from paper_1603_03820_amd import als, driver

    dev = torch.device("cuda", 0)
    p = synth.config(args.config, f=args.f)
    (tr, te) = synth.split(p.rowptr, p.colidx, p.vals, args.test_frac, p.recipe["seed"])
    ctx = als.Context(0, max(p.f, 16))
    dp = driver.DeviceProblem.from_host_csr(ctx, p.m, p.n, p.f, p.lam, *tr)   # CSC on the device
    test = driver.RatingSet.from_host(p.m, p.n, *te, dev)
    th0 = torch.from_numpy(p.theta0).to(dev)
    iters = args.steps
    driver.run(ctx, dp, th0, args.warmup, test=test)             # warm-up
    _, _, plain = driver.run(ctx, dp, th0, iters, test=test)
    tmp = tempfile.mkdtemp(prefix="als_ckpt_")
    try:
        ck = driver.AsyncCheckpointer(tmp, torch.empty((p.m, p.f), device=dev), th0)
        t0 = time.perf_counter()
        _, _, with_ck = driver.run(ctx, dp, th0, iters, test=test, checkpointer=ck,
                                   checkpoint_every=args.checkpoint_every)
        t_ck = time.perf_counter() - t0
        files = list(ck.saved)
        ck_bytes = 4 * (p.m + p.n) * p.f
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    wall = plain[-1]["wall_s"]
    out = {
        "metric": "ALS iterations/s with training and held-out test RMSE per iteration",
        "value": round(iters / wall, 3), "unit": "iterations/s", "n_gpus": 1, "steps": iters,
        "warmup": args.warmup, "higher_is_better": True, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{p.name} training split: m={p.m} n={p.n} "
                               f"nnz={int(tr[0][-1])} (test {int(te[0][-1])}) f={p.f} "
                               f"lambda={p.lam}", "test_frac": args.test_frac},
        "curve": [{k: (round(v, 6) if isinstance(v, float) else v) for k, v in h.items()}
                  for h in plain],
        "checkpoint": {"every": args.checkpoint_every, "files": len(files),
                       "bytes_each": ck_bytes,
                       "wall_s_with": round(t_ck, 4), "wall_s_without": round(wall, 4),
                       "overhead_ms_per_iteration": round((t_ck - wall) / iters * 1e3, 3),
                       "same_rmse": [h["test_rmse"] for h in with_ck] ==
                                    [h["test_rmse"] for h in plain]},
    }
    print(json.dumps(out), flush=True)


def stream_bench(args):
    """Half-sweeps with each side of R streamed from pinned host memory (row batches)."""
    import torch
    import synth
    from paper_1603_03820_amd import als, driver, stream

    dev = torch.device("cuda", 0)
    p = synth.config(args.config, f=args.f)
    csc = p.csc()
    f = p.f
    ctx = als.Context(0, max(f, 16))
    sw_u = stream.StreamedSweep(ctx, stream.HostCSR(p.rowptr, p.colidx, p.vals), p.n, f,
                                args.batch_entries)
    sw_i = stream.StreamedSweep(ctx, stream.HostCSR(*csc), p.m, f, args.batch_entries)
    theta = torch.from_numpy(p.theta0).to(dev)
    x = torch.empty((p.m, f), dtype=torch.float32, device=dev)

    def step():
        sw_u.half_sweep(p.lam, theta, x)
        sw_i.half_sweep(p.lam, x, theta)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    b0 = sw_u.h2d_bytes + sw_i.h2d_bytes
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    h2d = sw_u.h2d_bytes + sw_i.h2d_bytes - b0
    # reference: one pinned 1 GiB host-to-device copy, and the resident half-sweeps
    src = torch.empty(1 << 28, dtype=torch.float32).pin_memory()
    dst = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    copy_gbs = (1 << 30) / (time.perf_counter() - t1) / 1e9
    del src, dst
    dp = driver.DeviceProblem.from_host(p.m, p.n, f, p.lam, p.rowptr, p.colidx, p.vals, *csc,
                                        dev)
    driver.update_x(ctx, dp, theta, x)
    driver.update_theta(ctx, dp, x, theta)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        driver.update_x(ctx, dp, theta, x)
        driver.update_theta(ctx, dp, x, theta)
    torch.cuda.synchronize()
    resident = 2.0 * args.steps / (time.perf_counter() - t2)
    out = {
        "metric": "ALS half-sweeps/s with R streamed from pinned host memory (PCIe-inclusive)",
        "value": round(2.0 * args.steps / el, 3), "unit": "half-sweeps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "higher_is_better": True, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{p.name}: m={p.m} n={p.n} nnz={p.nnz} f={f} lambda={p.lam}",
                   "batch_entries": args.batch_entries,
                   "batches": {"user": len(sw_u.batches), "item": len(sw_i.batches)}},
        "h2d_bytes_per_step": h2d // args.steps,
        "h2d_gbs_achieved": round(h2d / el / 1e9, 2),
        "h2d_gbs_pinned_copy": round(copy_gbs, 2),
        "resident_half_sweeps_per_s": round(resident, 3),
    }
    print(json.dumps(out), flush=True)


def ablation_bench(args):
    """User and item half-sweeps under each design alternative the library can select (each a
    context created under its environment setting): the gather (bounded buffer loads straight
    into MFMA operands; 64-bit global loads, the analogue of the paper's texture-cache ablation;
    theta rows staged through LDS, the analogue of its shared-memory staging), the last block
    column (quad form vs 16x16 tiles), and where A_u accumulates (registers for the whole row vs
    device memory every 16 ratings, the analogue of the paper's register ablation)."""
    import torch
    import synth
    from paper_1603_03820_amd import als, driver

    dev = torch.device("cuda", 0)
    p = synth.config(args.config, f=args.f)
    csc = p.csc()
    f = p.f
    dp = driver.DeviceProblem.from_host(p.m, p.n, f, p.lam, p.rowptr, p.colidx, p.vals, *csc,
                                        dev)
    theta0 = torch.from_numpy(p.theta0).to(dev)
    x = torch.empty((p.m, f), dtype=torch.float32, device=dev)
    th = torch.empty_like(theta0)
    variants = [
        ("buffer", "quad", "registers", {}),
        ("buffer", "tiles", "registers", {"ALS_LAST_BLOCK": "tiles"}),
        ("global", "quad", "registers", {"ALS_GATHER": "global"}),
        ("global", "tiles", "registers", {"ALS_GATHER": "global", "ALS_LAST_BLOCK": "tiles"}),
        ("lds-staged", "tiles", "registers", {"ALS_GATHER": "lds"}),
        ("buffer", "quad", "memory every 16 ratings", {"ALS_PART_ENTRIES": "16"}),
    ]
    rows = []
    for gather, last, accum, env in variants:
        keys = ("ALS_GATHER", "ALS_LAST_BLOCK", "ALS_PART_ENTRIES")
        saved = {k: os.environ.get(k) for k in keys}
        for k in keys:
            os.environ.pop(k, None)
        os.environ.update(env)
        try:
            ctx = als.Context(0, max(f, 16))
        finally:
            for k, v in saved.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
        for _ in range(args.warmup):
            driver.update_x(ctx, dp, theta0, x)
            driver.update_theta(ctx, dp, x, th)
        torch.cuda.synchronize()
        als.als_profile_begin(ctx, 2 * args.steps)
        for _ in range(args.steps):
            driver.update_x(ctx, dp, theta0, x)
            driver.update_theta(ctx, dp, x, th)
        torch.cuda.synchronize()
        prof = np.array([sum(pr) for pr in als.als_profile_end(ctx, 2 * args.steps)])
        prof = prof.reshape(-1, 2)
        rows.append({"gather": gather, "last_block": last, "accumulation": accum,
                     "env": env,
                     "user_ms": round(float(np.median(prof[:, 0])), 4),
                     "item_ms": round(float(np.median(prof[:, 1])), 4)})
        print(f"[bench] ablation {gather}/{last}/{accum}: {rows[-1]}", file=sys.stderr,
              flush=True)
        ctx.close()
        del ctx
    base = rows[0]["user_ms"] + rows[0]["item_ms"]
    for r in rows:
        r["half_sweep_pair_vs_default"] = round((r["user_ms"] + r["item_ms"]) / base, 4)
    out = {"metric": "ALS half-sweep time under each kernel design alternative (median ms)",
           "value": round(2e3 / base, 3), "unit": "half-sweeps/s (default design)", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
           "dtype": "f32", "data": "synthetic",
           "config": {"workload": f"{p.name}: m={p.m} n={p.n} nnz={p.nnz} f={f} "
                                  f"lambda={p.lam}"},
           "variants": rows}
    print(json.dumps(out), flush=True)


def side_figures(ctx, rowptr_dev, rowptr, m, n, nnz, f, plan_ms, herm_ms, red_ms, tag, side,
                 workload):
    """Per half-sweep side: median times, k_herm_solve's algorithmic rate against the FP32 peak
    and against its own roofline (counter traffic if committed for this workload and source,
    else the compulsory bytes), and the algorithmic Gram / solve split."""
    from paper_1603_03820_amd import als
    cnt = np.diff(rowptr)
    rows = int((cnt > 0).sum())
    bounds, _ = als.als_plan(ctx, rowptr_dev, m, f)
    split = split_rows(bounds.cpu().numpy(), rowptr)
    gram = nnz * F_h(f)
    herm_fl = gram + (rows - split) * F_s(f)
    herm = float(np.median(herm_ms))
    achieved = herm_fl / (herm * 1e-3) / 1e12
    counted = measured_traffic(workload, tag, f"bytes_{side}_launch")
    nbytes = counted if counted is not None else algorithmic_bytes(nnz, m, n, f)
    bound, peak, ai = roofline_bound(herm_fl, nbytes)
    return {
        "half_sweep_ms": round(float(np.median(plan_ms + herm_ms + red_ms)), 4),
        "herm_ms": round(herm, 4), "reduce_ms": round(float(np.median(red_ms)), 4),
        "herm_tflops": round(achieved, 3), "herm_frac_fp32_peak": round(achieved / FP32_PEAK_TFLOPS, 4),
        "roofline": {"bound": bound, "peak_tflops": round(peak, 2), "ai_flop_per_byte": round(ai, 2),
                     "bytes": nbytes, "bytes_source": "counters" if counted is not None
                     else "algorithmic (no counters for this workload and source)",
                     "frac": round(achieved / peak, 4)},
        "flops": {"gram": gram, "solve": rows * F_s(f),
                  "gram_share": round(gram / (gram + rows * F_s(f)), 4)},
        "rows": rows, "split_rows": split,
    }


def time_workload(ctx, dp, theta0, steps, warmup, rowptr, colptr, tag, name):
    """update-X + update-Theta `steps` times (after `warmup`), each half-sweep's three kernels
    timed by the library's HIP events on the stream they run on; both sides' figures."""
    import torch
    from paper_1603_03820_amd import als, driver
    x = torch.empty((dp.m, dp.f), dtype=torch.float32, device=theta0.device)
    th = torch.empty_like(theta0)
    for _ in range(warmup):
        driver.update_x(ctx, dp, theta0, x)
        driver.update_theta(ctx, dp, x, th)
    torch.cuda.synchronize()
    als.als_profile_begin(ctx, 2 * steps)
    for _ in range(steps):
        driver.update_x(ctx, dp, theta0, x)
        driver.update_theta(ctx, dp, x, th)
    torch.cuda.synchronize()
    prof = np.array(als.als_profile_end(ctx, 2 * steps)).reshape(steps, 2, 3)
    assert als.als_status(ctx) == 0
    del x, th
    nnz = int(rowptr[-1])
    workload = f"{name}: m={dp.m} n={dp.n} nnz={nnz} f={dp.f} lambda={dp.lam}"
    user = side_figures(ctx, dp.rowptr, rowptr, dp.m, dp.n, nnz, dp.f, prof[:, 0, 0],
                        prof[:, 0, 1], prof[:, 0, 2], tag, "user", workload)
    item = side_figures(ctx, dp.colptr, colptr, dp.n, dp.m, nnz, dp.f, prof[:, 1, 0],
                        prof[:, 1, 1], prof[:, 1, 2], tag, "item", workload)
    fl = [nnz * F_h(dp.f) + user["rows"] * F_s(dp.f) - user["split_rows"] * F_s(dp.f),
          nnz * F_h(dp.f) + item["rows"] * F_s(dp.f) - item["split_rows"] * F_s(dp.f)]
    pair_ms = user["herm_ms"] + item["herm_ms"]
    pair = (fl[0] + fl[1]) / (pair_ms * 1e-3) / 1e12
    sweeps_ms = user["half_sweep_ms"] + item["half_sweep_ms"]
    return {"workload": workload, "steps": steps,
            "half_sweeps_per_s": round(2e3 / sweeps_ms, 3),
            "herm_pair_tflops": round(pair, 3),
            "herm_pair_frac_fp32_peak": round(pair / FP32_PEAK_TFLOPS, 4),
            "user": user, "item": item}


SHARE_GPUS = 8   # the node size whose one-GPU share is timed


def share_workload(ctx, dp, theta0, steps, rowptr, colptr, name, gpus=SHARE_GPUS):
    """One GPU's share of a G-GPU run at the workload's real shape (rows are independent, so G
    GPUs would take nnz-balanced contiguous row ranges with the other factor replicated): GPU 0's
    rows [0, u1) of the CSR and columns [0, v1) of the CSC, each holding about nnz / G ratings,
    half-swept `steps` times against the whole other factor, timed like time_workload.  Also
    reports the whole matrix's half-sweep per GPU (full / G) for comparison; the gap is what the
    persistent grid loses on 1 / G of the work (the all-gather of the updated factor is not
    run)."""
    import torch
    from paper_1603_03820_amd import als, driver
    nnz = int(rowptr[-1])
    u1 = max(1, int(np.searchsorted(rowptr, nnz / gpus, side="left")))
    v1 = max(1, int(np.searchsorted(colptr, nnz / gpus, side="left")))
    x = torch.empty((dp.m, dp.f), dtype=torch.float32, device=theta0.device)
    driver.update_x(ctx, dp, theta0, x)                   # the replicated X of the item share
    xs = torch.empty((u1, dp.f), dtype=torch.float32, device=theta0.device)
    ts = torch.empty((v1, dp.f), dtype=torch.float32, device=theta0.device)
    user = (dp.rowptr[:u1 + 1], dp.colidx, dp.vals, u1, dp.n, theta0, xs)
    item = (dp.colptr[:v1 + 1], dp.rowidx, dp.vals_t, v1, dp.m, x, ts)
    for sd in (user, item):
        als.als_half_sweep(ctx, *sd[:5], dp.f, dp.lam, sd[5], sd[6])
    torch.cuda.synchronize()
    als.als_profile_begin(ctx, 2 * steps)
    for _ in range(steps):
        for sd in (user, item):
            als.als_half_sweep(ctx, *sd[:5], dp.f, dp.lam, sd[5], sd[6])
    torch.cuda.synchronize()
    prof = np.array(als.als_profile_end(ctx, 2 * steps)).reshape(steps, 2, 3)
    assert als.als_status(ctx) == 0
    out = {"gpus": gpus, "rows_of": "GPU 0 of the node: the first rows of the CSR and the first "
                                    "columns of the CSC, nnz-balanced"}
    for k, (side, sd, ptr) in enumerate((("user", user, rowptr[:u1 + 1]),
                                         ("item", item, colptr[:v1 + 1]))):
        share_nnz = int(ptr[-1])
        w = f"{name} share 1/{gpus} {side}: m={sd[3]} n={sd[4]} nnz={share_nnz} f={dp.f}"
        fig = side_figures(ctx, sd[0], ptr, sd[3], sd[4], share_nnz, dp.f, prof[:, k, 0],
                           prof[:, k, 1], prof[:, k, 2], "share", side, w)
        fig["share_rows"], fig["share_nnz"] = sd[3], share_nnz
        out[side] = fig
    del x, xs, ts
    return out


def other_workloads(args, dev, movie):
    """The other paper-shaped workloads, measured after the headline: the rank sweep on the
    movie-shaped matrix (f = 32, 64, 128, fresh initial factors), the music shape and the
    wiki shape (its CSC built on the device), each timed as time_workload does."""
    import gc
    import torch
    import synth
    from paper_1603_03820_amd import als, driver
    out = {}
    p, dp100 = movie
    wanted = set(args.others.split(","))
    for f in synth.RANK_SWEEP_F:
        if f"movie_f{f}" not in wanted:
            continue
        t0 = time.perf_counter()
        dp = driver.DeviceProblem(p.m, p.n, f, p.lam, dp100.rowptr, dp100.colidx, dp100.vals,
                                  dp100.colptr, dp100.rowidx, dp100.vals_t)
        th0 = torch.from_numpy(synth.normal(synth.RANK_SWEEP_THETA_SEED, synth.THETA0_STREAM,
                                            (p.n, f), synth.THETA0_STD)).to(dev)
        ctx = als.Context(0, max(f, 16))
        r = time_workload(ctx, dp, th0, args.other_steps, 1, p.rowptr, p.csc()[0],
                          f"movie_f{f}", p.name)
        r["wall_s"] = round(time.perf_counter() - t0, 1)
        out[f"movie_f{f}"] = r
        print(f"[bench] movie f={f}: {r['half_sweeps_per_s']} half-sweeps/s", file=sys.stderr,
              flush=True)
        ctx.close()
    for name in ("music", "wiki"):
        if name not in wanted:
            continue
        t0 = time.perf_counter()
        q = synth.config(name)
        ctx = als.Context(0, max(q.f, 16))
        t = lambda a: torch.from_numpy(a).to(dev)  # noqa: E731
        rp, ci, v = t(q.rowptr), t(q.colidx), t(q.vals)
        colptr, rowidx, vt = als.als_csr_to_csc(ctx, rp, ci, v, q.m, q.n, nnz=q.nnz)
        dp = driver.DeviceProblem(q.m, q.n, q.f, q.lam, rp, ci, v, colptr, rowidx, vt)
        gen_s = time.perf_counter() - t0
        colptr_h = colptr.cpu().numpy()
        r = time_workload(ctx, dp, t(q.theta0), args.other_steps, 1, q.rowptr, colptr_h,
                          f"{name}_f{q.f}", q.name)
        if not args.no_share:
            r["share"] = share_workload(ctx, dp, t(q.theta0), args.other_steps, q.rowptr,
                                        colptr_h, q.name)
            for side in ("user", "item"):
                r["share"][side]["full_over_gpus_ms"] = round(
                    r[side]["half_sweep_ms"] / SHARE_GPUS, 4)
        r["wall_s"] = round(time.perf_counter() - t0, 1)
        r["gen_s"] = round(gen_s, 1)
        out[name] = r
        print(f"[bench] {name}: {r['half_sweeps_per_s']} half-sweeps/s", file=sys.stderr,
              flush=True)
        ctx.close()
        del q, rp, ci, v, colptr, rowidx, vt, dp
        gc.collect()
        torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.driver:
        driver_bench(args)
        return
    if args.stream:
        stream_bench(args)
        return
    if args.ablation:
        ablation_bench(args)
        return
    import torch
    import synth
    from paper_1603_03820_amd import als, driver

    assert torch.cuda.is_available(), "bench needs a GPU"
    dev = torch.device("cuda", 0)
    t_gen = time.perf_counter()
    p = synth.config(args.config, f=args.f)
    csc = p.csc()
    t_gen = time.perf_counter() - t_gen
    f = p.f
    dp = driver.DeviceProblem.from_host(p.m, p.n, f, p.lam, p.rowptr, p.colidx, p.vals, *csc, dev)
    theta = torch.from_numpy(p.theta0).to(dev)
    x = torch.empty((p.m, f), dtype=torch.float32, device=dev)
    rmse = torch.empty(1, dtype=torch.float64, device=dev)
    ctx = als.Context(0, max(f, 16))

    if args.pmc_pass:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)   # 1 GiB
        b = torch.empty_like(a)
        a.fill_(1.0)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
        driver.update_x(ctx, dp, theta, x)
        driver.update_theta(ctx, dp, x, theta)
        als.als_rmse(ctx, dp.rowptr, dp.colidx, dp.vals, p.m, p.n, f, x, theta, rmse)
        als.als_csr_to_csc(ctx, dp.rowptr, dp.colidx, dp.vals, p.m, p.n, nnz=p.nnz)
        torch.cuda.synchronize()
        print("pmc pass done", flush=True)
        return

    if not args.serial_rmse:
        # step k: X_k <- update-X(Theta_{k-1}) into xs[k % 2]; Theta_k <- update-Theta(X_k) into
        # ths[k % 2]; then RMSE_k(X_k, Theta_k) on the side stream, where it overlaps step k+1
        # (which only reads Theta_k and writes the other buffers).  Both factors are double-
        # buffered, so only step k+2, which overwrites X_k and Theta_k, waits for RMSE_k.
        ctx_r = als.Context(0, max(f, 16))
        als.als_rmse_waves(ctx_r, 1)
        main_s = torch.cuda.current_stream(dev)
        side_s = torch.cuda.Stream(dev)
        xs = [x, torch.empty_like(x)]
        ths = [torch.empty_like(theta), theta]   # Theta_{-1} (the initial factor) in ths[1]
        theta_ready = [torch.cuda.Event(), torch.cuda.Event()]
        rmse_done = [torch.cuda.Event(), torch.cuda.Event()]
        k_box = [0]
        last_k = args.warmup + args.steps - 1

        def step():
            k = k_box[0]
            xk, th_k = xs[k % 2], ths[k % 2]
            if k >= 2:
                main_s.wait_event(rmse_done[k % 2])
            driver.update_x(ctx, dp, ths[(k - 1) % 2], xk)
            driver.update_theta(ctx, dp, xk, th_k)
            theta_ready[k % 2].record(main_s)
            side_s.wait_event(theta_ready[k % 2])
            # the last step's RMSE has no update-X beside it: full width
            als.als_rmse_waves(ctx_r, 0 if k == last_k else 1)
            als.als_rmse(ctx_r, dp.rowptr, dp.colidx, dp.vals, p.m, p.n, f, xk, th_k, rmse,
                         stream=side_s)
            rmse_done[k % 2].record(side_s)
            k_box[0] = k + 1
    else:
        def step():
            driver.update_x(ctx, dp, theta, x)
            driver.update_theta(ctx, dp, x, theta)
            als.als_rmse(ctx, dp.rowptr, dp.colidx, dp.vals, p.m, p.n, f, x, theta, rmse)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    als.als_profile_begin(ctx, 2 * args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = als.als_profile_end(ctx, 2 * args.steps)
    nonspd = als.als_status(ctx)

    # algorithmic flops
    cnt_u, cnt_i = np.diff(p.rowptr), np.diff(csc[0])
    nnz = p.nnz
    fl_user = nnz * F_h(f) + (cnt_u > 0).sum() * F_s(f)
    fl_item = nnz * F_h(f) + (cnt_i > 0).sum() * F_s(f)
    fl_step = float(fl_user + fl_item)
    ms_step = elapsed * 1e3 / args.steps
    half_sweeps_s = 2.0 * args.steps / elapsed
    gflops = fl_step / (elapsed / args.steps) / 1e9

    # dominant kernel: herm_solve (all Gram flops + the solves of rows it finishes)
    bu, (C_u, _, _, _, W_u, _) = als.als_plan(ctx, dp.rowptr, p.m, f)
    bi, (C_i, _, _, _, W_i, _) = als.als_plan(ctx, dp.colptr, p.n, f)
    split_u = split_rows(bu.cpu().numpy(), p.rowptr)
    split_i = split_rows(bi.cpu().numpy(), csc[0])
    herm_fl = [nnz * F_h(f) + ((cnt_u > 0).sum() - split_u) * F_s(f),
               nnz * F_h(f) + ((cnt_i > 0).sum() - split_i) * F_s(f)]
    herm_ms = np.array([pr[1] for pr in prof]).reshape(-1, 2)      # [step, side]
    plan_ms = np.array([pr[0] for pr in prof]).reshape(-1, 2)
    red_ms = np.array([pr[2] for pr in prof]).reshape(-1, 2)
    herm_avg_ms = float(herm_ms.mean())
    sweep_ms = plan_ms + herm_ms + red_ms                              # per half-sweep, [step, side]
    herm_avg_fl = float(np.mean(herm_fl))
    achieved = herm_avg_fl / (herm_avg_ms * 1e-3) / 1e12
    workload = f"{p.name}: m={p.m} n={p.n} nnz={nnz} f={f} lambda={p.lam}"
    traffic = measured_traffic(workload)
    # the bound: min(FP32 peak, HBM peak x AI), AI from the counter bytes when they were taken
    # on this workload and kernel source, else from the compulsory bytes
    ai_bytes = traffic if traffic is not None else float(np.mean(
        [algorithmic_bytes(nnz, p.m, p.n, f), algorithmic_bytes(nnz, p.n, p.m, f)]))
    bound, _, ai = roofline_bound(herm_avg_fl, ai_bytes)
    if bound == "mfma":
        ach, peak, unit = achieved, FP32_PEAK_TFLOPS, "TFLOP/s"
    else:
        ach, peak, unit = ai_bytes / (herm_avg_ms * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s"
    roofline = {
        "kernel": f"k_herm_solve<{(f + 15) // 16}> (Gram via fp32 MFMA + in-register Cholesky)",
        "bound": bound, "achieved": round(ach, 3), "peak": peak,
        "unit": unit, "frac": round(ach / peak, 4),
        "traffic": traffic,
        "ai_flop_per_byte": round(ai, 2),
        "ai_bytes": "counters" if traffic is not None else "algorithmic",
        "avg_launch_ms": round(herm_avg_ms, 4),
        "flops_per_launch": herm_avg_fl,
        "tflops": round(achieved, 3),
    }

    out = {
        "metric": METRIC,
        "value": round(half_sweeps_s, 3),
        "unit": "half-sweeps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workload,
                   "m": p.m, "n": p.n, "nnz": nnz, "f": f, "lambda": p.lam,
                   "step": "update-X + update-Theta + training RMSE" + (
                       " (each RMSE on a second stream, beside the next update-X)"
                       if not args.serial_rmse else ""),
                   "recipe": {k: v for k, v in p.recipe.items() if k not in ("m", "n", "nnz")}},
        "gflops": round(gflops, 1),
        "pct_fp32_peak": round(100.0 * gflops / 1e3 / FP32_PEAK_TFLOPS, 2),
        "ms": {"user_sweep": round(float((plan_ms + herm_ms + red_ms)[:, 0].mean()), 4),
               "item_sweep": round(float((plan_ms + herm_ms + red_ms)[:, 1].mean()), 4),
               "herm_user": round(float(herm_ms[:, 0].mean()), 4),
               "herm_item": round(float(herm_ms[:, 1].mean()), 4),
               "reduce_user": round(float(red_ms[:, 0].mean()), 4),
               "reduce_item": round(float(red_ms[:, 1].mean()), 4),
               "plan": round(float(plan_ms.mean()), 4)},
        "half_sweep_ms": {side: {"median": round(float(np.median(sweep_ms[:, k])), 4),
                                 "min": round(float(sweep_ms[:, k].min()), 4)}
                          for k, side in enumerate(("user", "item"))},
        "waves": {"user": W_u, "item": W_i, "chunks_user": C_u, "chunks_item": C_i,
                  "split_rows_user": split_u, "split_rows_item": split_i},
        "nonspd_rows": nonspd,
        "train_rmse": float(rmse.item()),
        "roofline": roofline,
        "gen_s": round(t_gen, 1),
    }
    out["csc_build"] = csc_build(ctx, dp, p)
    if not args.no_share:
        out["share"] = share_workload(ctx, dp, torch.from_numpy(p.theta0).to(dev),
                                      max(3, min(args.steps, 10)),
                                      p.rowptr, csc[0], p.name)
        for k, side in enumerate(("user", "item")):
            out["share"][side]["full_over_gpus_ms"] = round(
                float(np.median(sweep_ms[:, k])) / SHARE_GPUS, 4)
    if not args.no_peaks:
        out["peaks_measured"] = measure_peaks(dev)
        roofline["frac_of_measured_mfma"] = round(
            achieved / out["peaks_measured"]["mfma_f32_tflops"], 4)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(p, csc, args.cpu_flops, args.cpu_stride)
    if not args.no_others and p.name == "movie":
        torch.cuda.synchronize()
        try:
            out["workloads"] = other_workloads(args, dev, (p, dp))
        except Exception as e:   # the headline line is printed whatever happens here
            out["workloads_error"] = f"{type(e).__name__}: {e}"
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
