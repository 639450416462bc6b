"""HIP half-sweep against the fp64 oracle, through the C ABI, on seeded synthetic inputs.

Bar (per factor row): max_i |x_gpu - x_oracle| / max(max_i |x_oracle|, 1e-6 max |x_oracle|)
<= 1e-3, the oracle fed the same fp32 inputs promoted to fp64.  Integer work (the partition)
is compared bit for bit.  Item-side inputs are synthetic factors from the generator, never
the GPU's own output.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import gpu_half_sweep, log, row_rel_err, to_dev

pytestmark = pytest.mark.gpu

TOL = 1e-3


@pytest.fixture(scope="module")
def ctx():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    return als.Context(0, 128)


@pytest.fixture(scope="module")
def orc():
    return oracle.get()


def synthetic_factor(rows, f, seed, std):
    return synth.normal(seed, 8, (rows, f), std)


def check_lockstep(ctx, orc, rowptr, colidx, vals, m, n, f, lam, theta, label, rows=None):
    log(f"{label}: half-sweep m={m} n={n} nnz={int(rowptr[-1])} f={f} lam={lam}")
    xg = gpu_half_sweep(ctx, rowptr, colidx, vals, m, n, f, lam, theta)
    xo, st = orc.half_sweep(rowptr, colidx, vals, m, n, f, lam,
                            np.asarray(theta, np.float64), rows=rows)
    if rows is not None:
        xg = xg[rows]
    assert not np.isnan(xg).any(), f"{label}: unwritten or NaN rows"
    err = row_rel_err(xg, xo)
    worst = int(np.argmax(err))
    assert err.max() <= TOL, f"{label}: row {worst} rel err {err.max():.3e}"
    return xg, err


def test_tiny_config_lockstep(ctx, orc):
    p = synth.config("tiny")
    check_lockstep(ctx, orc, p.rowptr, p.colidx, p.vals, p.m, p.n, p.f, p.lam, p.theta0,
                   "tiny user side")
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, p.f, p.recipe["seed"], 0.3)
    check_lockstep(ctx, orc, colptr, rowidx, vt, p.n, p.m, p.f, p.lam, xin, "tiny item side")


# every column-block count (NB = 1..9) and every residue of f mod 16 (the last block's real
# columns: tile form, quad form with no or one theta quad, the light last-block factor)
RANKS = [1, 2, 3, 5, 7, 16, 17, 20, 22, 31, 32, 33, 40, 57, 64, 74, 91, 100, 108, 109, 126,
         127, 128]
assert {f % 16 for f in RANKS} == set(range(16)) and {f // 16 + 1 for f in RANKS} == set(range(1, 10))


@pytest.mark.parametrize("f", RANKS)
def test_rank_lockstep_movie_shaped(ctx, orc, f):
    # a scaled-down movie-shaped matrix: long item rows get cut across waves
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                   plant_f=16, seed=777)
    check_lockstep(ctx, orc, p.rowptr, p.colidx, p.vals, p.m, p.n, f, 0.05, p.theta0,
                   f"movie-small f={f} user")
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, f, 778, 1.0 / np.sqrt(f))
    check_lockstep(ctx, orc, colptr, rowidx, vt, p.n, p.m, f, 0.05, xin,
                   f"movie-small f={f} item")


def _handmade(lengths, n, seed):
    rng = np.random.default_rng(seed)
    rowptr = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    cols = [np.sort(rng.choice(n, size=k, replace=False)) for k in lengths]
    colidx = np.concatenate(cols).astype(np.int32) if cols else np.zeros(0, np.int32)
    vals = rng.uniform(1, 5, size=int(rowptr[-1])).astype(np.float32)
    return rowptr, colidx, vals


@pytest.mark.parametrize("f", [5, 16, 100, 128])
def test_edge_row_lengths(ctx, orc, f):
    n = 30_000
    lengths = [0, 1, 2, f - 1, f, f + 1, 3, 15, 16, 17, 47, 48, 49, 95, 96, 97, 63, 64, 65, 0,
               127, 128, 129, 143, 144, 145, 255, 256, 257, 0, 0, 511, 1000, 4095, 4096, 4097,
               20_000, 1, 0]
    lengths = [max(0, k) for k in lengths]
    rowptr, colidx, vals = _handmade(lengths, n, seed=f)
    theta = synthetic_factor(n, f, 91 + f, 0.2)
    xg, _ = check_lockstep(ctx, orc, rowptr, colidx, vals, len(lengths), n, f, 0.05, theta,
                           f"edge lengths f={f}")
    empty = np.array(lengths) == 0
    assert np.all(xg[empty] == 0.0)


@pytest.fixture(scope="module")
def ctx_global():
    """A context that gathers with 64-bit global loads at every size (the form used when
    theta exceeds the buffer-load range)."""
    import os
    from paper_1603_03820_amd import als
    os.environ["ALS_GATHER"] = "global"
    try:
        return als.Context(0, 128)
    finally:
        del os.environ["ALS_GATHER"]


@pytest.fixture(scope="module")
def ctx_tiles():
    """A context that accumulates the last block column with 16x16 tiles even where the quad
    form applies (the design alternative the quad form replaced)."""
    import os
    from paper_1603_03820_amd import als
    os.environ["ALS_LAST_BLOCK"] = "tiles"
    try:
        return als.Context(0, 128)
    finally:
        del os.environ["ALS_LAST_BLOCK"]


@pytest.mark.parametrize("f", [16, 100, 128])
def test_tile_form_of_last_block(ctx_tiles, orc, f):
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                   plant_f=16, seed=779)
    check_lockstep(ctx_tiles, orc, p.rowptr, p.colidx, p.vals, p.m, p.n, f, 0.05, p.theta0,
                   f"tile-form last block movie-small f={f} user")
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, f, 780, 1.0 / np.sqrt(f))
    check_lockstep(ctx_tiles, orc, colptr, rowidx, vt, p.n, p.m, f, 0.05, xin,
                   f"tile-form last block movie-small f={f} item")


@pytest.mark.parametrize("f", [4, 7, 16, 21, 47, 90, 100, 116, 128])
def test_global_gather_form(ctx_global, orc, f):
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                   plant_f=16, seed=777)
    check_lockstep(ctx_global, orc, p.rowptr, p.colidx, p.vals, p.m, p.n, f, 0.05, p.theta0,
                   f"global gather movie-small f={f} user")
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, f, 778, 1.0 / np.sqrt(f))
    check_lockstep(ctx_global, orc, colptr, rowidx, vt, p.n, p.m, f, 0.05, xin,
                   f"global gather movie-small f={f} item")
    lengths = [0, 1, 2, f - 1, f, f + 1, 47, 48, 49, 95, 96, 97, 0, 1000, 4097, 0]
    rowptr, colidx, vals = _handmade(lengths, 20_000, seed=f + 5)
    theta = synthetic_factor(20_000, f, 95 + f, 0.2)
    check_lockstep(ctx_global, orc, rowptr, colidx, vals, len(lengths), 20_000, f, 0.05, theta,
                   f"global gather edge lengths f={f}")


def _env_ctx(**env):
    import os
    from paper_1603_03820_amd import als
    saved = {k: os.environ.get(k) for k in env}
    os.environ.update({k: str(v) for k, v in env.items()})
    try:
        return als.Context(0, 128)
    finally:
        for k, v in saved.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v


@pytest.mark.parametrize("form", ["buffer", "global", "tiles"])
@pytest.mark.parametrize("f", [7, 16, 100, 128])
def test_long_pieces_run_in_parts(orc, f, form):
    """Parts of 32 entries (the default is 65,536): every row and row piece longer than that is
    accumulated part by part and the part sums are added in the wave's slot (the two-level sum
    of a long piece).  Lockstep against the oracle on both sides, in every gather and last-block
    form."""
    env = {"ALS_PART_ENTRIES": 32}
    if form == "global":
        env["ALS_GATHER"] = "global"
    if form == "tiles":
        env["ALS_LAST_BLOCK"] = "tiles"
    c = _env_ctx(**env)
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                   plant_f=16, seed=781)
    check_lockstep(c, orc, p.rowptr, p.colidx, p.vals, p.m, p.n, f, 0.05, p.theta0,
                   f"parts of 32 ({form}) f={f} user")
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, f, 782, 1.0 / np.sqrt(f))
    check_lockstep(c, orc, colptr, rowidx, vt, p.n, p.m, f, 0.05, xin,
                   f"parts of 32 ({form}) f={f} item")
    lengths = [0, 1, 31, 32, 33, 47, 48, 49, 63, 64, 65, 1000, 4097, 0, 20_000]
    rowptr, colidx, vals = _handmade(lengths, 30_000, seed=f + 9)
    theta = synthetic_factor(30_000, f, 97 + f, 0.2)
    check_lockstep(c, orc, rowptr, colidx, vals, len(lengths), 30_000, f, 0.05, theta,
                   f"parts of 32 ({form}) edge lengths f={f}")
    c.close()


@pytest.mark.parametrize("f", [16, 100])
def test_accumulation_through_memory(orc, f):
    """The ablation form of the paper's register accumulation (section 5.2): parts of one
    pipeline group, 16 ratings, so that A_u is accumulated in the wave's slot in device memory
    every 16 ratings instead of staying in registers for the whole row.  Same results."""
    c = _env_ctx(ALS_PART_ENTRIES=16)
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                   plant_f=16, seed=785)
    check_lockstep(c, orc, p.rowptr, p.colidx, p.vals, p.m, p.n, f, 0.05, p.theta0,
                   f"memory accumulation f={f} user")
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, f, 786, 1.0 / np.sqrt(f))
    check_lockstep(c, orc, colptr, rowidx, vt, p.n, p.m, f, 0.05, xin,
                   f"memory accumulation f={f} item")
    c.close()


@pytest.mark.parametrize("f", [4, 16, 32, 100, 128])
def test_lds_staged_gather_form(orc, f):
    """The ablation form of the gather that stages theta rows through LDS (ALS_GATHER=lds; f a
    multiple of 4): lockstep against the oracle on both sides and on edge row lengths."""
    c = _env_ctx(ALS_GATHER="lds")
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                   plant_f=16, seed=787)
    check_lockstep(c, orc, p.rowptr, p.colidx, p.vals, p.m, p.n, f, 0.05, p.theta0,
                   f"lds-staged gather f={f} user")
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, f, 788, 1.0 / np.sqrt(f))
    check_lockstep(c, orc, colptr, rowidx, vt, p.n, p.m, f, 0.05, xin,
                   f"lds-staged gather f={f} item")
    lengths = [0, 1, 2, f - 1, f, f + 1, 47, 48, 49, 95, 96, 97, 0, 1000, 4097, 0]
    rowptr, colidx, vals = _handmade(lengths, 20_000, seed=f + 15)
    theta = synthetic_factor(20_000, f, 99 + f, 0.2)
    check_lockstep(c, orc, rowptr, colidx, vals, len(lengths), 20_000, f, 0.05, theta,
                   f"lds-staged gather edge lengths f={f}")
    c.close()


def test_lds_staged_gather_needs_f_multiple_of_4():
    from paper_1603_03820_amd import als
    c = _env_ctx(ALS_GATHER="lds")
    dev = c.device
    rp = torch.tensor([0, 1], dtype=torch.int64, device=dev)
    ci = torch.tensor([0], dtype=torch.int32, device=dev)
    v = torch.tensor([1.0], dtype=torch.float32, device=dev)
    th = torch.ones(256, dtype=torch.float32, device=dev)
    x = torch.zeros(256, dtype=torch.float32, device=dev)
    with pytest.raises(als.ALSError) as ei:
        als.als_half_sweep(c, rp, ci, v, 1, 1, 7, 0.1, th, x)
    assert ei.value.code == -2
    c.close()


def test_parts_leave_short_pieces_bit_identical(ctx):
    """Pieces no longer than one part run exactly as before: with parts of 65,536 entries (the
    default) and of 2^20, the movie-small half-sweeps are bit-identical."""
    c = _env_ctx(ALS_PART_ENTRIES=1 << 20)
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=100, model="movie",
                   plant_f=16, seed=783)
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, 100, 784, 0.1)
    a = gpu_half_sweep(ctx, colptr, rowidx, vt, p.n, p.m, 100, 0.05, xin)
    b = gpu_half_sweep(c, colptr, rowidx, vt, p.n, p.m, 100, 0.05, xin)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    c.close()


@pytest.mark.parametrize("f", [16, 100])
def test_long_row_in_small_chunks(ctx, orc, f):
    """A very long row at the end of the cost axis is cut by many small chunks; its pieces are
    summed in groups before the solve."""
    from paper_1603_03820_amd import als
    n = 250_000
    lengths = [40, 0, 3, 700] * 50 + [200_000, 5, 0, 90_000, 17]
    rowptr, colidx, vals = _handmade(lengths, n, seed=31 + f)
    m = len(lengths)
    bounds, (C, _, _, _, W, _) = als.als_plan(ctx, to_dev(rowptr, ctx.device), m, f)
    b = bounds.cpu().numpy()
    nus = np.diff(rowptr)
    cut = [(u, k) for u, k in b[1:C] if u < m and 0 < k < nus[u]]
    runs = np.bincount([u for u, _ in cut], minlength=m)
    log(f"long-row plan: C={C} W={W} longest run of cuts {runs.max()}")
    assert runs.max() > 16, "the grouped reduce must be exercised"
    theta = synthetic_factor(n, f, 300 + f, 0.1)
    check_lockstep(ctx, orc, rowptr, colidx, vals, m, n, f, 0.05, theta,
                   f"long rows in small chunks f={f}")


def test_partition_bit_exact(ctx, orc):
    from paper_1603_03820_amd import als
    cases = []
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=100, model="movie",
                   plant_f=16, seed=777)
    cases.append((p.rowptr, 100))
    cases.append((p.csc()[0], 100))
    cases.append((p.csc()[0], 16))
    cases.append((np.zeros(9, np.int64), 64))
    cases.append((np.array([0, 5, 5, 10_000, 10_001], np.int64), 128))
    for rowptr, f in cases:
        m = len(rowptr) - 1
        log(f"plan m={m} nnz={int(rowptr[-1])} f={f}")
        bounds, (C, c_nnz, c_row, q, W, tail_div) = als.als_plan(ctx, to_dev(rowptr, ctx.device),
                                                                 m, f)
        torch.cuda.synchronize()
        assert C > W >= 1
        ref = orc.partition(rowptr, m, W, c_nnz, c_row, q, C=C, tail_div=tail_div)
        assert np.array_equal(bounds.cpu().numpy(), ref)


def test_deterministic(ctx):
    p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=100, model="movie",
                   plant_f=16, seed=777)
    colptr, rowidx, vt = p.csc()
    xin = synthetic_factor(p.m, 100, 5, 0.1)
    a = gpu_half_sweep(ctx, colptr, rowidx, vt, p.n, p.m, 100, 0.05, xin)
    b = gpu_half_sweep(ctx, colptr, rowidx, vt, p.n, p.m, 100, 0.05, xin)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_not_spd_rows_are_nan_and_counted(ctx):
    from paper_1603_03820_amd import als
    # lambda = 0; columns 0..99 have theta_v[3:] = 0 exactly, so a row rating only those has an
    # exactly singular Gram matrix (a zero pivot); columns 100..199 are generic.
    f, n = 8, 200
    theta = synthetic_factor(n, f, 17, 0.5)
    theta[:100, 3:] = 0.0
    rng = np.random.default_rng(4)
    rows = [np.sort(rng.choice(100, 3, replace=False)),
            np.sort(100 + rng.choice(100, 40, replace=False)),
            np.zeros(0, np.int64),
            np.array([7])]
    rowptr = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int64)
    colidx = np.concatenate(rows).astype(np.int32)
    vals = rng.uniform(1, 5, len(colidx)).astype(np.float32)
    als.als_status(ctx)   # clear
    x = gpu_half_sweep(ctx, rowptr, colidx, vals, 4, n, f, 0.0, theta, sentinel=7.0)
    assert np.all(np.isnan(x[0])) and np.all(np.isnan(x[3]))
    assert np.all(np.isfinite(x[1])) and np.all(x[2] == 0.0)
    assert als.als_status(ctx) == 2
    assert als.als_status(ctx) == 0


def test_overflowing_gram_is_nan_and_counted(ctx):
    """A Gram matrix that overflows fp32 (theta entries of 1e20: squares of 1e40) has a +inf
    pivot; the row is NaN and counted, not solved to a finite wrong value."""
    from paper_1603_03820_amd import als
    for f in (8, 100):
        n = 300
        theta = synthetic_factor(n, f, 23 + f, 0.5)
        # columns 0..19: every entry at least 1e20, so every product of two overflows fp32
        theta[:20] = np.float32(1e20) * (1.0 + np.abs(theta[:20]))
        rng = np.random.default_rng(5)
        rows = [np.sort(rng.choice(20, 4, replace=False)),           # only overflowing columns
                np.sort(20 + rng.choice(n - 20, 150, replace=False)),  # generic
                np.array([3, 40, 41, 200]),                            # one overflowing column
                np.zeros(0, np.int64)]
        rowptr = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int64)
        colidx = np.concatenate(rows).astype(np.int32)
        vals = rng.uniform(1, 5, len(colidx)).astype(np.float32)
        als.als_status(ctx)   # clear
        log(f"overflowing Gram f={f}")
        x = gpu_half_sweep(ctx, rowptr, colidx, vals, 4, n, f, 0.05, theta, sentinel=7.0)
        assert np.all(np.isnan(x[0])) and np.all(np.isnan(x[2])), f
        assert np.all(np.isfinite(x[1])) and np.all(x[3] == 0.0), f
        assert als.als_status(ctx) == 2, f


def test_empty_inputs(ctx):
    from paper_1603_03820_amd import als
    dev = ctx.device
    # every row empty
    rowptr = np.zeros(6, np.int64)
    # (one-element index/value arrays: rowptr says there are no entries, none is read)
    x = gpu_half_sweep(ctx, rowptr, np.zeros(1, np.int32), np.zeros(1, np.float32), 5, 3, 4,
                       0.1, np.ones((3, 4), np.float32), sentinel=3.0)
    assert np.all(x == 0.0)
    # m = 0 is a no-op
    z = torch.zeros(1, dtype=torch.int64, device=dev)
    e = torch.zeros(1, dtype=torch.int32, device=dev)
    v = torch.zeros(1, dtype=torch.float32, device=dev)
    th = torch.ones(12, dtype=torch.float32, device=dev)
    xo = torch.zeros(4, dtype=torch.float32, device=dev)
    als.als_half_sweep(ctx, z, e, v, 0, 3, 4, 0.1, th, xo)
    out = als.als_rmse(ctx, torch.zeros(6, dtype=torch.int64, device=dev), e, v, 5, 3, 4,
                       torch.zeros(20, dtype=torch.float32, device=dev), th)
    assert out.item() == 0.0


def test_argument_errors(ctx):
    from paper_1603_03820_amd import als
    dev = ctx.device
    rp = torch.tensor([0, 1], dtype=torch.int64, device=dev)
    ci = torch.tensor([0], dtype=torch.int32, device=dev)
    v = torch.tensor([1.0], dtype=torch.float32, device=dev)
    th = torch.ones(256, dtype=torch.float32, device=dev)
    x = torch.zeros(256, dtype=torch.float32, device=dev)

    def code(fn):
        with pytest.raises(als.ALSError) as ei:
            fn()
        return ei.value.code

    assert code(lambda: als.als_half_sweep(ctx, rp, ci, v, 1, 1, 0, 0.1, th, x)) == -2
    assert code(lambda: als.als_half_sweep(ctx, rp, ci, v, 1, 1, 129, 0.1, th, x)) == -2
    assert code(lambda: als.als_half_sweep(ctx, rp, ci, v, 1, 1, 4, -1.0, th, x)) == -1
    assert code(lambda: als.als_half_sweep(ctx, rp, ci, v, 1, 1, 4, float("nan"), th, x)) == -1
    assert code(lambda: als.als_half_sweep(ctx, rp, ci, v, 1, 1, 4, 0.1, th, th[2:])) == -6
    assert code(lambda: als.als_half_sweep(ctx, rp, ci, v, -1, 1, 4, 0.1, th, x)) == -1
    # a float pointer one byte off its natural alignment
    bad = torch.zeros(64, dtype=torch.uint8, device=dev)
    import ctypes
    rc = als._lib.als_half_sweep(ctx.handle, ctypes.c_void_p(rp.data_ptr()),
                                 ctypes.c_void_p(ci.data_ptr()), ctypes.c_void_p(v.data_ptr()),
                                 1, 1, 4, ctypes.c_float(0.1), ctypes.c_void_p(th.data_ptr()),
                                 ctypes.c_void_p(bad.data_ptr() + 1), None)
    assert rc == -4


@pytest.mark.parametrize("form", ["buffer", "global"])
def test_rmse_matches_oracle(ctx, ctx_global, orc, form):
    """Both gather forms of the RMSE (buffer loads, 64-bit global loads), at widths that end a
    block exactly, inside a block and one past a block."""
    from paper_1603_03820_amd import als
    c = ctx if form == "buffer" else ctx_global
    for f in (4, 7, 33, 100, 124, 128):
        p = synth.make(3_000, 400, 90_000, rows="lognormal", zipf=0.9, f=f, model="movie",
                       plant_f=min(f, 16), seed=31)
        x = synthetic_factor(p.m, f, 32, 0.3)
        th = synthetic_factor(p.n, f, 33, 0.3)
        log(f"rmse {form} f={f}")
        dev = c.device
        out = als.als_rmse(c, to_dev(p.rowptr, dev), to_dev(p.colidx, dev),
                           to_dev(p.vals, dev), p.m, p.n, f, to_dev(x, dev), to_dev(th, dev))
        ref = orc.rmse(p.rowptr, p.colidx, p.vals, p.m, f, x.astype(np.float64),
                       th.astype(np.float64))
        assert abs(out.item() - ref) <= 1e-6 * ref, (form, f, out.item(), ref)


def test_rmse_does_not_depend_on_width(orc):
    """als_rmse at one wave per SIMD (the width that fits beside a half-sweep), at two, and at
    the default width: bit-identical (fixed chunks, fixed order), and within 1e-6 of the oracle.
    Also run at width one on a second stream while a half-sweep of another context runs."""
    from paper_1603_03820_amd import als
    p = synth.make(20_000, 3_000, 1_500_000, rows="lognormal", zipf=0.9, f=100, model="movie",
                   seed=35)
    x = synthetic_factor(p.m, 100, 36, 0.3)
    th = synthetic_factor(p.n, 100, 37, 0.3)
    ref = orc.rmse(p.rowptr, p.colidx, p.vals, p.m, 100, x.astype(np.float64),
                   th.astype(np.float64))
    c = als.Context(0, 100)
    dev = c.device
    rp, ci, v = to_dev(p.rowptr, dev), to_dev(p.colidx, dev), to_dev(p.vals, dev)
    xd, td = to_dev(x, dev), to_dev(th, dev)
    got = {}
    for w in (0, 1, 2, 8):
        log(f"rmse width {w}")
        als.als_rmse_waves(c, w)
        got[w] = als.als_rmse(c, rp, ci, v, p.m, p.n, 100, xd, td).item()
    assert len({np.float64(g).tobytes() for g in got.values()}) == 1, got
    assert abs(got[0] - ref) <= 1e-6 * ref, (got[0], ref)
    # beside a half-sweep on another stream (another context: its own workspace)
    log("rmse width 1 beside a half-sweep")
    h = als.Context(0, 100)
    xo = torch.empty((p.m, 100), dtype=torch.float32, device=dev)
    side = torch.cuda.Stream(dev)
    als.als_rmse_waves(c, 1)
    torch.cuda.synchronize()
    als.als_half_sweep(h, rp, ci, v, p.m, p.n, 100, p.lam, td, xo)
    with torch.cuda.stream(side):
        out = als.als_rmse(c, rp, ci, v, p.m, p.n, 100, xd, td, stream=side)
    torch.cuda.synchronize()
    assert np.float64(out.item()).tobytes() == np.float64(got[0]).tobytes()
    with pytest.raises(als.ALSError):
        als.als_rmse_waves(c, 9)
    c.close()
    h.close()


def test_tiny_trajectory_ten_iterations(ctx, orc):
    """Free-running: ten iterations on each side from the same theta0; training RMSE agrees
    within 1e-4 after every iteration."""
    from paper_1603_03820_amd import driver
    p = synth.config("tiny")
    colptr, rowidx, vt = p.csc()
    dp = driver.DeviceProblem.from_host(p.m, p.n, p.f, p.lam, p.rowptr, p.colidx, p.vals,
                                        colptr, rowidx, vt, ctx.device)
    log("tiny trajectory, 10 iterations")
    x, th, hist = driver.train(ctx, dp, to_dev(p.theta0, ctx.device), p.iters)
    theta = p.theta0.astype(np.float64)
    ref = []
    for _ in range(p.iters):
        xo, theta = oracle.iterate(p.rowptr, p.colidx, p.vals, p.m, p.n, p.f, p.lam, theta,
                                   csc=(colptr, rowidx, vt))
        ref.append(orc.rmse(p.rowptr, p.colidx, p.vals, p.m, p.f, xo, theta))
    diff = np.abs(np.array(hist) - np.array(ref))
    assert diff.max() <= 1e-4, (hist, ref)
    assert ref[-1] < ref[0]
