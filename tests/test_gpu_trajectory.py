"""Free-running ALS against the fp64 oracle on the paper-shaped workloads: ten iterations
(update-X then update-Theta, section 2.1) from the same initial factor on each side, the
training RMSE (the evaluation metric of section 5) compared after every iteration.

The GPU iterates in fp32 from its own previous factors and the oracle in fp64 from its own, so
rounding differences accumulate over the iterations; the bar is on the RMSE: within 1e-4 after
every iteration (for the music shape, whose ratings lie on a 0-100 scale, 1e-4 max(1, RMSE)).
The factors after the last iteration are compared per row as well, to the lockstep bar (1e-3).

Sizes: the movie shape at a quarter of its rows and ratings (120,000 x 17,770, 25M ratings,
the same row-length law, column law and n), the music shape at a tenth (100,000 x 625,000,
25M ratings), so that the oracle's ten fp64 iterations take about a minute per workload.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import log, row_rel_err, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    return als.Context(0, 128)


def scaled(name, div):
    c = synth.CONFIGS[name]
    return synth.make(c["m"] // div, c["n"], c["nnz"] // div, rows=c["rows"], mean=c["mean"],
                      zipf=c["zipf"], f=c["f"], lam=c["lam"], model=c["model"], seed=c["seed"],
                      iters=c["iters"], name=f"{name}/{div}")


@pytest.mark.parametrize("name,div", [("movie", 4), ("music", 10)])
def test_ten_iterations_track_the_oracle(ctx, name, div):
    from paper_1603_03820_amd import driver
    orc = oracle.get()
    p = scaled(name, div)
    log(f"{p.name}: m={p.m} n={p.n} nnz={p.nnz} f={p.f} lambda={p.lam}, 10 iterations")
    csc = p.csc()
    dp = driver.DeviceProblem.from_host(p.m, p.n, p.f, p.lam, p.rowptr, p.colidx, p.vals, *csc,
                                        ctx.device)
    x, th, hist = driver.train(ctx, dp, to_dev(p.theta0, ctx.device), 10)
    theta = p.theta0.astype(np.float64)
    worst = 0.0
    for it in range(10):
        xo, theta = oracle.iterate(p.rowptr, p.colidx, p.vals, p.m, p.n, p.f, p.lam, theta,
                                   csc=csc)
        ref = orc.rmse(p.rowptr, p.colidx, p.vals, p.m, p.f, xo, theta)
        d = abs(hist[it] - ref)
        tol = 1e-4 * max(1.0, ref)
        worst = max(worst, d / tol)
        log(f"{p.name} iteration {it + 1}: rmse gpu {hist[it]:.8f} oracle {ref:.8f} "
            f"|diff| {d:.2e} (bar {tol:.1e})")
        assert d <= tol, (it, hist[it], ref)
    assert hist[-1] < hist[0]
    ex = row_rel_err(x.cpu().numpy(), xo)
    et = row_rel_err(th.cpu().numpy(), theta)
    log(f"{p.name} after 10 iterations: max row rel err X {ex.max():.2e} "
        f"(median {np.median(ex):.1e}), Theta {et.max():.2e} (median {np.median(et):.1e}); "
        f"worst RMSE diff / bar {worst:.3f}")
    assert ex.max() <= 1e-3 and et.max() <= 1e-3
