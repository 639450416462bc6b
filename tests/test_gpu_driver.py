"""The ALS driver on the device (NEXT row f1): held-out test RMSE per iteration against the fp64
oracle's trajectory, and asynchronous checkpoints that resume bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_util import log, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    from paper_1603_03820_amd import als
    assert torch.cuda.is_available()
    return als.Context(0, 128)


def _problem(ctx, frac=0.1, seed=17):
    from paper_1603_03820_amd import driver
    p = synth.config("tiny")
    (tr, te) = synth.split(p.rowptr, p.colidx, p.vals, frac, seed)
    csc = synth.transpose(p.m, p.n, *tr)
    dp = driver.DeviceProblem.from_host(p.m, p.n, p.f, p.lam, *tr, *csc, ctx.device)
    test = driver.RatingSet.from_host(p.m, p.n, *te, ctx.device)
    return p, tr, te, csc, dp, test


def test_test_rmse_trajectory_matches_oracle(ctx):
    """Ten iterations on a 90/10 split: training and test RMSE after every iteration within
    1e-4 of the oracle iterating on the same training set in fp64."""
    from paper_1603_03820_amd import driver
    orc = oracle.get()
    p, tr, te, csc, dp, test = _problem(ctx)
    log(f"tiny 90/10 split: train {int(tr[0][-1])}, test {int(te[0][-1])} ratings")
    _, _, hist = driver.run(ctx, dp, to_dev(p.theta0, ctx.device), p.iters, test=test)
    theta = p.theta0.astype(np.float64)
    for h in hist:
        xo, theta = oracle.iterate(*tr, p.m, p.n, p.f, p.lam, theta, csc=csc)
        r_tr = orc.rmse(*tr, p.m, p.f, xo, theta)
        r_te = orc.rmse(*te, p.m, p.f, xo, theta)
        log(f"iter {h['iteration']}: train {h['train_rmse']:.6f}/{r_tr:.6f} "
            f"test {h['test_rmse']:.6f}/{r_te:.6f}")
        assert abs(h["train_rmse"] - r_tr) <= 1e-4
        assert abs(h["test_rmse"] - r_te) <= 1e-4
        assert h["ms"] > 0
    # the held-out error is the larger one, and both fall from the first iteration
    assert hist[-1]["test_rmse"] > hist[-1]["train_rmse"]
    assert hist[-1]["train_rmse"] < hist[0]["train_rmse"]


def test_checkpoint_resume_is_bit_exact(ctx, tmp_path):
    """Checkpoints every 2 iterations while running 6; resuming from iteration 4 for 2 more
    iterations ends on the uninterrupted run's X and Theta bit for bit, and each checkpoint
    holds exactly the factors of that iteration."""
    from paper_1603_03820_amd import driver
    p, tr, te, csc, dp, test = _problem(ctx)
    th0 = to_dev(p.theta0, ctx.device)
    x_like = torch.empty((p.m, p.f), device=ctx.device)
    ck = driver.AsyncCheckpointer(str(tmp_path), x_like, th0)
    log("6 iterations with checkpoints at 2, 4, 6")
    x6, t6, _ = driver.run(ctx, dp, th0, 6, test=test, checkpointer=ck, checkpoint_every=2)
    assert ck.saved == [driver.CHECKPOINT_FILE.format(i) for i in (2, 4, 6)]
    it, x4, t4 = driver.load_checkpoint(str(tmp_path), ctx.device, iteration=4)
    assert it == 4
    xr, tr_, hist = driver.run(ctx, dp, t4, 2, start_iteration=4, x0=x4)
    assert [h["iteration"] for h in hist] == [5, 6]
    assert torch.equal(xr, x6) and torch.equal(tr_, t6)
    x4b, t4b, _ = driver.run(ctx, dp, th0, 4, rmse_every=False)
    assert torch.equal(x4b, x4) and torch.equal(t4b, t4)
    it, xl, tl = driver.load_checkpoint(str(tmp_path), ctx.device)
    assert it == 6 and torch.equal(xl, x6) and torch.equal(tl, t6)


def test_device_built_csc_gives_the_same_run(ctx):
    """DeviceProblem.from_host_csr builds the item side's CSC with als_csr_to_csc: the same CSC
    as the host transpose bit for bit, hence the same ten iterations bit for bit."""
    from paper_1603_03820_amd import driver
    p, tr, te, csc, dp, test = _problem(ctx)
    log("tiny: CSC built on the device")
    dd = driver.DeviceProblem.from_host_csr(ctx, p.m, p.n, p.f, p.lam, *tr)
    assert torch.equal(dd.colptr, dp.colptr) and torch.equal(dd.rowidx, dp.rowidx)
    assert torch.equal(dd.vals_t.view(torch.int32), dp.vals_t.view(torch.int32))
    th0 = to_dev(p.theta0, ctx.device)
    x1, t1, _ = driver.run(ctx, dp, th0, 3)
    x2, t2, _ = driver.run(ctx, dd, th0, 3)
    assert torch.equal(x1, x2) and torch.equal(t1, t2)
