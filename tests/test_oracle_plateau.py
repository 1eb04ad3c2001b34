"""Pins for the oracle's plateau schedule of lr and eps (Section 4; Table
experimental-setup).  It is torch's ReduceLROnPlateau in absolute-threshold
mode (a decay when the count of updates without improvement exceeds
patience - 1, i.e. reaches patience; no cooldown; min_lr = floor; a decay
only when it lowers the rate), applied to lr and, identically, to eps."""
import numpy as np
import pytest
import torch

F = np.float32


def torch_schedule(rate0, losses, patience, factor, threshold, floor):
    p = torch.zeros(1, requires_grad=True)
    opt = torch.optim.SGD([p], lr=float(F(rate0)))
    sch = torch.optim.lr_scheduler.ReduceLROnPlateau(opt, mode="min", factor=float(F(factor)),
                                                     patience=patience - 1, threshold=float(F(threshold)),
                                                     threshold_mode="abs", cooldown=0,
                                                     min_lr=float(F(floor)), eps=0.0)
    out = []
    for v in losses:
        sch.step(float(F(v)))
        out.append(opt.param_groups[0]["lr"])
    return np.array(out)


# The paper's threshold (1e-8) is below fp32's spacing near a loss of 5, so
# only the larger thresholds make the curves improve by less than the
# threshold and test that such a step is no improvement.
@pytest.mark.parametrize("patience,threshold", [(1, 1e-8), (3, 1e-8), (7, 1e-8), (3, 5e-4), (2, 2e-3)])
def test_plateau_equals_torch_reduce_on_plateau(oracle_mod, patience, threshold):
    rng = np.random.default_rng(patience)
    n, steps = 3, 400
    # noisy decreasing curves with long flat stretches, per expert
    base = np.cumsum(rng.exponential(1e-3, (steps, n)) * (rng.random((steps, n)) < 0.2), axis=0)
    losses = (5.0 - base + rng.normal(0, 1e-4, (steps, n))).astype(np.float32)
    if threshold > 1e-6:
        # some improvements on the running best fall below the threshold
        best, small = np.full(n, np.inf), 0
        for t in range(steps):
            gain = best - losses[t].astype(np.float64)
            small += int(np.sum((gain > 0) & (gain <= threshold)))
            best = np.minimum(best, losses[t])
        assert small >= 5
    sch = oracle_mod.Plateau(n, 1e-3, 2e-3, factor=0.5, patience=patience, threshold=threshold, floor=1e-5)
    lrs, epss = [], []
    for t in range(steps):
        sch.observe(losses[t])
        lr, eps, best, since = sch.state()
        lrs.append(lr)
        epss.append(eps)
    lrs, epss = np.array(lrs), np.array(epss)
    for e in range(n):
        ref_lr = torch_schedule(1e-3, losses[:, e], patience, 0.5, threshold, 1e-5)
        ref_eps = torch_schedule(2e-3, losses[:, e], patience, 0.5, threshold, 1e-5)
        np.testing.assert_array_equal(lrs[:, e].astype(np.float64), ref_lr.astype(np.float32).astype(np.float64))
        np.testing.assert_array_equal(epss[:, e].astype(np.float64), ref_eps.astype(np.float32).astype(np.float64))
    assert lrs.min() < 1e-3 and lrs.min() >= F(1e-5)       # decays happened, none below the floor


def test_plateau_floor_and_update_counting(oracle_mod):
    sch = oracle_mod.Plateau(1, 3e-5, 8e-6, patience=1000)
    sch.observe([5.0], updates=10)          # first observation improves on +inf
    for _ in range(99):
        sch.observe([5.0], updates=10)      # 990 updates without improvement
    assert sch.state()[0][0] == F(3e-5)
    sch.observe([5.0], updates=10)          # 1,000: decay; eps is already below the floor
    lr, eps, best, since = sch.state()
    assert lr[0] == F(1.5e-5) and eps[0] == F(8e-6) and since[0] == 0 and best[0] == F(5.0)
    for _ in range(100):
        sch.observe([5.0], updates=10)
    assert sch.state()[0][0] == F(1e-5)      # the floor
    sch.observe([float("nan")], updates=10)  # NaN is no improvement
    assert sch.state()[3][0] == 10
    sch.observe([4.99999], updates=10)
    assert sch.state()[2][0] == F(4.99999) and sch.state()[3][0] == 0
