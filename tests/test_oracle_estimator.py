"""Pins for the oracle's SPSA estimator and update.

Closed forms used (Gaussian probes z ~ N(0, I_d); the paper's Prop. 1 in
Appendix F gives the Rademacher analogue (d-1)/n_pert):
  * for small eps the single-direction estimate is z z^T g + O(eps^2) and
    E||z z^T g - g||^2 = (d+1) ||g||^2 (because E z^4 = 3), so with P
    directions  E||g_hat - g||^2 / ||g||^2 = (d+1)/P;
  * summing the losses of N experts (Appendix J) makes each expert's estimate
    carry every expert's probe noise: the ratio of summed to independent
    relative error is (M+1)/(d+1) for M = N d perturbed coordinates;
  * flipping z -> -z swaps L+ and L- and leaves the update unchanged
    (Section 4, Eq. main-spsa is even in z);
  * with independent losses expert e's update reads only its own loss
    (separability, Section 4 and Appendix F).
"""
import numpy as np
import pytest
import torch

import torch_reference as tref
from paper_2609_37899_amd import synth

L, E, H, B, T = 1, 4, 8, 2, 16


def tiny(oracle_mod, N=1, P=4, mode=0):
    return oracle_mod.make_cfg(N, L, E, H, B, T, P, mode)


def exact_grad(theta_e, data_e):
    t = torch.tensor(theta_e.astype(np.float64), requires_grad=True)
    tref.loss(t, L, E, H, data_e).backward()
    return t.grad.numpy()


def test_antithetic_flip_is_bit_identical(oracle_mod):
    cfg = tiny(oracle_mod, N=2, P=3)
    theta = synth.init_theta(2, L, E, H, distinct=True)
    data = synth.expert_batches([1, 2], B, T)
    seeds = synth.expert_seeds(2)
    a = oracle_mod.spsa_step(cfg, theta, seeds, 0, 1e-3, 1e-2, data)
    b = oracle_mod.spsa_step(cfg, theta, seeds, 0, -1e-3, 1e-2, data)
    assert np.array_equal(a["losses"][..., 0], b["losses"][..., 1])
    assert np.array_equal(a["losses"][..., 1], b["losses"][..., 0])
    assert np.array_equal(a["coef"], b["coef"])
    assert np.array_equal(a["theta"], b["theta"])
    assert not np.array_equal(a["theta"], theta)


def test_separability_bit_identity_and_summed_control(oracle_mod):
    theta = synth.init_theta(2, L, E, H, distinct=True)
    seeds = synth.expert_seeds(2)
    d1 = synth.expert_batches([1, 2], B, T)
    d2 = d1.copy()
    d2[1] = synth.expert_batches([77], B, T)[0]          # change expert 1's data only
    ind = tiny(oracle_mod, N=2, P=3, mode=0)
    a = oracle_mod.spsa_step(ind, theta, seeds, 0, 1e-3, 1e-2, d1)
    b = oracle_mod.spsa_step(ind, theta, seeds, 0, 1e-3, 1e-2, d2)
    assert np.array_equal(a["theta"][0], b["theta"][0])
    assert np.array_equal(a["losses"][0], b["losses"][0])
    assert not np.array_equal(a["theta"][1], b["theta"][1])
    summ = tiny(oracle_mod, N=2, P=3, mode=1)
    c = oracle_mod.spsa_step(summ, theta, seeds, 0, 1e-3, 1e-2, d1)
    e = oracle_mod.spsa_step(summ, theta, seeds, 0, 1e-3, 1e-2, d2)
    assert not np.array_equal(c["theta"][0], e["theta"][0])
    # same forwards in both modes; only the reduction differs
    assert np.array_equal(a["losses"], c["losses"])
    # summed coefficient is the sum over experts of the independent ones
    np.testing.assert_allclose(c["coef"][0], a["coef"].sum(axis=0), rtol=1e-12)


def test_zero_lr_leaves_theta_unchanged(oracle_mod):
    cfg = tiny(oracle_mod, P=2)
    theta = synth.init_theta(1, L, E, H)
    out = oracle_mod.spsa_step(cfg, theta, synth.expert_seeds(1), 0, 1e-3, 0.0,
                               synth.expert_batches([1], B, T))
    assert np.array_equal(out["theta"], theta)


@pytest.mark.slow
def test_estimate_converges_to_exact_gradient_at_rate_d_plus_1_over_P(oracle_mod):
    theta = synth.init_theta(1, L, E, H, init_seed=2) * np.float32(3.0)
    data = synth.expert_batches([4], B, T)
    g = exact_grad(theta[0], data[0])
    d = g.size
    ratios = []
    for P in (64, 256, 1024):
        cfg = tiny(oracle_mod, P=P)
        out = oracle_mod.spsa_step(cfg, theta, synth.expert_seeds(1), 1, 1e-3, 1e-3, data,
                                   want_ghat=True)
        err = np.sum((out["ghat"][0] - g) ** 2) / np.sum(g ** 2)
        ratios.append(err * P / (d + 1))
        assert abs(ratios[-1] - 1) < 5 * np.sqrt(2 / P) + 0.02, (P, ratios[-1])
    slope = np.polyfit(np.log([64, 256, 1024]), np.log(np.array(ratios) * (d + 1) / [64, 256, 1024]), 1)[0]
    assert abs(slope + 1) < 0.2


@pytest.mark.slow
def test_summed_to_independent_error_ratio(oracle_mod):
    N, P, R = 2, 16, 48
    theta = synth.init_theta(N, L, E, H, init_seed=3, distinct=True) * np.float32(3.0)
    data = synth.expert_batches([5, 6], B, T)
    G = np.stack([exact_grad(theta[e], data[e]) for e in range(N)])
    d = G.shape[1]
    M = N * d
    errs = {0: [], 1: []}
    means = {0: 0.0, 1: 0.0}
    for mode in (0, 1):
        cfg = tiny(oracle_mod, N=N, P=P, mode=mode)
        for r in range(R):
            out = oracle_mod.spsa_step(cfg, theta, synth.expert_seeds(N, base=1000 * r), r, 1e-3, 1e-3,
                                       data, want_ghat=True)
            errs[mode].append(np.sum((out["ghat"] - G) ** 2) / np.sum(G ** 2))
            means[mode] = means[mode] + out["ghat"] / R
    ratio = np.mean(errs[1]) / np.mean(errs[0])
    pred = (M + 1) / (d + 1)
    assert abs(ratio / pred - 1) < 0.2, (ratio, pred)
    for mode in (0, 1):
        assert abs(np.mean(errs[mode]) * P / (((M if mode else d) + 1)) - 1) < 0.25
        # both modes are unbiased: the mean over R repeats is closer to G than one draw
        assert np.sum((means[mode] - G) ** 2) < np.mean(errs[mode]) * np.sum(G ** 2) / R * 2.5
