"""Pins for the oracle's forward pass and cross entropy (Appendix C body,
Appendix E loss L_CE(h) = log sum_v exp(w_v . h) - w_y . h)."""
import numpy as np
import pytest
import torch

import torch_reference as tref
from paper_2609_37899_amd import synth


def _cfg(oracle_mod, L, E, H, B, T, P=1, N=1):
    return oracle_mod.make_cfg(N, L, E, H, B, T, P)


@pytest.mark.parametrize("L,E,H", [(1, 32, 64), (2, 16, 24), (3, 8, 12)])
def test_forward_matches_torch_lstm(oracle_mod, L, E, H):
    B, T = 3, 17
    cfg = _cfg(oracle_mod, L, E, H, B, T)
    theta = synth.init_theta(1, L, E, H, init_seed=4)[0] * 3.0   # larger weights: exercise saturation
    data = synth.expert_batches([11], B, T)[0]
    ours = oracle_mod.forward_loss(cfg, theta, data)
    ref = tref.loss(torch.tensor(theta, dtype=torch.float64), L, E, H, data).item()
    assert abs(ours - ref) <= 1e-12 * abs(ref)


def test_zero_weights_give_ln256(oracle_mod):
    cfg = _cfg(oracle_mod, 2, 16, 32, 4, 33)
    d = oracle_mod.param_count(cfg)
    data = synth.expert_batches([3], 4, 33)[0]
    assert abs(oracle_mod.forward_loss(cfg, np.zeros(d, np.float32), data) - np.log(256.0)) < 1e-14


def test_init_loss_near_ln256(oracle_mod):
    cfg = _cfg(oracle_mod, 1, 32, 64, 8, 64)
    theta = synth.init_theta(1, 1, 32, 64)[0]
    data = synth.expert_batches([1], 8, 64)[0]
    assert abs(oracle_mod.forward_loss(cfg, theta, data) - np.log(256.0)) < 5e-2


def test_param_count(oracle_mod):
    # 256 E + sum_l 4H (in_l + H) + 256 H
    for (L, E, H) in [(1, 32, 64), (2, 512, 512), (2, 384, 384), (2, 704, 704)]:
        cfg = _cfg(oracle_mod, L, E, H, 1, 2)
        assert oracle_mod.param_count(cfg) == synth.param_count(L, E, H)
    assert synth.param_count(1, 32, 64) == 49_152
    assert synth.param_count(2, 512, 512) == 4_456_448
    assert synth.param_count(2, 384, 384) == 2_555_904
    assert synth.param_count(2, 704, 704) == 8_290_304


def test_directional_difference_matches_autograd(oracle_mod):
    """The fp64 central difference along z equals z . grad L (autograd) up to
    an O(eps^2) truncation term: below 1e-7 relative at eps = 1e-5, and the
    error shrinks 100x per decade of eps (Appendix G reports directional
    differences within 6e-7 of exact derivatives at eps = 1e-4)."""
    L, E, H, B, T = 2, 8, 12, 2, 16
    cfg = _cfg(oracle_mod, L, E, H, B, T)
    theta = synth.init_theta(1, L, E, H, init_seed=9)[0].astype(np.float64) * 3.0
    data = synth.expert_batches([5], B, T)[0]
    t = torch.tensor(theta, dtype=torch.float64, requires_grad=True)
    tref.loss(t, L, E, H, data).backward()
    g = t.grad.numpy()
    rng = np.random.default_rng(0)
    for _ in range(3):
        z = rng.standard_normal(theta.size)
        errs = []
        for eps in (1e-3, 1e-4, 1e-5):
            lp = oracle_mod.forward_loss_f64(cfg, theta + eps * z, data)
            lm = oracle_mod.forward_loss_f64(cfg, theta - eps * z, data)
            errs.append(abs((lp - lm) / (2 * eps) - z @ g) / abs(z @ g))
        assert errs[2] < 1e-7
        assert 50 < errs[0] / errs[1] < 200


def test_perturb_is_single_rounding_fma(oracle_mod):
    cfg = _cfg(oracle_mod, 1, 32, 64, 1, 2)
    d = oracle_mod.param_count(cfg)
    theta = synth.init_theta(1, 1, 32, 64)[0]
    z = oracle_mod.gaussian(99, 3, 2, 0, d).astype(np.float64)
    for s in (+1, -1):
        eps = np.float32(1e-3)
        w = oracle_mod.perturb(cfg, theta, 99, 3, 2, float(s * eps))
        exact = theta.astype(np.float64) + s * np.float64(eps) * z   # product exact in fp64
        # where the fp64 sum is itself exact, one rounding to fp32 must agree bit for bit
        assert np.array_equal(w, exact.astype(np.float32)) or \
            np.mean(w != exact.astype(np.float32)) < 1e-4
        assert np.all(np.abs(w.astype(np.float64) - exact) <= np.spacing(np.abs(w)) * 0.5 + 1e-30)
