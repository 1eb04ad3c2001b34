"""Pins for the oracle's Adam-style update (Appendix E, Eq. localspsa, with
coupled weight decay added to the estimate before the moments).

* It is torch.optim.Adam with weight_decay = lambda fed the SPSA estimate as
  the gradient (torch's weight decay is the coupled kind, added to the
  gradient before the moments), checked over three consecutive updates;
* the first update from zero moments has the closed form
  m = (1 - beta1) g, v = (1 - beta2) g^2, theta' = theta - lr g / (|g| + delta),
  g = g_hat + lambda theta.
"""
import numpy as np
import pytest
import torch

from paper_2609_37899_amd import synth

L, E, H, B, T, P = 1, 4, 8, 2, 16, 6
HP = dict(beta1=0.9, beta2=0.999, delta=1e-8, weight_decay=1e-4)


def cfg_of(oracle_mod, probe):
    return oracle_mod.make_cfg(1, L, E, H, B, T, P, 0, probe)


@pytest.mark.parametrize("probe", [0, 1])
def test_adam_equals_torch_adam_over_three_updates(oracle_mod, probe):
    cfg = cfg_of(oracle_mod, probe)
    theta = synth.init_theta(1, L, E, H, init_seed=5)[0]
    d = theta.size
    m = np.zeros(d, np.float32)
    v = np.zeros(d, np.float32)
    rng = np.random.default_rng(0)
    lr = float(np.float32(1e-3))        # the learning rate crosses the boundary as fp32
    for t in (1, 2, 3):
        coef = rng.normal(0, 1e-2, P)
        th1, m1, v1, gh = oracle_mod.apply_adam(cfg, theta, m, v, t, 0x50A10000, t, lr, coef,
                                                want_ghat=True, **HP)
        # torch, started from the same (fp32) state
        p = torch.tensor(theta.astype(np.float64), requires_grad=True)
        opt = torch.optim.Adam([p], lr=lr, betas=(HP["beta1"], HP["beta2"]), eps=HP["delta"],
                               weight_decay=HP["weight_decay"])
        p.grad = torch.tensor(gh)
        opt.step()                      # creates the state at step 1 with zero moments
        st = opt.state[p]
        if t > 1:                       # redo from the oracle's moments at step t
            with torch.no_grad():
                p.copy_(torch.tensor(theta.astype(np.float64)))
            st["exp_avg"] = torch.tensor(m.astype(np.float64))
            st["exp_avg_sq"] = torch.tensor(v.astype(np.float64))
            st["step"] = torch.tensor(float(t - 1))
            p.grad = torch.tensor(gh)
            opt.step()
        assert np.array_equal(p.detach().numpy().astype(np.float32), th1) or \
            np.max(np.abs(p.detach().numpy() - th1) / np.maximum(np.abs(th1), 1e-30)) < 2 ** -23
        np.testing.assert_allclose(st["exp_avg"].numpy(), m1, rtol=2 ** -23, atol=0)
        np.testing.assert_allclose(st["exp_avg_sq"].numpy(), v1, rtol=2 ** -23, atol=0)
        assert not np.array_equal(th1, theta)
        theta, m, v = th1, m1, v1


def test_first_update_closed_form(oracle_mod):
    cfg = cfg_of(oracle_mod, 0)
    theta = synth.init_theta(1, L, E, H, init_seed=6)[0]
    d = theta.size
    coef = np.linspace(-0.02, 0.03, P)
    lr = float(np.float32(2e-3))
    th1, m1, v1, gh = oracle_mod.apply_adam(cfg, theta, np.zeros(d, np.float32), np.zeros(d, np.float32), 1,
                                            7, 3, lr, coef, want_ghat=True, **HP)
    g = gh + HP["weight_decay"] * theta.astype(np.float64)
    np.testing.assert_allclose(m1, (1 - HP["beta1"]) * g, rtol=2 ** -23)
    np.testing.assert_allclose(v1, (1 - HP["beta2"]) * g * g, rtol=2 ** -23)
    expect = theta - lr * g / (np.abs(g) + HP["delta"])
    np.testing.assert_allclose(th1, expect, rtol=2 ** -23, atol=lr * 1e-6)
    # the estimate is the plain SPSA one (the SGD path's g_hat)
    _, gh_sgd = oracle_mod.apply_update(cfg, theta, 7, 3, 0.0, coef, want_ghat=True)
    assert np.array_equal(gh, gh_sgd)
