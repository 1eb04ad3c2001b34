"""Pins for the oracle's plain update theta' = theta - lr g_hat (Section 4,
Eq. main-spsa: the estimate drives a gradient step).

* It is torch.optim.SGD(lr) fed the oracle's own estimate g_hat as the
  gradient: a library optimiser, not a retyping of the update, so a flipped
  sign, a dropped or rescaled learning rate, or an update applied to the wrong
  coordinates fails;
* descent: with many directions and a small learning rate the step lowers
  the expected loss, and the decrease matches the first-order prediction
  lr g . g_hat (exact gradient g by autograd in fp64, a different code path
  from the oracle's forward), so a step along +g_hat, or one whose size is not
  lr, fails.
"""
import numpy as np
import pytest
import torch

import torch_reference as tref
from paper_2609_37899_amd import synth

L, E, H, B, T = 1, 4, 8, 2, 16


def test_sgd_step_equals_torch_sgd(oracle_mod):
    N, P = 2, 5
    cfg = oracle_mod.make_cfg(N, L, E, H, B, T, P)
    theta = synth.init_theta(N, L, E, H, init_seed=4, distinct=True)
    data = synth.expert_batches([11, 12], B, T)
    seeds = synth.expert_seeds(N)
    for lr in (1e-2, 0.37, 3.0):
        out = oracle_mod.spsa_step(cfg, theta, seeds, 2, 1e-3, lr, data, want_ghat=True)
        for e in range(N):
            p = torch.nn.Parameter(torch.tensor(theta[e].astype(np.float64)))
            opt = torch.optim.SGD([p], lr=float(np.float32(lr)))   # lr crosses the boundary as fp32
            p.grad = torch.tensor(out["ghat"][e])
            opt.step()
            want = p.detach().numpy().astype(np.float32)
            got = out["theta"][e]
            # one rounding to fp32 on both sides (fp64 products may differ in the last bit)
            ulp = np.spacing(np.abs(want))
            assert np.all(np.abs(got.astype(np.float64) - want) <= ulp), lr
            assert not np.array_equal(got, theta[e])
        # the estimate is the coefficients times the regenerated probes
        z = np.stack([oracle_mod.probe(0, int(seeds[0]), 2, j, 0, theta.shape[1]) for j in range(P)])
        np.testing.assert_allclose(out["ghat"][0], out["coef"][0] @ z.astype(np.float64), rtol=1e-12,
                                   atol=1e-15)


def test_sgd_step_descends_by_the_first_order_prediction(oracle_mod):
    P = 512
    cfg = oracle_mod.make_cfg(1, L, E, H, B, T, P)
    theta = synth.init_theta(1, L, E, H, init_seed=6) * np.float32(3.0)
    data = synth.expert_batches([13], B, T)
    t = torch.tensor(theta[0].astype(np.float64), requires_grad=True)
    l0 = tref.loss(t, L, E, H, data[0])
    l0.backward()
    g = t.grad.numpy()
    lr = 2e-2
    out = oracle_mod.spsa_step(cfg, theta, synth.expert_seeds(1), 0, 1e-3, lr, data, want_ghat=True)
    l1 = float(tref.loss(torch.tensor(out["theta"][0].astype(np.float64)), L, E, H, data[0]))
    drop = float(l0.detach()) - l1
    pred = lr * float(g @ out["ghat"][0])
    print(f"loss {float(l0.detach()):.6f} -> {l1:.6f}: drop {drop:.3e}, first-order {pred:.3e}, "
          f"lr |g|^2 = {lr * float(g @ g):.3e}")
    assert drop > 0
    assert abs(drop / pred - 1) < 0.1
    # with P = 512 directions the estimate is aligned with the gradient
    assert pred > 0.5 * lr * float(g @ g)


@pytest.mark.parametrize("lr", [0.0, -1.0])
def test_sgd_step_lr_special_values(oracle_mod, lr):
    """lr = 0 leaves theta bit-identical; lr = -1 adds the estimate itself."""
    P = 3
    cfg = oracle_mod.make_cfg(1, L, E, H, B, T, P)
    theta = synth.init_theta(1, L, E, H, init_seed=7)
    out = oracle_mod.spsa_step(cfg, theta, synth.expert_seeds(1), 0, 1e-3, lr, synth.expert_batches([14], B, T),
                               want_ghat=True)
    want = (theta[0].astype(np.float64) - lr * out["ghat"][0]).astype(np.float32)
    assert np.array_equal(out["theta"][0], want)
