"""Pins for the oracle's perturbation mask (cfg.perturb_mask) and for
per-expert radii.

The paper keeps parts of the model out of the search: its decoder/embedding E
is never perturbed (Section 4; Appendix E), so the estimate lives on the
perturbed coordinates only.  For the stacked LSTM the groups are the
embedding (bit 0), the LSTM layers (bit 1) and the head (bit 2).

* Masked coordinates keep their value bit for bit in every perturbed weight
  vector and in the update (SGD and Adam: theta, m and v); mask 7 is the
  unmasked step bit for bit.
* The unmasked coordinates follow the restricted model: losses from
  torch.nn.LSTM at theta +- eps (z masked), probes from the pinned generator,
  coefficients and the update formed in numpy -- a different code path.
* The masked estimate converges to the exact gradient restricted to the
  unmasked coordinates at the rate (d_m + 1)/P of a d_m-dimensional problem
  (Gaussian probes, E z^4 = 3), with exact zeros elsewhere.
* Per-expert radii: with independent losses expert e's step is the
  single-radius step at eps_e bit for bit; with the summed loss every
  expert's coefficient is the one shared loss difference over 2 eps_e D, so
  c_e eps_e is the same for every expert, and the estimate of expert e has
  the closed-form error ((d+1)|g_e|^2 + d sum_{e' != e} (eps_e'/eps_e)^2
  |g_e'|^2)/P in the linear regime (Gaussian probes).
"""
import numpy as np
import pytest
import torch

import torch_reference as tref
from paper_2609_37899_amd import synth

L, E, H, B, T = 1, 4, 8, 2, 16
EMB, LSTM, HEAD = 1, 2, 4


def groups(oracle_mod, n_layers=L, embed=E, hidden=H):
    """Index ranges of the embedding, the LSTM layers and the head."""
    d = oracle_mod.param_count(oracle_mod.make_cfg(1, n_layers, embed, hidden, B, T, 1))
    e_end = 256 * embed
    h_start = d - 256 * hidden
    return {EMB: np.arange(0, e_end), LSTM: np.arange(e_end, h_start), HEAD: np.arange(h_start, d)}, d


def unmasked_index(grp, mask):
    return np.concatenate([grp[b] for b in (EMB, LSTM, HEAD) if mask & b])


@pytest.mark.parametrize("mask", [LSTM, EMB | HEAD, HEAD, EMB])
def test_masked_coordinates_are_untouched(oracle_mod, mask):
    grp, d = groups(oracle_mod)
    cfg = oracle_mod.make_cfg(2, L, E, H, B, T, 3, perturb_mask=mask)
    theta = synth.init_theta(2, L, E, H, init_seed=8, distinct=True)
    data = synth.expert_batches([21, 22], B, T)
    seeds = synth.expert_seeds(2)
    out = oracle_mod.spsa_step(cfg, theta, seeds, 1, 1e-3, 1e-2, data, want_ghat=True)
    on = unmasked_index(grp, mask)
    off = np.setdiff1d(np.arange(d), on)
    assert np.array_equal(out["theta"][:, off], theta[:, off])
    assert np.all(out["ghat"][:, off] == 0.0)
    assert not np.array_equal(out["theta"][:, on], theta[:, on])
    w = oracle_mod.perturb(cfg, theta[0], int(seeds[0]), 1, 0, 1e-3)
    assert np.array_equal(w[off], theta[0, off])
    assert not np.array_equal(w[on], theta[0, on])
    # Adam: masked coordinates keep theta and both moments
    m = np.full(d, 0.25, np.float32)
    v = np.full(d, 0.5, np.float32)
    th1, m1, v1 = oracle_mod.apply_adam(cfg, theta[0], m, v, 3, int(seeds[0]), 1, 1e-3, out["coef"][0])
    assert np.array_equal(th1[off], theta[0, off]) and np.all(m1[off] == 0.25) and np.all(v1[off] == 0.5)
    assert not np.array_equal(m1[on], m[on])


def test_full_mask_is_the_unmasked_step(oracle_mod):
    theta = synth.init_theta(2, L, E, H, init_seed=9, distinct=True)
    data = synth.expert_batches([23, 24], B, T)
    seeds = synth.expert_seeds(2)
    a = oracle_mod.spsa_step(oracle_mod.make_cfg(2, L, E, H, B, T, 3), theta, seeds, 0, 1e-3, 1e-2, data)
    b = oracle_mod.spsa_step(oracle_mod.make_cfg(2, L, E, H, B, T, 3, perturb_mask=7), theta, seeds, 0, 1e-3,
                             1e-2, data)
    for k in ("losses", "coef", "theta"):
        assert np.array_equal(a[k], b[k])


@pytest.mark.parametrize("mask", [LSTM, LSTM | HEAD])
def test_unmasked_coordinates_follow_the_restricted_model(oracle_mod, mask):
    """Losses by torch.nn.LSTM at theta +- eps (z * m), the update in numpy."""
    P, eps, lr, step = 4, 1e-3, 5e-2, 3
    grp, d = groups(oracle_mod)
    on = unmasked_index(grp, mask)
    m = np.zeros(d, np.float32)
    m[on] = 1.0
    cfg = oracle_mod.make_cfg(1, L, E, H, B, T, P, perturb_mask=mask)
    theta = synth.init_theta(1, L, E, H, init_seed=10) * np.float32(2.0)
    data = synth.expert_batches([25], B, T)
    seed = int(synth.expert_seeds(1)[0])
    out = oracle_mod.spsa_step(cfg, theta, [seed], step, eps, lr, data)
    z = np.stack([oracle_mod.probe(0, seed, step, j, 0, d) for j in range(P)])
    ref_l = np.empty((P, 2))
    for j in range(P):
        for s, sgn in enumerate((1.0, -1.0)):
            # fp32 weights: the product of two fp32 values is exact in fp64, then rounded to fp32
            pert = (theta[0].astype(np.float64) + np.float64(np.float32(sgn * eps)) * z[j]).astype(np.float32)
            w = np.where(m > 0, pert, theta[0])
            ref_l[j, s] = float(tref.loss(torch.tensor(w.astype(np.float64)), L, E, H, data[0]))
    np.testing.assert_allclose(out["losses"][0], ref_l.astype(np.float32), rtol=2e-7)
    c = (ref_l[:, 0] - ref_l[:, 1]) / (2 * np.float64(np.float32(eps)) * P)
    np.testing.assert_allclose(out["coef"][0], c, rtol=1e-8, atol=1e-12)
    ghat = c @ z.astype(np.float64) * m
    want = (theta[0].astype(np.float64) - np.float64(np.float32(lr)) * ghat).astype(np.float32)
    err = np.abs(out["theta"][0].astype(np.float64) - want) / np.maximum(np.abs(want), 1e-3)
    assert err.max() < 1e-6, err.max()


@pytest.mark.slow
@pytest.mark.parametrize("mask", [LSTM, EMB | HEAD])
def test_masked_estimate_converges_at_the_restricted_rate(oracle_mod, mask):
    grp, d = groups(oracle_mod)
    on = unmasked_index(grp, mask)
    theta = synth.init_theta(1, L, E, H, init_seed=2) * np.float32(3.0)
    data = synth.expert_batches([4], B, T)
    t = torch.tensor(theta[0].astype(np.float64), requires_grad=True)
    tref.loss(t, L, E, H, data[0]).backward()
    g = t.grad.numpy()[on]
    dm = on.size
    for P in (128, 1024):
        cfg = oracle_mod.make_cfg(1, L, E, H, B, T, P, perturb_mask=mask)
        out = oracle_mod.spsa_step(cfg, theta, synth.expert_seeds(1), 1, 1e-3, 1e-3, data, want_ghat=True)
        err = np.sum((out["ghat"][0, on] - g) ** 2) / np.sum(g ** 2)
        ratio = err * P / (dm + 1)
        print(f"mask {mask}: d_m = {dm} of {d}, P = {P}: error / ((d_m+1)/P) = {ratio:.3f}")
        assert abs(ratio - 1) < 5 * np.sqrt(2 / P) + 0.05, (P, ratio)


def test_per_expert_radii(oracle_mod):
    N, P = 3, 4
    theta = synth.init_theta(N, L, E, H, init_seed=11, distinct=True)
    data = synth.expert_batches([31, 32, 33], B, T)
    seeds = synth.expert_seeds(N)
    eps = np.array([1e-3, 4e-3, 5e-4], np.float32)
    lr = np.array([1e-2, 2e-2, 5e-3], np.float32)
    ind = oracle_mod.make_cfg(N, L, E, H, B, T, P)
    a = oracle_mod.spsa_step(ind, theta, seeds, 0, eps, lr, data)
    for e in range(N):
        one = oracle_mod.spsa_step(oracle_mod.make_cfg(1, L, E, H, B, T, P), theta[e:e + 1], seeds[e:e + 1], 0,
                                   float(eps[e]), float(lr[e]), data[e:e + 1])
        for k in ("losses", "coef", "theta"):
            assert np.array_equal(a[k][e], one[k][0]), (e, k)
    s = oracle_mod.spsa_step(oracle_mod.make_cfg(N, L, E, H, B, T, P, 1), theta, seeds, 0, eps, lr, data)
    assert np.array_equal(s["losses"], a["losses"])          # the same forwards
    scaled = s["coef"] * eps.astype(np.float64)[:, None]     # c_e eps_e = dF / (2 D)
    np.testing.assert_allclose(scaled, np.broadcast_to(scaled[0], scaled.shape), rtol=1e-12)
    # the losses come out rounded to fp32: each difference carries up to one ulp of L
    dF = (a["losses"][..., 0].astype(np.float64) - a["losses"][..., 1]).sum(axis=0)
    ulp = float(np.spacing(np.float32(np.abs(a["losses"]).max())))
    np.testing.assert_allclose(scaled[0], dF / (2 * P), rtol=0, atol=N * ulp / (2 * P))


@pytest.mark.slow
def test_summed_estimate_with_unequal_radii_has_the_closed_form_error(oracle_mod):
    N, P, R = 2, 16, 48
    eps = np.array([1e-3, 4e-3], np.float32)
    theta = synth.init_theta(N, L, E, H, init_seed=3, distinct=True) * np.float32(3.0)
    data = synth.expert_batches([5, 6], B, T)
    G = []
    for e in range(N):
        t = torch.tensor(theta[e].astype(np.float64), requires_grad=True)
        tref.loss(t, L, E, H, data[e]).backward()
        G.append(t.grad.numpy())
    G = np.stack(G)
    d = G.shape[1]
    g2 = np.sum(G ** 2, axis=1)
    cfg = oracle_mod.make_cfg(N, L, E, H, B, T, P, 1)
    err = np.zeros(N)
    for r in range(R):
        out = oracle_mod.spsa_step(cfg, theta, synth.expert_seeds(N, base=1000 * r), r, eps, 1e-3, data,
                                   want_ghat=True)
        err += np.sum((out["ghat"] - G) ** 2, axis=1) / R
    for e in range(N):
        o = 1 - e
        pred = ((d + 1) * g2[e] + d * (eps[o] / eps[e]) ** 2 * g2[o]) / P
        print(f"expert {e}: error / closed form = {err[e] / pred:.3f}")
        assert abs(err[e] / pred - 1) < 0.25, (e, err[e] / pred)
