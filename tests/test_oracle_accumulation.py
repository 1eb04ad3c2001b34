"""Pins for accumulation over A independently sampled batches (Appendix E:
the estimate of an update averages the estimates of A batches, each with its
own n_pert directions).

* A = 1 is the single-batch step;
* the accumulated estimate is the mean of A single-batch estimates, batch a
  using directions a P .. a P + P - 1 of the update's probe stream, and its
  losses are those single-batch forwards;
* the accumulation-variance identity (Eq. accumulation-variance): averaging
  A independent (batch, directions) estimates divides the centered variance
  of one estimate by A (checked over repeated draws at fixed weights).
"""
import numpy as np
import pytest

from paper_2609_37899_amd import synth

L, E, H, B, T, P = 1, 4, 8, 3, 12, 4


def test_accum_1_is_the_single_batch_step(oracle_mod):
    theta = synth.init_theta(2, L, E, H, distinct=True)
    data = synth.expert_batches([1, 2], B, T)
    seeds = synth.expert_seeds(2)
    a = oracle_mod.spsa_step(oracle_mod.make_cfg(2, L, E, H, B, T, P), theta, seeds, 3, 1e-3, 1e-2, data)
    b = oracle_mod.spsa_step(oracle_mod.make_cfg(2, L, E, H, B, T, P, accum=1), theta, seeds, 3, 1e-3, 1e-2,
                             data[None])
    for k in ("losses", "coef", "theta"):
        assert np.array_equal(a[k], b[k])


def test_accumulated_estimate_is_the_mean_of_batch_estimates(oracle_mod):
    A, N = 3, 2
    theta = synth.init_theta(N, L, E, H, distinct=True)
    batches = np.stack([synth.expert_batches([10 + e for e in range(N)], B, T, data_seed=a) for a in range(A)])
    seeds = synth.expert_seeds(N)
    cfg = oracle_mod.make_cfg(N, L, E, H, B, T, P, 0, 0, accum=A)
    out = oracle_mod.spsa_step(cfg, theta, seeds, 5, 1e-3, 1e-2, batches, want_ghat=True)
    assert out["losses"].shape == (N, A * P, 2)
    one = oracle_mod.make_cfg(N, L, E, H, B, T, P)
    for e in range(N):
        gh = np.zeros(theta.shape[1])
        for a in range(A):
            lf = np.zeros((P, 2))
            for jj in range(P):
                j = a * P + jj
                for s, sign in enumerate((1, -1)):
                    lf[jj, s] = oracle_mod.perturbed_loss(one, theta[e], int(seeds[e]), 5, j, sign, 1e-3,
                                                          batches[a, e])
                    assert out["losses"][e, j, s] == np.float32(lf[jj, s])
            # batch a's own estimate, with its P directions (fp64 losses)
            c = (lf[:, 0] - lf[:, 1]) / (2 * np.float64(np.float32(1e-3)) * P)
            z = np.stack([oracle_mod.probe(0, int(seeds[e]), 5, a * P + jj, 0, theta.shape[1]) for jj in range(P)])
            gh += (c @ z.astype(np.float64)) / A
        np.testing.assert_allclose(out["ghat"][e], gh, rtol=1e-9, atol=1e-12 * np.abs(gh).max())


@pytest.mark.slow
def test_accumulation_divides_the_centered_variance(oracle_mod):
    """Fixed weights and a fixed pool of A batches: over R repeated draws of
    the directions, the spread of the accumulated estimate around its mean is
    1/A of the batches' mean single-batch spread, Var(mean_a X_a) =
    (1/A^2) sum_a Var(X_a) for independent directions (the perturbation term
    of Eq. accumulation-variance; the batch term is fixed here)."""
    A, R = 4, 60
    theta = synth.init_theta(1, L, E, H, init_seed=2) * np.float32(3.0)
    batches = np.stack([synth.expert_batches([7], B, T, data_seed=a) for a in range(A)])
    single = [[] for _ in range(A)]
    accum = []
    cfg1 = oracle_mod.make_cfg(1, L, E, H, B, T, P)
    cfgA = oracle_mod.make_cfg(1, L, E, H, B, T, P, accum=A)
    for r in range(R):
        seeds = synth.expert_seeds(1, base=5000 + r)
        for a in range(A):
            single[a].append(oracle_mod.spsa_step(cfg1, theta, seeds, 10 * r + a, 1e-3, 0.0, batches[a],
                                                  want_ghat=True)["ghat"][0])
        accum.append(oracle_mod.spsa_step(cfgA, theta, seeds, r, 1e-3, 0.0, batches, want_ghat=True)["ghat"][0])
    v_single = np.mean([np.sum(np.var(np.array(x), axis=0, ddof=1)) for x in single])
    vA = np.sum(np.var(np.array(accum), axis=0, ddof=1))
    # a trace of ~3,500 coordinate variances from R draws: ~2/sqrt(R) relative spread
    assert abs(vA * A / v_single - 1) < 3 * np.sqrt(2 / R), (vA * A / v_single)
