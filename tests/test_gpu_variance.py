"""The variance harness on the GPU (Appendix estimator-iso): moments of the
single-direction estimates at fixed weights, against numpy on the oracle's
probes, and the paper's variance measurements reproduced on synthetic data --
the single-probe covariance against the R_g prediction
q (1 + s - 2q) ||g||^2 (s = q d; exact gradient by autograd in fp64), and the
averaging law tr Cov(mean of n probes) = tr Cov(one probe) / n."""
import numpy as np
import pytest
import torch as _torch

import torch_reference as tref
from gpu_common import require_gpu
from paper_2609_37899_amd import soma, synth, workloads

pytestmark = pytest.mark.gpu


def _setup(D, probe):
    w = workloads.TINY
    shape = soma.Shape(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, D, probe=probe)
    theta = synth.init_theta(1, w.n_layers, w.embed, w.hidden, init_seed=3) * np.float32(3.0)
    data = synth.expert_batches(w.cluster_seeds, w.batch, w.seq_len)
    return w, shape, theta, data


def test_moments_match_numpy_on_oracle_probes(oracle_mod):
    torch = require_gpu()
    D, G = 16, 4
    w, shape, theta, data = _setup(D, 1)
    seeds = synth.expert_seeds(1)
    coef = (np.random.default_rng(1).standard_normal((1, D)) * 1e-2).astype(np.float32)
    ctx = soma.Context(shape)
    out = torch.zeros((1, 2), dtype=torch.float64, device="cuda")
    ctx.estimator_moments(soma.seeds_tensor(seeds), 4, torch.from_numpy(coef).cuda(), D // G, out)
    torch.cuda.synchronize()
    d = theta.shape[1]
    X = np.stack([D * np.float64(coef[0, j]) * oracle_mod.probe(1, int(seeds[0]), 4, j, 0, d).astype(np.float64)
                  for j in range(D)])
    s0 = np.sum(X.reshape(G, D // G, d).sum(axis=1) ** 2)
    s1 = np.sum(X.sum(axis=0) ** 2)
    np.testing.assert_allclose(out.cpu().numpy()[0], [s0, s1], rtol=1e-12)


@pytest.mark.parametrize("probe,q", [(1, 0.5), (2, 1.0)])
def test_single_probe_covariance_and_averaging_law(probe, q):
    """A step at fixed weights (lr = 0) with D = 128 directions; the moments
    give tr Cov of single probes and of means of n = 2 .. 16 probes."""
    torch = require_gpu()
    D = 128
    w, shape, theta, data = _setup(D, probe)
    seeds = synth.expert_seeds(1, base=77)
    ctx = soma.Context(shape)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((1, D, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step(th, soma.seeds_tensor(seeds), 0, 1e-3, 0.0, torch.from_numpy(data).cuda(), losses)
    coef = torch.zeros((1, D), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    out = torch.zeros((1, 2), dtype=torch.float64, device="cuda")
    traces = {}
    for n in (1, 2, 4, 8, 16):
        ctx.estimator_moments(soma.seeds_tensor(seeds), 0, coef, n, out)
        traces[n] = float(soma.group_covariance_trace(out.cpu().numpy(), D, n)[0])
    t = _torch.tensor(theta[0].astype(np.float64), requires_grad=True)
    tref.loss(t, w.n_layers, w.embed, w.hidden, data[0]).backward()
    g2 = float(np.sum(t.grad.numpy() ** 2))
    d = theta.shape[1]
    pred = q * (1 + q * d - 2 * q) * g2
    print(f"law {probe}: tr Cov single / prediction = {traces[1] / pred:.3f}; traces {traces}")
    # 128 probes: the trace of d coordinate variances sharing the same probes
    assert abs(traces[1] / pred - 1) < 0.3
    slope = np.polyfit(np.log([1, 2, 4, 8, 16]), np.log([traces[n] for n in (1, 2, 4, 8, 16)]), 1)[0]
    assert abs(slope + 1) < 0.25, slope
