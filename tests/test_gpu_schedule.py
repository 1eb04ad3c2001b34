"""GPU parity of the plateau schedule and of the step that reads each
expert's eps and lr from it (Section 4; Table experimental-setup)."""
import numpy as np
import pytest

from gpu_common import assert_losses_close, require_gpu
from paper_2609_37899_amd import soma, synth

pytestmark = pytest.mark.gpu
F = np.float32


def test_schedule_matches_oracle_bitwise(oracle_mod):
    torch = require_gpu()
    n, steps = 5, 300
    rng = np.random.default_rng(2)
    base = np.cumsum(rng.exponential(1e-3, (steps, n)) * (rng.random((steps, n)) < 0.15), axis=0)
    losses = (5.0 - base + rng.normal(0, 1e-4, (steps, n))).astype(np.float32)
    losses[37, 2] = np.nan
    updates = rng.integers(1, 4, steps)
    rule = soma.Plateau(factor=0.5, patience=7, threshold=1e-8, floor=1e-5)
    sched = soma.schedule_tensor(n)
    soma.schedule_init(sched, 1e-3, 2e-3)
    ref = oracle_mod.Plateau(n, 1e-3, 2e-3, factor=0.5, patience=7, threshold=1e-8, floor=1e-5)
    dl = torch.from_numpy(losses).cuda()
    decays = 0
    for t in range(steps):
        soma.schedule_observe(sched, dl[t], int(updates[t]), rule)
        ref.observe(losses[t], int(updates[t]))
        if t % 25 == 24 or t == steps - 1:
            got = soma.schedule_fields(sched)
            for g, r in zip(got, ref.state()):
                assert np.array_equal(g, r, equal_nan=True), (t, g, r)
            decays = int(np.sum(got[0] < F(1e-3)))
    assert decays > 0


def _step_inputs(N=2, L=2, E=48, H=64, B=20, T=13, P=3):
    theta = synth.init_theta(N, L, E, H, init_seed=4, distinct=True)
    data = synth.expert_batches([300 + e for e in range(N)], B, T)
    return (N, L, E, H, B, T, P), theta, data, synth.expert_seeds(N)


def _sched_with(torch, lrs, epss):
    n = len(lrs)
    a = np.zeros((n, 4), np.int32)
    f = a.view(np.float32)
    f[:, 0] = lrs
    f[:, 1] = epss
    f[:, 2] = np.inf
    return torch.from_numpy(a).cuda()


def test_scheduled_step_uses_each_experts_rates(oracle_mod):
    """Two experts with different (lr, eps): losses against oracle forwards
    at each expert's own radius, coefficients (L+ - L-)/(2 eps_e P), and the
    Adam update at each expert's own rate (applied by the oracle to the GPU's
    coefficients)."""
    torch = require_gpu()
    (N, L, E, H, B, T, P), theta, data, seeds = _step_inputs()
    lrs, epss = F([1e-3, 2.5e-4]), F([1e-3, 4e-3])
    shape = soma.Shape(N, L, E, H, B, T, P, probe=1)
    ctx = soma.Context(shape)
    adam = soma.Adam()
    th = torch.from_numpy(theta.copy()).cuda()
    m = torch.zeros_like(th)
    v = torch.zeros_like(th)
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step_adam_sched(th, m, v, 1, adam, soma.seeds_tensor(seeds), 6, _sched_with(torch, lrs, epss),
                             torch.from_numpy(data).cuda(), losses)
    coef = torch.zeros((N, P), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    cfg = oracle_mod.cfg_from(shape)
    lg, cg = losses.cpu().numpy(), coef.cpu().numpy()
    ref = np.array([[[oracle_mod.perturbed_loss(cfg, theta[e], int(seeds[e]), 6, j, s, float(epss[e]), data[e])
                      for s in (1, -1)] for j in range(P)] for e in range(N)])
    assert_losses_close(lg, ref)
    cref = (ref[..., 0] - ref[..., 1]) / (2.0 * epss[:, None].astype(np.float64) * P)
    assert np.abs(cg - cref).max() <= 2e-2 * np.abs(cref).max()
    hp = dict(beta1=float(adam.beta1), beta2=float(adam.beta2), delta=float(adam.delta),
              weight_decay=float(adam.weight_decay))
    from test_gpu_update import _adam_compare
    got = [x.cpu().numpy() for x in (th, m, v)]
    for e in range(N):
        to, mo, vo, gh = oracle_mod.apply_adam(cfg, theta[e], np.zeros_like(theta[e]), np.zeros_like(theta[e]), 1,
                                               int(seeds[e]), 6, float(lrs[e]), cg[e].astype(np.float64),
                                               want_ghat=True, **hp)
        g = gh + hp["weight_decay"] * theta[e].astype(np.float64)
        _adam_compare([x[e] for x in got], (to, mo, vo), theta[e].astype(np.float64), g, float(lrs[e]), 1, True)


def test_scheduled_step_with_equal_rates_is_the_scalar_step():
    torch = require_gpu()
    (N, L, E, H, B, T, P), theta, data, seeds = _step_inputs()
    shape = soma.Shape(N, L, E, H, B, T, P)
    adam = soma.Adam()
    outs = []
    for sched in (False, True):
        ctx = soma.Context(shape)
        th = torch.from_numpy(theta.copy()).cuda()
        m = torch.zeros_like(th)
        v = torch.zeros_like(th)
        losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
        args = (soma.seeds_tensor(seeds), 2)
        if sched:
            ctx.spsa_step_adam_sched(th, m, v, 3, adam, *args, _sched_with(torch, F([7e-4] * N), F([1e-3] * N)),
                                     torch.from_numpy(data).cuda(), losses)
        else:
            ctx.spsa_step_adam(th, m, v, 3, adam, *args, 1e-3, 7e-4, torch.from_numpy(data).cuda(), losses)
        torch.cuda.synchronize()
        outs.append([x.cpu().numpy() for x in (th, m, v, losses)])
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def test_invalid_rate_aborts_the_step_on_the_device():
    """An entry with eps = 0 is caught by the step's own check: the losses
    read NaN and theta, m and v are left as they were (every kernel still
    runs to completion)."""
    torch = require_gpu()
    (N, L, E, H, B, T, P), theta, data, seeds = _step_inputs()
    ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P))
    th = torch.from_numpy(theta.copy()).cuda()
    m = torch.full_like(th, 0.25)
    v = torch.full_like(th, 0.5)
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step_adam_sched(th, m, v, 1, soma.Adam(), soma.seeds_tensor(seeds), 0,
                             _sched_with(torch, F([1e-3, 1e-3]), F([1e-3, 0.0])), torch.from_numpy(data).cuda(),
                             losses)
    torch.cuda.synchronize()
    assert torch.isnan(losses).all()
    assert np.array_equal(th.cpu().numpy(), theta)
    assert bool((m == 0.25).all()) and bool((v == 0.5).all())
