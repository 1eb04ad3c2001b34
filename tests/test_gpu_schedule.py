"""GPU parity of the plateau schedule and of the step that reads each
expert's eps and lr from it (Section 4; Table experimental-setup)."""
import numpy as np
import pytest

from gpu_common import assert_losses_close, assert_theta_close, require_gpu
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


@pytest.mark.parametrize("mode", [0, 1])
def test_scheduled_step_uses_each_experts_rates(oracle_mod, mode):
    """Two experts with different (lr, eps), independent and summed losses,
    against the oracle's whole step at the same per-expert rates (its own
    forwards, coefficients and Adam update from the same seeded moments):
    losses, coefficients c_{e,j} = dL_e / (2 eps_e P) (independent) or
    dF / (2 eps_e P) with the shared difference dF (summed), theta' at the
    parity bar."""
    from test_gpu_step import adam_oracle_step, assert_moments_close, seeded_moments
    torch = require_gpu()
    (N, L, E, H, B, T, P), theta, data, seeds = _step_inputs()
    lrs, epss = F([1e-3, 2.5e-4]), F([1e-3, 4e-3])
    shape = soma.Shape(N, L, E, H, B, T, P, mode, probe=1)
    cfg = oracle_mod.cfg_from(shape)
    ghat = oracle_mod.spsa_step(cfg, theta, seeds, 6, epss, lrs, data, want_ghat=True)["ghat"]
    m0, v0 = seeded_moments(ghat)
    ctx = soma.Context(shape)
    adam = soma.Adam()
    th = torch.from_numpy(theta.copy()).cuda()
    m = torch.from_numpy(m0.copy()).cuda()
    v = torch.from_numpy(v0.copy()).cuda()
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step_adam_sched(th, m, v, 3, adam, soma.seeds_tensor(seeds), 6, _sched_with(torch, lrs, epss),
                             torch.from_numpy(data).cuda(), losses)
    coef = torch.zeros((N, P), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    o, (to, mo, vo) = adam_oracle_step(oracle_mod, cfg, theta, seeds, 6, epss, lrs, data, m0, v0, 3, adam)
    assert_losses_close(losses.cpu().numpy(), o["losses"])
    cg = coef.cpu().numpy()
    cerr = np.abs(cg - o["coef"]).max() / np.abs(o["coef"]).max()
    assert cerr <= 2e-2
    if mode == 1:   # one shared loss difference: c_e eps_e is the same for every expert
        scaled = cg.astype(np.float64) * epss[:, None]
        np.testing.assert_allclose(scaled[1], scaled[0], rtol=1e-6, atol=0)
    terr = assert_theta_close(th.cpu().numpy(), to)
    assert_moments_close(m.cpu().numpy(), mo, np.abs(mo).max())
    assert_moments_close(v.cpu().numpy(), vo, np.abs(vo).max())
    print(f"mode {mode}: coef rel {cerr:.2e}  theta rel {terr:.2e}")
    ctx.close()


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
