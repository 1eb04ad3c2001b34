"""GPU parity of the paper's expert body (Section 3; Appendix C: pre-norm
residual LSTM + GELU-MLP blocks, gain-only LayerNorm, frozen tied E;
Appendix E: dense gains under the sparse law, the decoder-path delta rule)
against the oracle, through the C ABI, on shapes that span several
sequence tiles and ragged tails."""
import numpy as np
import pytest

from gpu_common import assert_losses_close, assert_theta_close, require_gpu, update_rel_error
from paper_2609_37899_amd import soma, synth, workloads

pytestmark = pytest.mark.gpu
V = 256

# name: (N, D, d, B, T, P, eps, lr, probe, per_expert_E, accum, loss_mode)
CASES = {
    "d16_l1_gauss": (2, 1, 16, 20, 13, 3, 1e-3, 1e-2, 0, False, 1, 0),
    "d32_l2_sparse": (2, 2, 32, 20, 13, 3, 1e-3, 1e-2, 1, True, 1, 0),
    "d32_l2_b70_ragged": (1, 2, 32, 70, 9, 2, 2e-3, 5e-3, 1, False, 1, 0),
    "d32_l1_dense_accum": (2, 1, 32, 16, 11, 2, 1e-3, 1e-2, 2, True, 2, 0),
    "d16_l2_sparse_summed": (3, 2, 16, 5, 17, 2, 1e-3, 1e-2, 1, True, 1, 1),
}


def _inputs(name):
    N, D, d, B, T, P, eps, lr, probe, per_e, A, mode = CASES[name]
    theta = synth.init_body(N, D, d, init_seed=3, distinct=True)
    E = synth.init_tied_head(d, init_seed=5, n_experts=N if per_e else 0)
    if A > 1:
        data = np.stack([synth.expert_batches([500 + e for e in range(N)], B, T, data_seed=a) for a in range(A)])
    else:
        data = synth.expert_batches([500 + e for e in range(N)], B, T)
    shape = soma.Shape(N, D, d, d, B, T, P, mode, probe=probe, accum=A, arch=soma.ARCH_BODY)
    return shape, theta, E, data, synth.expert_seeds(N), eps, lr, per_e


def _oracle_cfg(oracle_mod, shape, E):
    return oracle_mod.make_cfg(shape.n_experts, shape.n_layers, shape.embed, shape.hidden, shape.batch,
                               shape.seq_len, shape.n_pairs, shape.loss_mode, shape.probe, shape.accum,
                               arch=1, tied_head=E)


def _expert_cfg(oracle_mod, shape, E, e, per_e):
    """The oracle's configuration for expert e alone (its own tied matrix)."""
    return _oracle_cfg(oracle_mod, shape, E[e] if per_e else E)


def _context(torch, shape, E, per_e):
    ctx = soma.Context(shape)
    dE = torch.from_numpy(E.copy()).cuda()
    ctx.set_tied_head(dE, per_expert=per_e)
    return ctx, dE


@pytest.mark.parametrize("name", list(CASES))
def test_body_step_matches_oracle(oracle_mod, name):
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr, per_e = _inputs(name)
    N, D = shape.n_experts, shape.directions
    ctx, dE = _context(torch, shape, E, per_e)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((N, D, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step(th, soma.seeds_tensor(seeds), 4, eps, lr, torch.from_numpy(data).cuda(), losses)
    coef = torch.zeros((N, D), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    o = oracle_mod.spsa_step(_oracle_cfg(oracle_mod, shape, E), theta, seeds, 4, eps, lr, data)
    lerr = assert_losses_close(losses.cpu().numpy(), o["losses"])
    got = th.cpu().numpy()
    terr = assert_theta_close(got, o["theta"])
    uerr = update_rel_error(theta, got, o["theta"])
    cg = coef.cpu().numpy()
    cerr = np.abs(cg - o["coef"]).max() / np.abs(o["coef"]).max()
    print(f"{name}: loss rel {lerr:.2e}  theta rel {terr:.2e}  update rel {uerr:.2e}  coef rel {cerr:.2e}")
    assert cerr < 2e-2
    assert uerr < 2e-2
    assert not np.array_equal(got, theta)
    assert np.array_equal(dE.cpu().numpy(), E)     # E is read, never perturbed or written


@pytest.mark.parametrize("name", ["d16_l1_gauss", "d32_l2_b70_ragged"])
def test_body_eval_loss_matches_oracle(oracle_mod, name):
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr, per_e = _inputs(name)
    ctx, _ = _context(torch, shape, E, per_e)
    loss = torch.zeros(shape.n_experts, dtype=torch.float32, device="cuda")
    ctx.eval_loss(torch.from_numpy(theta).cuda(), torch.from_numpy(data).cuda(), loss)
    torch.cuda.synchronize()
    ref = oracle_mod.eval_loss(_oracle_cfg(oracle_mod, shape, E), theta, data)
    assert_losses_close(loss.cpu().numpy(), ref)


def test_body_probe_law_is_bit_exact(oracle_mod):
    """theta = 0, one direction, coefficient 1, lr = -1: the update writes
    z itself (exact in fp32), which must equal the oracle's probe under the
    body's per-coordinate law (dense gains, sparse weights) bit for bit."""
    torch = require_gpu()
    N, D, d = 2, 2, 32
    shape = soma.Shape(N, D, d, d, 4, 3, 1, probe=1, arch=soma.ARCH_BODY)
    ctx = soma.Context(shape)
    dp = ctx.d
    th = torch.zeros((N, dp), dtype=torch.float32, device="cuda")
    seeds = synth.expert_seeds(N)
    ctx.apply_update(th, soma.seeds_tensor(seeds), 9, -1.0, torch.ones((N, 1), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    got = th.cpu().numpy()
    cfg = oracle_mod.make_cfg(N, D, d, d, 4, 3, 1, 0, 1, arch=1, tied_head=np.zeros((V, d), np.float32))
    for e in range(N):
        ref = oracle_mod.perturb(cfg, np.zeros(dp, np.float32), int(seeds[e]), 9, 0, 1.0)
        assert np.array_equal(got[e], ref)
    blk = 16 * d * d + 2 * d
    gains = np.r_[0:d, d + 8 * d * d:2 * d + 8 * d * d]
    assert set(np.unique(got[0][gains])) == {-1.0, 1.0}
    assert set(np.unique(got[0][blk + 3 * d:blk + 3 * d + 4096])) == {-1.0, 0.0, 1.0}


def test_body_adam_step_uses_the_gain_law(oracle_mod):
    """The Adam step on the body under the sparse law (update number 3,
    seeded moments) against the oracle's whole step: losses, coefficients,
    theta' at the parity bar, the moments at the coefficients' bar."""
    from test_gpu_step import adam_oracle_step, assert_moments_close, seeded_moments
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr, per_e = _inputs("d32_l2_sparse")
    N, P = shape.n_experts, shape.n_pairs
    cfg = _oracle_cfg(oracle_mod, shape, E)
    ghat = oracle_mod.spsa_step(cfg, theta, seeds, 2, eps, 1e-3, data, want_ghat=True)["ghat"]
    m0, v0 = seeded_moments(ghat)
    ctx, _ = _context(torch, shape, E, per_e)
    adam = soma.Adam()
    th = torch.from_numpy(theta.copy()).cuda()
    m = torch.from_numpy(m0.copy()).cuda()
    v = torch.from_numpy(v0.copy()).cuda()
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step_adam(th, m, v, 3, adam, soma.seeds_tensor(seeds), 2, eps, 1e-3, torch.from_numpy(data).cuda(),
                       losses)
    coef = torch.zeros((N, P), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    o, (to, mo, vo) = adam_oracle_step(oracle_mod, cfg, theta, seeds, 2, eps, 1e-3, data, m0, v0, 3, adam)
    assert_losses_close(losses.cpu().numpy(), o["losses"])
    cerr = np.abs(coef.cpu().numpy() - o["coef"]).max() / np.abs(o["coef"]).max()
    assert cerr <= 2e-2
    terr = assert_theta_close(th.cpu().numpy(), to)
    assert_moments_close(m.cpu().numpy(), mo, np.abs(mo).max())
    assert_moments_close(v.cpu().numpy(), vo, np.abs(vo).max())
    print(f"body Adam: coef rel {cerr:.2e}  theta rel {terr:.2e}")
    ctx.close()


@pytest.mark.parametrize("name", ["d32_l2_sparse", "d16_l1_gauss"])
def test_head_delta_matches_oracle(oracle_mod, name):
    """The delta rule's gradient and loss (Appendix E, Eq. delta), then its
    in-place descent step on per-expert tied matrices."""
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr, per_e = _inputs(name)
    N, d = shape.n_experts, shape.hidden
    ctx, dE = _context(torch, shape, E, per_e)
    grad = torch.zeros((N, V, d), dtype=torch.float32, device="cuda")
    loss = torch.zeros(N, dtype=torch.float32, device="cuda")
    dth = torch.from_numpy(theta).cuda()
    dbytes = torch.from_numpy(data).cuda()
    step_lr = 0.5 if per_e else 0.0
    ctx.head_delta(dth, dbytes, step_lr, grad, loss)
    torch.cuda.synchronize()
    gg, lg = grad.cpu().numpy(), loss.cpu().numpy()
    for e in range(N):
        Ee = E[e] if per_e else E
        cfg = oracle_mod.make_cfg(1, shape.n_layers, d, d, shape.batch, shape.seq_len, 1, arch=1, tied_head=Ee)
        lo, go = oracle_mod.head_delta(cfg, theta[e], data[e])
        assert abs(lg[e] - lo) <= 1e-4 * abs(lo)
        err = np.abs(gg[e] - go).max() / np.abs(go).max()
        print(f"{name} expert {e}: grad rel {err:.2e}")
        assert err <= 1e-4
        if step_lr:
            newE = dE.cpu().numpy()[e]
            np.testing.assert_allclose(newE, Ee - step_lr * go, rtol=0, atol=1e-4 * np.abs(step_lr * go).max() + 1e-7)
    if not step_lr:
        assert np.array_equal(dE.cpu().numpy(), E)


def test_body_separability():
    """Changing one expert's batch leaves every other expert's losses and
    update bit for bit unchanged (independent losses)."""
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr, per_e = _inputs("d32_l2_sparse")
    outs = []
    for variant in range(2):
        x = data.copy()
        if variant:
            x[1] = synth.expert_batches([999], shape.batch, shape.seq_len)[0]
        ctx, _ = _context(torch, shape, E, per_e)
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((shape.n_experts, shape.n_pairs, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, soma.seeds_tensor(seeds), 1, eps, lr, torch.from_numpy(x).cuda(), losses)
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy()))
    assert np.array_equal(outs[0][0][0], outs[1][0][0])
    assert np.array_equal(outs[0][1][0], outs[1][1][0])
    assert not np.array_equal(outs[0][1][1], outs[1][1][1])


def test_body_fullsize_sampled(oracle_mod):
    """The paper's width-32 configuration at full size (eight experts, 64
    directions, 64 x 1,024 bytes), in the launch configuration the benchmark
    times: sampled losses, and for two experts every loss, coefficient and a
    sampled set of updated weights against the oracle alone."""
    torch = require_gpu()
    w = workloads.PAPER_BODY_N8
    N, P = w.n_experts, w.n_pairs
    theta = synth.init_body(N, w.n_layers, w.hidden, init_seed=w.init_seed)
    E = synth.init_tied_head(w.hidden, init_seed=1)
    data = synth.expert_batches_in_child(w.cluster_seeds, w.batch, w.seq_len)
    seeds = synth.expert_seeds(N)
    shape = soma.Shape(N, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, P, probe=w.probe, arch=1)
    ctx, _ = _context(torch, shape, E, False)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step(th, soma.seeds_tensor(seeds), 0, w.eps, w.lr, torch.from_numpy(data).cuda(), losses)
    coef = torch.zeros((N, P), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    lg, cg, got = losses.cpu().numpy(), coef.cpu().numpy(), th.cpu().numpy()
    assert np.all(np.isfinite(lg))
    cfg = _oracle_cfg(oracle_mod, shape, E)
    for (e, j, s) in ((5, 37, 0), (2, 63, 1)):
        ref = oracle_mod.perturbed_loss(cfg, theta[e], int(seeds[e]), 0, j, 1 - 2 * s, w.eps, data[e])
        assert abs(lg[e, j, s] - ref) <= 1e-4 * abs(ref), (e, j, s, lg[e, j, s], ref)
    # Experts 0 and 7: every coefficient from the oracle's own forwards (128
    # each at full size, a few seconds), then theta' at sampled coordinates
    # from the oracle's update -- nothing from the GPU enters the reference.
    ks = np.random.default_rng(0).choice(ctx.d, 4000, replace=False)
    denom = 2.0 * np.float64(np.float32(w.eps)) * P
    for e in (0, 7):
        print(f"oracle forwards of expert {e} (all {P} directions, both signs)", flush=True)
        lo = np.array([[oracle_mod.perturbed_loss(cfg, theta[e], int(seeds[e]), 0, j, sgn, w.eps, data[e])
                        for sgn in (1, -1)] for j in range(P)])
        co = (lo[:, 0] - lo[:, 1]) / denom
        assert_losses_close(lg[e], lo)
        cerr = np.abs(cg[e] - co).max() / np.abs(co).max()
        assert cerr <= 2e-2
        ref = oracle_mod.apply_update(cfg, theta[e], int(seeds[e]), 0, w.lr, co, ks)
        terr = assert_theta_close(got[e][ks], ref)
        print(f"expert {e}: coef rel {cerr:.2e}  theta' rel {terr:.2e} (oracle coefficients only)")
