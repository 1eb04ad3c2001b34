"""GPU parity of the wide controls' body (SOMA_ARCH_WIDE; Appendix C: the
width-d_t residual LSTM + GELU-MLP blocks between input and output
projections to the head width d_E = 32, each expert's own tied E; Appendix
E: dense gains under the sparse law, the decoder-path delta rule) against the
oracle, through the C ABI.  Widths are odd or otherwise not multiples of 64
(the kernels pad to d_p = 64 ceil(d_t / 64)), batches and sequence lengths
span several row tiles with ragged tails."""
import numpy as np
import pytest

from gpu_common import assert_losses_close, assert_theta_close, require_gpu, update_rel_error
from paper_2609_37899_amd import soma, synth, workloads

pytestmark = pytest.mark.gpu
V = 256
DE = 32

# name: (N, D, d_t, B, T, P, eps, lr, probe, accum, loss_mode)
CASES = {
    "d13_l1_gauss": (2, 1, 13, 5, 9, 3, 1e-3, 1e-2, 0, 1, 0),
    "d37_l2_sparse": (2, 2, 37, 20, 13, 3, 1e-3, 1e-2, 1, 1, 0),
    "d70_l2_dense_b64": (1, 2, 70, 64, 6, 2, 2e-3, 5e-3, 2, 1, 0),
    "d100_l1_sparse_summed": (3, 1, 100, 16, 11, 2, 1e-3, 1e-2, 1, 1, 1),
    "d21_l1_gauss_accum": (2, 1, 21, 8, 9, 2, 1e-3, 1e-2, 0, 2, 0),
}


def _inputs(name):
    N, D, dt, B, T, P, eps, lr, probe, A, mode = CASES[name]
    theta = synth.init_wide(N, D, dt, DE, init_seed=3, distinct=True)
    E = synth.init_tied_head(DE, init_seed=5, n_experts=N)
    if A > 1:
        data = np.stack([synth.expert_batches([600 + e for e in range(N)], B, T, data_seed=a) for a in range(A)])
    else:
        data = synth.expert_batches([600 + e for e in range(N)], B, T)
    shape = soma.Shape(N, D, DE, dt, B, T, P, mode, probe=probe, accum=A, arch=soma.ARCH_WIDE)
    return shape, theta, E, data, synth.expert_seeds(N), eps, lr


def _oracle_cfg(oracle_mod, shape, E):
    return oracle_mod.make_cfg(shape.n_experts, shape.n_layers, shape.embed, shape.hidden, shape.batch,
                               shape.seq_len, shape.n_pairs, shape.loss_mode, shape.probe, shape.accum,
                               arch=oracle_mod.ARCH_WIDE, tied_head=E)


def _context(torch, shape, E):
    ctx = soma.Context(shape)
    dE = torch.from_numpy(E.copy()).cuda()
    ctx.set_tied_head(dE, per_expert=True)
    return ctx, dE


@pytest.mark.parametrize("name", list(CASES))
def test_wide_step_matches_oracle(oracle_mod, name):
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr = _inputs(name)
    N, D = shape.n_experts, shape.directions
    print(f"{name}: step", flush=True)
    ctx, dE = _context(torch, shape, E)
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
    ctx.close()


@pytest.mark.parametrize("name", ["d13_l1_gauss", "d70_l2_dense_b64"])
def test_wide_eval_loss_matches_oracle(oracle_mod, name):
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr = _inputs(name)
    ctx, _ = _context(torch, shape, E)
    loss = torch.zeros(shape.n_experts, dtype=torch.float32, device="cuda")
    ctx.eval_loss(torch.from_numpy(theta).cuda(), torch.from_numpy(data).cuda(), loss)
    torch.cuda.synchronize()
    ref = oracle_mod.eval_loss(_oracle_cfg(oracle_mod, shape, E), theta, data)
    assert_losses_close(loss.cpu().numpy(), ref)
    ctx.close()


def test_wide_probe_law_is_bit_exact(oracle_mod):
    """theta = 0, one direction, coefficient 1, lr = -1: the update writes
    z itself, which must equal the oracle's probe under the wide body's
    per-coordinate law (sparse matrices, dense gains at the end) bit for bit."""
    torch = require_gpu()
    N, D, dt = 2, 2, 37
    shape = soma.Shape(N, D, DE, dt, 4, 3, 1, probe=1, arch=soma.ARCH_WIDE)
    ctx = soma.Context(shape)
    d = ctx.d
    assert d == synth.wide_param_count(D, dt, DE)
    th = torch.zeros((N, d), dtype=torch.float32, device="cuda")
    seeds = synth.expert_seeds(N)
    ctx.apply_update(th, soma.seeds_tensor(seeds), 9, -1.0, torch.ones((N, 1), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    got = th.cpu().numpy()
    cfg = oracle_mod.make_cfg(N, D, DE, dt, 4, 3, 1, 0, 1, arch=oracle_mod.ARCH_WIDE,
                              tied_head=np.zeros((V, DE), np.float32))
    for e in range(N):
        ref = oracle_mod.perturb(cfg, np.zeros(d, np.float32), int(seeds[e]), 9, 0, 1.0)
        assert np.array_equal(got[e], ref)
    ng = (2 * D + 1) * dt
    assert set(np.unique(got[0][-ng:])) == {-1.0, 1.0}
    assert set(np.unique(got[0][:-ng])) == {-1.0, 0.0, 1.0}
    ctx.close()


@pytest.mark.parametrize("name", ["d37_l2_sparse", "d100_l1_sparse_summed"])
def test_wide_head_delta_matches_oracle(oracle_mod, name):
    """The delta rule on each expert's own head (Appendix E): gradient and
    loss, then its in-place descent step."""
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr = _inputs(name)
    N = shape.n_experts
    ctx, dE = _context(torch, shape, E)
    grad = torch.zeros((N, V, DE), dtype=torch.float32, device="cuda")
    loss = torch.zeros(N, dtype=torch.float32, device="cuda")
    ctx.head_delta(torch.from_numpy(theta).cuda(), torch.from_numpy(data).cuda(), 0.5, grad, loss)
    torch.cuda.synchronize()
    gg, lg = grad.cpu().numpy(), loss.cpu().numpy()
    for e in range(N):
        cfg = oracle_mod.make_cfg(1, shape.n_layers, DE, shape.hidden, shape.batch, shape.seq_len, 1,
                                  arch=oracle_mod.ARCH_WIDE, tied_head=E[e])
        lo, go = oracle_mod.head_delta(cfg, theta[e], data[e])
        assert abs(lg[e] - lo) <= 1e-4 * abs(lo)
        err = np.abs(gg[e] - go).max() / np.abs(go).max()
        print(f"{name} expert {e}: grad rel {err:.2e}")
        assert err <= 1e-4
        newE = dE.cpu().numpy()[e]
        np.testing.assert_allclose(newE, E[e] - 0.5 * go, rtol=0, atol=1e-4 * np.abs(0.5 * go).max() + 1e-7)
    ctx.close()


def test_wide_separability():
    """Changing one expert's batch leaves the other expert's losses and
    update bit for bit unchanged (independent losses)."""
    torch = require_gpu()
    shape, theta, E, data, seeds, eps, lr = _inputs("d37_l2_sparse")
    outs = []
    for variant in range(2):
        x = data.copy()
        if variant:
            x[1] = synth.expert_batches([999], shape.batch, shape.seq_len)[0]
        ctx, _ = _context(torch, shape, E)
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((shape.n_experts, shape.n_pairs, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, soma.seeds_tensor(seeds), 1, eps, lr, torch.from_numpy(x).cuda(), losses)
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy()))
        ctx.close()
    assert np.array_equal(outs[0][0][0], outs[1][0][0])
    assert np.array_equal(outs[0][1][0], outs[1][1][0])
    assert not np.array_equal(outs[0][1][1], outs[1][1][1])


def test_wide_fullsize_sampled(oracle_mod):
    """The paper's N = 2 wide control (d_t = 361, B = 64, T = 1,024, 32
    directions, sparse probes) in the benchmark's launch configuration: every
    loss finite and near ln 256, one direction of expert 1 at both signs
    against the oracle, its coefficient, and theta' at sampled coordinates of
    expert 1 from oracle.apply_update fed the oracle's coefficient for that
    direction and the step's own for the others."""
    torch = require_gpu()
    w = workloads.WIDE_N2
    N, P = w.n_experts, w.n_pairs
    theta = synth.init_wide(N, w.n_layers, w.hidden, w.embed, init_seed=w.init_seed)
    E = synth.init_tied_head(w.embed, init_seed=1, n_experts=N)
    data = synth.expert_batches_in_child(w.cluster_seeds, w.batch, w.seq_len)
    seeds = synth.expert_seeds(N)
    shape = soma.Shape(N, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, P, probe=w.probe, arch=w.arch)
    print(f"{w.name}: step", flush=True)
    ctx, _ = _context(torch, shape, E)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step(th, soma.seeds_tensor(seeds), 0, w.eps, w.lr, torch.from_numpy(data).cuda(), losses)
    coef = torch.zeros((N, P), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    lg, cg, got = losses.cpu().numpy(), coef.cpu().numpy(), th.cpu().numpy()
    ctx.close()
    assert np.all(np.isfinite(lg)) and np.all(np.abs(lg - np.log(256.0)) < 0.5)
    e, j = 1, 29
    cfg = _oracle_cfg(oracle_mod, shape, E)
    ce = oracle_mod.make_cfg(1, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, P, 0, w.probe,
                             arch=oracle_mod.ARCH_WIDE, tied_head=E[e])
    ref = []
    for sgn in (1, -1):
        print(f"{w.name}: oracle forward e={e} j={j} sign={sgn}", flush=True)
        ref.append(oracle_mod.perturbed_loss(ce, theta[e], int(seeds[e]), 0, j, sgn, w.eps, data[e]))
    err = assert_losses_close(lg[e, j], ref)
    denom = 2.0 * np.float64(np.float32(w.eps)) * P
    c_mix = cg[e].astype(np.float64)
    c_mix[j] = (ref[0] - ref[1]) / denom
    cerr = abs(c_mix[j] - cg[e, j]) / np.abs(c_mix).max()
    assert cerr <= 2e-2
    ks = np.random.default_rng(2).choice(theta.shape[1], 3000, replace=False)
    want = oracle_mod.apply_update(cfg, theta[e], int(seeds[e]), 0, w.lr, c_mix, ks)
    terr = assert_theta_close(got[e][ks], want)
    print(f"{w.name}: loss rel {err:.2e}  coef rel {cerr:.2e}  theta' rel {terr:.2e}")
