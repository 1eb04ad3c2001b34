"""GPU parity of the regenerate-and-update kernel on seeded synthetic
coefficients (so that no oracle input comes from the GPU)."""
import numpy as np
import pytest

from gpu_common import assert_theta_close, require_gpu
from paper_2609_37899_amd import soma, synth, workloads

pytestmark = pytest.mark.gpu


def _shape(w):
    return soma.Shape(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, w.n_pairs)


@pytest.mark.parametrize("wname,sampled", [("tiny_n1_h64", False), ("soma_n2_l2_h512", True)])
def test_apply_update_matches_oracle(oracle_mod, wname, sampled):
    torch = require_gpu()
    w = workloads.ALL[wname]
    shape = _shape(w)
    theta = synth.init_theta(w.n_experts, w.n_layers, w.embed, w.hidden, distinct=True)
    seeds = synth.expert_seeds(w.n_experts)
    coef = np.random.default_rng(5).standard_normal((w.n_experts, w.n_pairs)).astype(np.float32) * 0.3
    ctx = soma.Context(shape)
    th = torch.from_numpy(theta.copy()).cuda()
    ctx.apply_update(th, soma.seeds_tensor(seeds), 3, w.lr, torch.from_numpy(coef).cuda())
    torch.cuda.synchronize()
    got = th.cpu().numpy()
    cfg = oracle_mod.cfg_from(w)
    d = theta.shape[1]
    for e in range(w.n_experts):
        ks = np.random.default_rng(e).choice(d, 20000, replace=False) if sampled else None
        ref = oracle_mod.apply_update(cfg, theta[e], int(seeds[e]), 3, w.lr, coef[e].astype(np.float64), ks)
        g = got[e] if ks is None else got[e][ks]
        assert_theta_close(g, ref)
        # the change itself is accurate too (fp32 sum of P terms vs fp64)
        t0 = theta[e] if ks is None else theta[e][ks]
        dg, do = g.astype(np.float64) - t0, ref.astype(np.float64) - t0
        assert np.linalg.norm(dg - do) <= 1e-3 * np.linalg.norm(do)


def _adam_compare(got, ref, theta0, g, lr, t, zero_start):
    """theta', m', v' of the GPU against the oracle's (fp64, rounded once).
    From zero moments the first step is lr g / (|g| + delta), which jumps at
    g = 0: where |g| < 1e-6 (within fp32 summation error of a sign change)
    either sign is a correct result, so only a valid step is required."""
    th_g, m_g, v_g = got
    th_o, m_o, v_o = ref
    amb = (np.abs(g) < 1e-6) if (zero_start and t == 1) else np.zeros(g.shape, bool)
    ok = ~amb
    assert_theta_close(th_g[ok], th_o[ok])
    assert np.all(np.abs(th_g[amb].astype(np.float64) - theta0[amb]) <= lr * (1 + 1e-5))
    gs = np.sqrt(np.mean(g ** 2))
    np.testing.assert_allclose(m_g, m_o, rtol=1e-5, atol=1e-5 * gs)
    np.testing.assert_allclose(v_g, v_o, rtol=1e-5, atol=1e-5 * gs * gs)
    return int(amb.sum())


@pytest.mark.parametrize("wname,t,zero_start,probe", [("tiny_n1_h64", 1, True, 0), ("tiny_n1_h64", 7, False, 1),
                                                      ("soma_n2_l2_h512", 1, True, 0),
                                                      ("soma_n2_l2_h512", 3, False, 0)])
def test_apply_adam_matches_oracle(oracle_mod, wname, t, zero_start, probe):
    """The paper's Adam-style update (coupled decay, bias corrections) from
    seeded coefficients and moment states."""
    torch = require_gpu()
    w = workloads.ALL[wname]
    shape = soma.Shape(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, w.n_pairs, probe=probe)
    theta = synth.init_theta(w.n_experts, w.n_layers, w.embed, w.hidden, distinct=True)
    seeds = synth.expert_seeds(w.n_experts)
    rng = np.random.default_rng(11)
    coef = (rng.standard_normal((w.n_experts, w.n_pairs)) * 0.01).astype(np.float32)
    if zero_start:
        m0 = np.zeros_like(theta)
        v0 = np.zeros_like(theta)
    else:
        m0 = (rng.standard_normal(theta.shape) * 1e-3).astype(np.float32)
        v0 = (rng.random(theta.shape) * 1e-5).astype(np.float32)
    lr = np.float32(1e-3)
    adam = soma.Adam()
    ctx = soma.Context(shape)
    th, m, v = (torch.from_numpy(x.copy()).cuda() for x in (theta, m0, v0))
    ctx.apply_adam(th, m, v, t, adam, soma.seeds_tensor(seeds), 5, float(lr), torch.from_numpy(coef).cuda())
    torch.cuda.synchronize()
    got = [x.cpu().numpy() for x in (th, m, v)]
    cfg = oracle_mod.cfg_from(shape)
    hp = dict(beta1=float(adam.beta1), beta2=float(adam.beta2), delta=float(adam.delta),
              weight_decay=float(adam.weight_decay))
    d = theta.shape[1]
    for e in range(w.n_experts):
        ks = np.random.default_rng(e).choice(d, 20000, replace=False) if d > 100000 else np.arange(d)
        to, mo, vo, gh = oracle_mod.apply_adam(cfg, theta[e], m0[e], v0[e], t, int(seeds[e]), 5, float(lr),
                                               coef[e].astype(np.float64), ks=ks, want_ghat=True, **hp)
        g = gh + hp["weight_decay"] * theta[e][ks].astype(np.float64)
        n_amb = _adam_compare([x[e][ks] for x in got], (to, mo, vo), theta[e][ks].astype(np.float64), g,
                              float(lr), t, zero_start)
        print(f"{wname} t={t} expert {e}: {n_amb} coordinates with |g| < 1e-6")
        assert not np.array_equal(got[0][e][ks], theta[e][ks])
