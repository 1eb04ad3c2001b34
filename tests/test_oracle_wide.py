"""Pins for the oracle's body of the wider fixed-size controls (arch 2;
Appendix C, counting rules and Table fixed-parameter-counts; Appendix E):
the paper's residual LSTM + GELU-MLP blocks at width d_t between an input
projection P_in and an output projection P_out to the head width d_E, with
each expert's own tied E.

* parameter counts: N (32 d_t^2 + 5 d_t + 2 d_E d_t + V d_E) reproduces the
  table's ensemble totals (8.33M, 8.41M, 8.55M), its body sizes (8.33M,
  4.20M, 1.06M, head excluded) and 8.19k per head (golden values);
* the loss equals the same network assembled from torch.nn.Linear,
  torch.nn.LSTM, torch.nn.LayerNorm(bias=False) and the exact GELU in fp64,
  read from the documented layout (a transposed or swapped matrix fails:
  none of the matrices is square);
* the delta rule (Appendix E, Eq. delta) with the decoder input u = P_out f
  equals torch autograd through the decoder only;
* with d_t = d_E and identity projections the body is the paper's width-d
  body (arch 1, pinned separately) with its matrices re-laid out;
* under the sparse law the gains, which sit at the end, draw dense +-1, and
  the body is one mask group.
"""
import json
import os

import numpy as np
import pytest
import torch

from paper_2609_37899_amd import synth

V = 256
HERE = os.path.dirname(os.path.abspath(__file__))


def split_wide(theta, D, dt, de):
    """The canonical arch-2 layout, as numpy views."""
    d4 = 4 * dt
    o = 0
    pin = theta[o:o + dt * de].reshape(dt, de)
    o += dt * de
    blocks = []
    for _ in range(D):
        mats = []
        for _ in range(4):
            mats.append(theta[o:o + dt * d4].reshape(dt, d4))
            o += dt * d4
        blocks.append(mats)
    pout = theta[o:o + dt * de].reshape(dt, de)
    o += dt * de
    gains = theta[o:].reshape(2 * D + 1, dt)
    assert gains.size == (2 * D + 1) * dt
    return pin, blocks, pout, gains


def torch_wide(theta, E, D, dt, de, seqs, detach_decoder_input=False):
    """The wide body assembled from torch modules (fp64); returns (mean CE, E)."""
    t = theta.astype(np.float64)
    pin, blocks, pout, gains = split_wide(t, D, dt, de)
    Et = torch.tensor(E.astype(np.float64), requires_grad=True)
    inp = torch.nn.Linear(de, dt, bias=False).double()
    outp = torch.nn.Linear(dt, de, bias=False).double()
    mods = []
    for l, (A, R, U, Vd) in enumerate(blocks):
        ln1 = torch.nn.LayerNorm(dt, eps=1e-5, bias=False).double()
        ln2 = torch.nn.LayerNorm(dt, eps=1e-5, bias=False).double()
        lstm = torch.nn.LSTM(dt, dt, bias=False, batch_first=True).double()
        up = torch.nn.Linear(dt, 4 * dt, bias=False).double()
        down = torch.nn.Linear(4 * dt, dt, bias=False).double()
        with torch.no_grad():
            ln1.weight.copy_(torch.tensor(gains[2 * l]))
            ln2.weight.copy_(torch.tensor(gains[2 * l + 1]))
            lstm.weight_ih_l0.copy_(torch.tensor(A.T))      # [4 d_t][d_t], rows gate-major
            lstm.weight_hh_l0.copy_(torch.tensor(R.T))
            up.weight.copy_(torch.tensor(U.T))              # [4 d_t][d_t]
            down.weight.copy_(torch.tensor(Vd))             # [d_t][4 d_t]
        mods.append((ln1, lstm, ln2, up, down))
    lnf = torch.nn.LayerNorm(dt, eps=1e-5, bias=False).double()
    with torch.no_grad():
        inp.weight.copy_(torch.tensor(pin))                 # [d_t][d_E]
        outp.weight.copy_(torch.tensor(pout.T))             # [d_E][d_t]
        lnf.weight.copy_(torch.tensor(gains[2 * D]))
    ce, n = 0.0, 0
    for seq in seqs:
        x = inp(Et.detach()[torch.tensor(seq[:-1].astype(np.int64))])
        for ln1, lstm, ln2, up, down in mods:
            h, _ = lstm(ln1(x)[None])
            r = x + h[0]
            x = r + down(torch.nn.functional.gelu(up(ln2(r))))
        u = outp(lnf(x))
        if detach_decoder_input:
            u = u.detach()
        logits = u @ Et.T
        ce = ce + torch.nn.functional.cross_entropy(logits, torch.tensor(seq[1:].astype(np.int64)),
                                                    reduction="sum")
        n += len(seq) - 1
    return ce / n, Et


def wide_cfg(oracle_mod, D, dt, de, E, B=1, T=2, P=1, probe=0, mask=0, N=1):
    return oracle_mod.make_cfg(N, D, de, dt, B, T, P, 0, probe, arch=oracle_mod.ARCH_WIDE, tied_head=E,
                               perturb_mask=mask)


def test_parameter_counts_match_the_paper_table(oracle_mod):
    gold = json.load(open(os.path.join(HERE, "golden", "wide_controls_parameter_counts.json")))
    for row in gold["rows"]:
        N, dt, de = row["N"], row["d_t"], 32
        cfg = wide_cfg(oracle_mod, 2, dt, de, np.zeros((V, de), np.float32))
        body = oracle_mod.param_count(cfg)
        assert body == 32 * dt * dt + 5 * dt + 2 * de * dt == synth.wide_param_count(2, dt, de)
        head = V * de
        assert round(head / 1e3, 2) == row["head_per_expert_k"]
        assert round(N * (body + head) / 1e6, 2) == row["ensemble_M"], (N, N * (body + head))
        assert round(body / 1e6, 2) == row["expert_body_M"], (N, body)
    # the exact totals the formula gives
    tot = {(r["N"], r["d_t"]): r["N"] * (synth.wide_param_count(2, r["d_t"], 32) + V * 32) for r in gold["rows"]}
    assert tot == {(1, 509): 8_333_905, (2, 361): 8_406_746, (8, 181): 8_552_264}


@pytest.mark.parametrize("D,dt,de", [(1, 7, 4), (2, 13, 8)])
def test_wide_loss_equals_torch_modules(oracle_mod, D, dt, de):
    theta = synth.init_wide(1, D, dt, de, init_seed=3)[0]
    theta[-(2 * D + 1) * dt:] = (1.0 + 0.2 * np.random.default_rng(5).standard_normal((2 * D + 1) * dt))
    E = (np.random.default_rng(2).standard_normal((V, de)) * 0.5).astype(np.float32)
    data = synth.expert_batches([9], 3, 17)[0]
    cfg = wide_cfg(oracle_mod, D, dt, de, E, B=3, T=17)
    ours = oracle_mod.forward_loss_f64(cfg, theta.astype(np.float64), data)
    ref, _ = torch_wide(theta, E, D, dt, de, data)
    assert abs(ours - float(ref.detach())) < 1e-12 * abs(float(ref.detach()))
    assert abs(ours - np.log(256.0)) > 1e-3          # the weights matter


def test_delta_rule_is_the_decoder_path_gradient(oracle_mod):
    D, dt, de = 2, 11, 8
    theta = synth.init_wide(1, D, dt, de, init_seed=4)[0]
    E = (np.random.default_rng(4).standard_normal((V, de)) * 0.5).astype(np.float32)
    data = synth.expert_batches([11], 2, 13)[0]
    cfg = wide_cfg(oracle_mod, D, dt, de, E, B=2, T=13)
    loss, g = oracle_mod.head_delta(cfg, theta, data)
    assert g.shape == (V, de)
    ref, Et = torch_wide(theta, E, D, dt, de, data, detach_decoder_input=True)
    ref.backward()
    assert abs(loss - float(ref.detach())) < 1e-12 * abs(float(ref.detach()))
    np.testing.assert_allclose(g, Et.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_identity_projections_give_the_paper_body(oracle_mod):
    D, d = 2, 8
    rng = np.random.default_rng(6)
    body = synth.init_body(1, D, d, init_seed=6)[0].astype(np.float64)
    blk = 16 * d * d + 2 * d
    wide = [np.eye(d).ravel()]
    gains = []
    for l in range(D):
        o = l * blk
        g1, W = body[o:o + d], body[o + d:o + d + 8 * d * d].reshape(4 * d, 2 * d)
        o2 = o + d + 8 * d * d
        g2, W1 = body[o2:o2 + d], body[o2 + d:o2 + d + 4 * d * d].reshape(4 * d, d)
        W2 = body[o2 + d + 4 * d * d:o2 + d + 8 * d * d].reshape(d, 4 * d)
        wide += [W[:, :d].T.ravel(), W[:, d:].T.ravel(), W1.T.ravel(), W2.ravel()]
        gains += [g1, g2]
    wide.append(np.eye(d).ravel())
    wide += gains + [body[D * blk:]]
    wide = np.concatenate(wide)
    E = (rng.standard_normal((V, d)) * 0.5).astype(np.float32)
    data = synth.expert_batches([12], 2, 11)[0]
    c1 = oracle_mod.make_cfg(1, D, d, d, 2, 11, 1, arch=oracle_mod.ARCH_PAPER_BODY, tied_head=E)
    c2 = wide_cfg(oracle_mod, D, d, d, E, B=2, T=11)
    assert oracle_mod.param_count(c2) == wide.size == oracle_mod.param_count(c1) + 2 * d * d
    a = oracle_mod.forward_loss_f64(c1, body, data)
    b = oracle_mod.forward_loss_f64(c2, wide, data)
    assert abs(a - b) < 1e-13 * abs(a)


def test_sparse_law_draws_dense_gains_and_the_body_is_one_group(oracle_mod):
    D, dt, de = 2, 9, 4
    theta = synth.init_wide(1, D, dt, de, init_seed=7)[0]
    E = np.zeros((V, de), np.float32)
    cfg = wide_cfg(oracle_mod, D, dt, de, E, probe=1)
    w = oracle_mod.perturb(cfg, theta, 0x50A10000, 0, 3, 1.0)
    z = np.rint(w.astype(np.float64) - theta)
    ng = (2 * D + 1) * dt
    assert set(np.unique(z[-ng:])) == {-1.0, 1.0}
    zw = z[:-ng]
    assert set(np.unique(zw)) == {-1.0, 0.0, 1.0}
    assert abs(np.mean(zw == 0) - 0.5) < 5 * np.sqrt(0.25 / zw.size)
    # the body is one group (bit 1): masking it leaves every coordinate
    off = wide_cfg(oracle_mod, D, dt, de, E, probe=1, mask=oracle_mod.PERTURB_EMBEDDING | oracle_mod.PERTURB_HEAD)
    assert np.array_equal(oracle_mod.perturb(off, theta, 0x50A10000, 0, 3, 1.0), theta)
