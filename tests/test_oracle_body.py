"""Pins for the oracle's paper body (arch 1; Section 3, Appendix C, Fig. arch):
pre-norm residual blocks of a bias-free LSTM and a GELU MLP (hidden 4d) with
gain-only LayerNorm, a final gain-only LayerNorm and the frozen tied E.

* parameter count 16 D d^2 + (2D + 1) d, and the paper's 32.9k body
  parameters at d_t = 32, D = 2 (golden value, Appendix C);
* the loss equals the same network assembled from torch.nn.LSTM,
  torch.nn.LayerNorm(bias=False), torch.nn.GELU() and torch.nn.Linear(bias=
  False) in fp64;
* the delta rule (Appendix E, Eq. delta) equals torch autograd of the cross
  entropy with respect to E through the decoder only (decoder input detached);
* under the sparse probe law the gains draw dense +-1 (Appendix E).
"""
import json
import os

import numpy as np
import pytest
import torch

from paper_2609_37899_amd import synth

V = 256
HERE = os.path.dirname(os.path.abspath(__file__))


def body_params(D, d, seed):
    rng = np.random.default_rng(seed)
    parts = []
    for _ in range(D):
        parts += [1.0 + 0.1 * rng.standard_normal(d),                 # g1
                  rng.uniform(-1, 1, 8 * d * d) / np.sqrt(d),         # W (4d x 2d)
                  1.0 + 0.1 * rng.standard_normal(d),                 # g2
                  rng.uniform(-1, 1, 4 * d * d) / np.sqrt(d),         # W1 (4d x d)
                  rng.uniform(-1, 1, 4 * d * d) / np.sqrt(4 * d)]     # W2 (d x 4d)
    parts.append(1.0 + 0.1 * rng.standard_normal(d))                  # g_f
    return np.concatenate(parts).astype(np.float32)


def torch_body(theta, E, D, d, seqs, detach_decoder_input=False):
    """The body assembled from torch modules (fp64); returns (mean CE, E tensor)."""
    t = torch.tensor(theta.astype(np.float64))
    Et = torch.tensor(E.astype(np.float64), requires_grad=True)
    blk = 16 * d * d + 2 * d
    ce, n = 0.0, 0
    for seq in seqs:
        x = Et.detach()[torch.tensor(seq[:-1].astype(np.int64))]          # [T-1][d]
        for l in range(D):
            o = l * blk
            g1, W = t[o:o + d], t[o + d:o + d + 8 * d * d].reshape(4 * d, 2 * d)
            o2 = o + d + 8 * d * d
            g2, W1 = t[o2:o2 + d], t[o2 + d:o2 + d + 4 * d * d].reshape(4 * d, d)
            W2 = t[o2 + d + 4 * d * d:o2 + d + 8 * d * d].reshape(d, 4 * d)
            ln1 = torch.nn.LayerNorm(d, eps=1e-5, bias=False).double()
            ln2 = torch.nn.LayerNorm(d, eps=1e-5, bias=False).double()
            lstm = torch.nn.LSTM(d, d, bias=False, batch_first=True).double()
            up = torch.nn.Linear(d, 4 * d, bias=False).double()
            down = torch.nn.Linear(4 * d, d, bias=False).double()
            with torch.no_grad():
                ln1.weight.copy_(g1)
                ln2.weight.copy_(g2)
                lstm.weight_ih_l0.copy_(W[:, :d])
                lstm.weight_hh_l0.copy_(W[:, d:])
                up.weight.copy_(W1)
                down.weight.copy_(W2)
            h, _ = lstm(ln1(x)[None])
            r = x + h[0]
            x = r + down(torch.nn.functional.gelu(up(ln2(r))))
        lnf = torch.nn.LayerNorm(d, eps=1e-5, bias=False).double()
        with torch.no_grad():
            lnf.weight.copy_(t[D * blk:])
        f = lnf(x)
        if detach_decoder_input:
            f = f.detach()
        logits = f @ Et.T
        ce = ce + torch.nn.functional.cross_entropy(logits, torch.tensor(seq[1:].astype(np.int64)),
                                                    reduction="sum")
        n += len(seq) - 1
    return ce / n, Et


def test_parameter_count_matches_the_paper(oracle_mod):
    gold = json.load(open(os.path.join(HERE, "golden", "paper_compute_accounting.json")))
    E = np.zeros((V, 32), np.float32)
    cfg = oracle_mod.make_cfg(1, 2, 32, 32, 1, 2, 1, arch=1, tied_head=E)
    assert oracle_mod.param_count(cfg) == 32 * 32 * 32 + 5 * 32 == 32928
    assert round(oracle_mod.param_count(cfg) / 1000, 1) == gold["expert_body_params_k"]["value"]
    for D, d in ((1, 16), (3, 48)):
        cfg = oracle_mod.make_cfg(1, D, d, d, 1, 2, 1, arch=1, tied_head=np.zeros((V, d), np.float32))
        assert oracle_mod.param_count(cfg) == 16 * D * d * d + (2 * D + 1) * d


@pytest.mark.parametrize("D,d", [(1, 16), (2, 32)])
def test_body_loss_equals_torch_modules(oracle_mod, D, d):
    theta = body_params(D, d, 1)
    E = (np.random.default_rng(2).standard_normal((V, d)) * 0.3).astype(np.float32)
    data = synth.expert_batches([9], 3, 17)[0]
    cfg = oracle_mod.make_cfg(1, D, d, d, 3, 17, 1, arch=1, tied_head=E)
    ours = oracle_mod.forward_loss_f64(cfg, theta.astype(np.float64), data)
    ref, _ = torch_body(theta, E, D, d, data)
    assert abs(ours - float(ref.detach())) < 1e-12 * abs(float(ref.detach()))


def test_delta_rule_is_the_decoder_path_gradient(oracle_mod):
    D, d = 2, 16
    theta = body_params(D, d, 3)
    E = (np.random.default_rng(4).standard_normal((V, d)) * 0.3).astype(np.float32)
    data = synth.expert_batches([11], 2, 13)[0]
    cfg = oracle_mod.make_cfg(1, D, d, d, 2, 13, 1, arch=1, tied_head=E)
    loss, g = oracle_mod.head_delta(cfg, theta, data)
    ref, Et = torch_body(theta, E, D, d, data, detach_decoder_input=True)
    ref.backward()
    assert abs(loss - float(ref.detach())) < 1e-12 * abs(float(ref.detach()))
    np.testing.assert_allclose(g, Et.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_sparse_law_draws_dense_gains(oracle_mod):
    D, d = 2, 16
    theta = body_params(D, d, 5)
    E = np.zeros((V, d), np.float32)
    cfg = oracle_mod.make_cfg(1, D, d, d, 1, 2, 1, 0, 1, arch=1, tied_head=E)
    w = oracle_mod.perturb(cfg, theta, 0x50A10000, 0, 3, 1.0)
    z = (w.astype(np.float64) - theta) / 1.0
    z = np.rint(z)
    blk = 16 * d * d + 2 * d
    gain = np.zeros(theta.size, bool)
    for l in range(D):
        gain[l * blk:l * blk + d] = True
        gain[l * blk + d + 8 * d * d:l * blk + 2 * d + 8 * d * d] = True
    gain[D * blk:] = True
    assert set(np.unique(z[gain])) == {-1.0, 1.0}
    zw = z[~gain]
    assert set(np.unique(zw)) == {-1.0, 0.0, 1.0}
    assert abs(np.mean(zw == 0) - 0.5) < 5 * np.sqrt(0.25 / zw.size)
