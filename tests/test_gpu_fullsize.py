"""Full-size parity in the benchmark's launch configuration.

At these sizes the oracle cannot run a whole step in seconds, so the test
compares sampled outputs it can compute one by one: individual perturbed
losses L(theta_e +- eps z_{e,j}) at the workload's full B and T.  Properties
that hold at any size are checked on the whole output: every loss is finite
and near ln 256 at initialisation, separability holds bit for bit, and the
step leaves the experts of independent runs identical where their inputs are.
"""
import gc

import numpy as np
import pytest

from gpu_common import assert_losses_close, require_gpu
from paper_2609_37899_amd import soma, synth, workloads

pytestmark = pytest.mark.gpu

SAMPLES = {   # (expert, direction, sign) checked against the oracle
    "soma_n2_l2_h512": [(0, 0, 0), (1, 31, 1)],
    "soma_n4_l2_h384": [(0, 5, 1), (3, 31, 0)],
    "monolith_l2_h704": [(0, 127, 0), (0, 60, 1)],   # 128 directions: the last chunk is ragged
    "soma_n256_l1_h64": [(0, 0, 0), (255, 31, 1), (131, 7, 0)],
}


def run_full(w, data=None):
    torch = require_gpu()
    shape = soma.Shape(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, w.n_pairs,
                       w.loss_mode, 0)
    theta = synth.init_theta(w.n_experts, w.n_layers, w.embed, w.hidden, w.init_seed)
    if data is None:
        data = synth.expert_batches_in_child(w.cluster_seeds, w.batch, w.seq_len, pool=w.pool_clusters)
    seeds = synth.expert_seeds(w.n_experts)
    ctx = soma.Context(shape)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((w.n_experts, w.n_pairs, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step(th, soma.seeds_tensor(seeds), 0, w.eps, w.lr, torch.from_numpy(data).cuda(), losses)
    torch.cuda.synchronize()
    out = dict(theta0=theta, data=data, seeds=seeds, theta=th.cpu().numpy(), losses=losses.cpu().numpy())
    del ctx, th, losses
    gc.collect()
    torch.cuda.empty_cache()
    return out


@pytest.mark.parametrize("wname", list(SAMPLES))
def test_full_size_sampled_losses(oracle_mod, wname):
    w = workloads.ALL[wname]
    r = run_full(w)
    L = r["losses"]
    assert np.all(np.isfinite(L))
    assert np.all(np.abs(L - np.log(256.0)) < 0.1)
    cfg = oracle_mod.cfg_from(w)
    got, ref = [], []
    for (e, j, s) in SAMPLES[wname]:
        print(f"{wname}: oracle forward e={e} j={j} sign={'+-'[s]}", flush=True)
        ref.append(oracle_mod.perturbed_loss(cfg, r["theta0"][e], int(r["seeds"][e]), 0, j,
                                             +1 if s == 0 else -1, w.eps, r["data"][e]))
        got.append(L[e, j, s])
    err = assert_losses_close(got, ref)
    print(f"{wname}: sampled loss rel err {err:.2e}")
    assert not np.array_equal(r["theta"], r["theta0"])


def test_full_size_separability_bit_identity():
    w = workloads.SOMA_N2
    data = synth.expert_batches_in_child(w.cluster_seeds, w.batch, w.seq_len)
    a = run_full(w, data)
    data2 = data.copy()
    data2[1] = synth.expert_batches_in_child([4242], w.batch, w.seq_len)[0]
    b = run_full(w, data2)
    assert np.array_equal(a["theta"][0], b["theta"][0])
    assert np.array_equal(a["losses"][0], b["losses"][0])
    assert not np.array_equal(a["theta"][1], b["theta"][1])
