"""GPU parity of the whole SPSA step and of the evaluation loss against the
oracle, on shapes that span several tiles and ragged tails."""
import numpy as np
import pytest

from gpu_common import assert_losses_close, assert_theta_close, require_gpu, update_rel_error
from paper_2609_37899_amd import soma, synth, workloads

pytestmark = pytest.mark.gpu

# name: (N, L, E, H, B, T, P, eps, lr, mode, pair_chunk)
CASES = {
    "tiny": (1, 1, 32, 64, 8, 64, 4, 1e-3, 1e-2, 0, 0),
    "ragged_l2": (2, 2, 48, 32, 20, 37, 3, 1e-3, 1e-2, 0, 2),
    "ragged_l2_summed": (2, 2, 48, 32, 20, 37, 3, 1e-3, 1e-2, 1, 2),
    "l3_b70": (3, 3, 16, 80, 70, 9, 2, 2e-3, 5e-3, 0, 0),
    "h512_short": (1, 2, 512, 512, 16, 6, 2, 1e-3, 1e-3, 0, 0),
    "h512_b50": (1, 2, 64, 512, 50, 7, 2, 1e-3, 1e-3, 0, 0),   # four row tiles, rows 50..63 past the batch
    "t2_b1_p1": (1, 2, 32, 64, 1, 2, 1, 1e-3, 1e-2, 0, 0),    # one target per sequence: a single recurrence step
    "h16_fallback": (2, 2, 16, 16, 5, 11, 2, 1e-3, 1e-2, 0, 0),  # H % 64 != 0: per-step and tiled kernels
    "h64_b50_l2": (2, 2, 32, 64, 50, 9, 3, 1e-3, 1e-2, 0, 2),   # one block per job, four row tiles, ragged
    "h64_b20": (1, 1, 48, 64, 20, 13, 2, 1e-3, 1e-2, 0, 0),      # one block per job, two row tiles
    "h64_e64_b33": (1, 2, 64, 64, 33, 10, 2, 1e-3, 1e-2, 0, 0),  # one block per job, embedding in LDS (two chunks)
    "h64_bt_big": (1, 1, 32, 64, 64, 257, 1, 1e-3, 1e-2, 0, 0),  # B T = 16448 > 16 KiB: the fold and per-step gathers
    "b64_h128": (2, 2, 64, 128, 64, 20, 3, 1e-3, 1e-2, 0, 2),
    "h128_b10": (1, 1, 32, 128, 10, 9, 2, 1e-3, 1e-2, 0, 0),     # one-pass head at H = 128, R = 80: a ragged tile
    "b40_h384": (1, 2, 32, 384, 40, 9, 2, 1e-3, 1e-2, 0, 0),    # persistent, 12-wave blocks, four row tiles
    "b32_h384": (2, 2, 48, 384, 32, 11, 3, 1e-3, 1e-2, 0, 2),   # persistent, 12-wave blocks, two row tiles
    "h704_b12": (1, 2, 32, 704, 12, 5, 1, 1e-3, 1e-3, 0, 0),    # persistent at H = 704 (pieces of 64 K), streaming projection and head
    "h704_b64": (1, 2, 32, 704, 64, 6, 2, 1e-3, 1e-3, 0, 0),    # persistent at H = 704 with four row tiles
    "h96_b70": (1, 2, 32, 96, 70, 7, 2, 1e-3, 1e-2, 0, 0),      # per-step split products, two batch groups
    "h96_b24": (2, 1, 32, 96, 24, 6, 2, 1e-3, 1e-2, 0, 0),      # per-step split products, two row tiles
    "h64_e64_b12": (1, 1, 64, 64, 12, 11, 2, 1e-3, 1e-2, 0, 0),  # one block per job, embedding in LDS, one row tile
    "h512_jobs": (1, 2, 32, 512, 56, 4, 12, 1e-3, 1e-3, 0, 0),   # pipelined exchange, 2 jobs in half the groups, ragged last tile
    "h256_b64_jobs": (2, 2, 32, 256, 64, 6, 20, 1e-3, 1e-2, 0, 0),  # pipelined exchange, 32 groups, uneven jobs
    "h192_b64": (1, 2, 32, 192, 64, 7, 3, 1e-3, 1e-2, 0, 0),     # faulted the device with the pipelined exchange (skipped)
    "h128_b64_t3": (2, 1, 32, 128, 64, 3, 2, 1e-3, 1e-2, 0, 0),  # pipelined exchange, two steps per sequence
    "h128_b49_t2": (1, 2, 16, 128, 49, 2, 2, 1e-3, 1e-2, 0, 0),  # one step per sequence (no exchange), one row of tile 4
}


# Longer sequences through the pipelined exchange, for the repeatability test
# only (the oracle would take minutes on them).
LONG_CASES = {
    "h512_b64_t40": (1, 2, 32, 512, 64, 40, 4, 1e-3, 1e-3, 0, 0),   # fragment-order exchange, 39 steps
    "h704_b64_t24": (1, 2, 32, 704, 64, 24, 2, 1e-3, 1e-3, 0, 0),   # 16-byte word exchange, 23 steps
}

# Cases that faulted the device and whose cause is not found: kept, skipped.
FAULTED = {
    "h192_b64": "the pipelined exchange recurrence at H = 192, B = 64 faulted the device (cause not found); "
                "H = 192 now takes the staged recurrence, and this case stays off the device",
}


def run_case(name, distinct=True, data=None, probe=0, head_scale=1.0):
    if name in FAULTED:
        pytest.skip(FAULTED[name])
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name] if name in CASES else LONG_CASES[name]
    shape = soma.Shape(N, L, E, H, B, T, P, mode, pc, probe=probe)
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=distinct)
    if head_scale != 1.0:                      # Whead is the last 256 H parameters of each expert
        theta[:, -256 * H:] *= np.float32(head_scale)
    if data is None:
        data = synth.expert_batches([100 + e for e in range(N)], B, T)
    seeds = synth.expert_seeds(N)
    ctx = soma.Context(shape)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step(th, soma.seeds_tensor(seeds), 0, eps, lr, torch.from_numpy(data).cuda(), losses)
    coef = torch.zeros((N, P), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    return dict(theta0=theta, data=data, seeds=seeds, theta=th.cpu().numpy(),
                losses=losses.cpu().numpy(), coef=coef.cpu().numpy(), shape=shape,
                eps=eps, lr=lr)


def oracle_step(oracle_mod, r):
    s = r["shape"]
    cfg = oracle_mod.make_cfg(s.n_experts, s.n_layers, s.embed, s.hidden, s.batch, s.seq_len,
                              s.n_pairs, s.loss_mode, s.probe)
    return oracle_mod.spsa_step(cfg, r["theta0"], r["seeds"], 0, r["eps"], r["lr"], r["data"])


@pytest.mark.parametrize("name", list(CASES))
def test_step_matches_oracle(oracle_mod, name):
    r = run_case(name)
    o = oracle_step(oracle_mod, r)
    lerr = assert_losses_close(r["losses"], o["losses"])
    terr = assert_theta_close(r["theta"], o["theta"])
    uerr = update_rel_error(r["theta0"], r["theta"], o["theta"])
    cerr = np.abs(r["coef"] - o["coef"]).max() / np.abs(o["coef"]).max()
    print(f"{name}: loss rel {lerr:.2e}  theta rel {terr:.2e}  update rel {uerr:.2e}  coef rel {cerr:.2e}")
    assert not np.array_equal(r["theta"], r["theta0"])


@pytest.mark.parametrize("name", ["tiny", "b64_h128", "h128_b10"])
def test_large_head_weights_match_oracle(oracle_mod, name):
    """Whead scaled 200-fold (row L1 norms near 1000): the one-pass head at
    H <= 128 then subtracts each row's maximum logit before exponentiating
    (below a row L1 norm of 64 on every row it need not, since |h| <= 1
    bounds every logit by it; the other tests run that path)."""
    N, L, E, H = CASES[name][:4]
    r = run_case(name, head_scale=200.0)
    l1 = np.abs(r["theta0"][:, -256 * H:].reshape(N, 256, H)).sum(axis=2).max()
    assert l1 > 64.0
    o = oracle_step(oracle_mod, r)
    lerr = assert_losses_close(r["losses"], o["losses"])
    terr = assert_theta_close(r["theta"], o["theta"])
    print(f"{name} head x200 (row L1 up to {l1:.0f}): loss {r['losses'].mean():.3f}, rel {lerr:.2e}  "
          f"theta rel {terr:.2e}")


@pytest.mark.parametrize("probe", [1, 2])
@pytest.mark.parametrize("name", ["tiny", "ragged_l2_summed", "l3_b70", "h64_e64_b33", "b64_h128", "b40_h384"])
def test_rademacher_step_matches_oracle(oracle_mod, name, probe):
    """Whole steps under the paper's sparse Rademacher law (1) and the dense
    law (2): the tiled kernels (H = 32, 80), the persistent recurrence and the
    streaming projection and head (H = 64, 128, 384)."""
    r = run_case(name, probe=probe)
    o = oracle_step(oracle_mod, r)
    lerr = assert_losses_close(r["losses"], o["losses"])
    terr = assert_theta_close(r["theta"], o["theta"])
    print(f"{name} law {probe}: loss rel {lerr:.2e}  theta rel {terr:.2e}")
    assert not np.array_equal(r["theta"], r["theta0"])


@pytest.mark.parametrize("name", ["tiny", "ragged_l2", "l3_b70", "h64_b50_l2", "b64_h128", "b32_h384",
                                  "h704_b12", "h96_b70"])
def test_eval_loss_matches_oracle(oracle_mod, name):
    """The evaluation runs the step's kernels at radius 0 (split fp16
    products; persistent, one-block or per-step recurrence by shape); the
    reference kernels (fp32 products, one launch per time step, tiled
    weights) run under the execution flags.  Both against the oracle, and
    against each other."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name]
    theta = synth.init_theta(N, L, E, H, init_seed=2, distinct=True) * np.float32(2.0)
    data = synth.expert_batches([200 + e for e in range(N)], B, T)
    ref = oracle_mod.eval_loss(oracle_mod.make_cfg(N, L, E, H, B, T, P), theta, data)
    out = []
    for flags in (0, soma.FLAG_PER_STEP_RECURRENCE | soma.FLAG_TILED_WEIGHTS):
        ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, mode, pc, flags=flags))
        loss = torch.zeros(N, dtype=torch.float32, device="cuda")
        ctx.eval_loss(torch.from_numpy(theta).cuda(), torch.from_numpy(data).cuda(), loss)
        torch.cuda.synchronize()
        out.append(loss.cpu().numpy())
        ctx.close()
        err = assert_losses_close(out[-1], ref)
        print(f"{name} flags {flags}: eval loss rel {err:.2e}")
    np.testing.assert_allclose(out[0], out[1], rtol=2e-5)


def test_eval_loss_full_size(oracle_mod):
    """The N = 2 workload's evaluation at full size (B = 64, T = 256,
    H = 512): both experts' losses against the oracle."""
    torch = require_gpu()
    w = workloads.SOMA_N2
    theta = synth.init_theta(w.n_experts, w.n_layers, w.embed, w.hidden, init_seed=5, distinct=True) * np.float32(2.0)
    data = synth.expert_batches_in_child(w.cluster_seeds, w.batch, w.seq_len)
    ctx = soma.Context(soma.Shape(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, w.n_pairs))
    loss = torch.zeros(w.n_experts, dtype=torch.float32, device="cuda")
    ctx.eval_loss(torch.from_numpy(theta).cuda(), torch.from_numpy(data).cuda(), loss)
    torch.cuda.synchronize()
    ctx.close()
    print("oracle evaluation at full size", flush=True)
    ref = oracle_mod.eval_loss(oracle_mod.cfg_from(w), theta, data)
    err = assert_losses_close(loss.cpu().numpy(), ref)
    print(f"full-size eval loss rel {err:.2e}")


def test_zero_weights_give_ln256():
    torch = require_gpu()
    N, L, E, H, B, T = 2, 2, 32, 32, 4, 17
    shape = soma.Shape(N, L, E, H, B, T, 1)
    ctx = soma.Context(shape)
    data = synth.expert_batches([1, 2], B, T)
    loss = torch.zeros(N, dtype=torch.float32, device="cuda")
    ctx.eval_loss(torch.zeros((N, ctx.d), dtype=torch.float32, device="cuda"),
                  torch.from_numpy(data).cuda(), loss)
    torch.cuda.synchronize()
    assert np.allclose(loss.cpu().numpy(), np.log(256.0), rtol=1e-6)


def test_separability_bit_identity_on_gpu():
    r1 = run_case("ragged_l2")
    data2 = r1["data"].copy()
    data2[1] = synth.expert_batches([999], data2.shape[1], data2.shape[2])[0]
    r2 = run_case("ragged_l2", data=data2)
    assert np.array_equal(r1["theta"][0], r2["theta"][0])
    assert np.array_equal(r1["losses"][0], r2["losses"][0])
    assert not np.array_equal(r1["theta"][1], r2["theta"][1])
    s1 = run_case("ragged_l2_summed")
    s2 = run_case("ragged_l2_summed", data=data2)
    assert not np.array_equal(s1["theta"][0], s2["theta"][0])
    # the forwards are the same in both modes
    assert np.array_equal(r1["losses"], s1["losses"])


@pytest.mark.parametrize("name,probe", [("b64_h128", 2), ("h512_b64_t40", 0), ("h704_b64_t24", 1)])
def test_exchange_recurrence_is_repeatable(name, probe):
    """The same step four times through the pipelined exchange gives
    bit-identical losses and weights: every word of h a block reads was
    published and flagged before its DMA.  A ring word that sometimes reads
    two steps old (halves of one word stored by two waves) passes the oracle
    tolerances on short cases but shows here as run-to-run differences."""
    runs = [run_case(name, probe=probe) for _ in range(4)]
    for r in runs[1:]:
        assert np.array_equal(r["losses"], runs[0]["losses"])
        assert np.array_equal(r["theta"], runs[0]["theta"])


@pytest.mark.parametrize("name,probe", [("h64_b50_l2", 0), ("h64_b50_l2", 1), ("h64_e64_b33", 0)])
def test_local_recurrence_is_repeatable(name, probe):
    """The same step four times through the one-block recurrence at H = 64
    (its h stored for the next layer's projection and the head) gives
    bit-identical losses and weights."""
    runs = [run_case(name, probe=probe) for _ in range(4)]
    for r in runs[1:]:
        assert np.array_equal(r["losses"], runs[0]["losses"])
        assert np.array_equal(r["theta"], runs[0]["theta"])


@pytest.mark.parametrize("name,probe", [("b64_h128", 0), ("b64_h128", 2), ("h256_b64_jobs", 1)])
def test_presplit_sequence_is_bit_identical(name, probe):
    """Layer 1's exchange recurrence stores its h pre-split in fragment order
    and layer 2's projection stages it by DMA (k_proj_dma); with
    SOMA_FLAG_FP32_SEQUENCE the sequence stays fp32 and the streaming
    projection splits it while staging.  Both split the same values the same
    way: losses and weights agree bit for bit."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name]
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = synth.expert_batches([100 + e for e in range(N)], B, T)
    seeds = soma.seeds_tensor(synth.expert_seeds(N))
    outs = []
    for flags in (0, soma.FLAG_FP32_SEQUENCE):
        ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, mode, pc, flags, probe))
        ctx.set_phase_timing(True)
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, seeds, 2, eps, lr, torch.from_numpy(data).cuda(), losses)
        pt = ctx.phase_times()
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy(), pt["xchg_launches"]))
    (t0, l0, x0), (t1, l1, x1) = outs
    assert x0 > 0 and x1 > 0                  # both through the exchange recurrence
    assert np.all(np.isfinite(l0))
    assert np.array_equal(l0, l1)
    assert np.array_equal(t0, t1)


def test_chunking_does_not_change_the_result():
    torch = require_gpu()
    N, L, E, H, B, T, P = 2, 2, 32, 32, 8, 12, 5
    theta = synth.init_theta(N, L, E, H, distinct=True)
    data = synth.expert_batches([7, 8], B, T)
    seeds = soma.seeds_tensor(synth.expert_seeds(N))
    outs = []
    for pc in (0, 1, 2, 5):
        ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, 0, pc))
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, seeds, 4, 1e-3, 1e-2, torch.from_numpy(data).cuda(), losses)
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy()))
    for th, ls in outs[1:]:
        assert np.array_equal(th, outs[0][0]) and np.array_equal(ls, outs[0][1])


@pytest.mark.parametrize("name,probe", [("h512_b50", 0), ("b64_h128", 1), ("h704_b64", 2), ("h512_jobs", 0),
                                        ("h256_b64_jobs", 1), pytest.param("h192_b64", 0, marks=pytest.mark.skip(
                                            reason=FAULTED["h192_b64"])), ("h128_b64_t3", 2), ("h128_b49_t2", 0),
                                        pytest.param("h128_b10", 0, marks=pytest.mark.skip(
                                            reason="two 8-wave exchange blocks per compute unit faulted the device "
                                                   "here; that placement is disabled (cause not found)"))])
def test_exchange_and_staged_recurrence_agree(name, probe):
    """The persistent recurrence with the pipelined split exchange (four row
    tiles in flight, h published once as fp16 parts in fragment order and
    staged by LDS DMA) against the one that stages fp32 h in every block: the
    same split products, the gate inputs added after them instead of before,
    so the results agree within that rounding; the exchange kernel ran once
    per layer and chunk, the staged one not at all."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name]
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = synth.expert_batches([100 + e for e in range(N)], B, T)
    seeds = soma.seeds_tensor(synth.expert_seeds(N))
    outs = []
    for flags in (0, soma.FLAG_STAGED_RECURRENCE):
        ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, mode, pc, flags, probe))
        ctx.set_phase_timing(True)
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, seeds, 3, eps, lr, torch.from_numpy(data).cuda(), losses)
        pt = ctx.phase_times()
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy(), pt["rec_launches"], pt["xchg_launches"]))
    (t0, l0, r0, x0), (t1, l1, r1, x1) = outs
    chunks = (P + (pc or P) - 1) // (pc or P)
    print(f"{name} law {probe}: exchange launches {x0} of {r0}; staged {x1} of {r1}")
    assert x0 == r0 == L * chunks and x1 == 0 and r1 == L * chunks
    assert np.all(np.isfinite(l0))
    rel = np.abs(l0.astype(np.float64) - l1) / np.abs(l1)
    print(f"{name} law {probe}: exchange vs staged loss rel {rel.max():.2e}")
    assert rel.max() <= 1e-5, rel.max()
    assert_theta_close(t0, t1)


@pytest.mark.parametrize("name,probe", [("tiny", 0), ("h512_short", 0), ("h512_b50", 0), ("b64_h128", 0),
                                        ("b40_h384", 0), ("b64_h128", 1), ("h64_b50_l2", 1), ("h64_b20", 0),
                                        ("h64_e64_b33", 2), ("b32_h384", 1), ("h704_b12", 0), ("h704_b64", 2)])
def test_persistent_and_per_step_recurrence_agree(name, probe):
    """The persistent recurrence (weights resident in registers, group
    barriers, products on the fp16 matrix cores from split operands) against
    the per-step launches (fp32 products): one launch per layer and chunk
    against one per time step, and the same losses and update up to the
    split's rounding (about 2^-21 per operand; each path is also held to the
    oracle by the parity tests)."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name]
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = synth.expert_batches([100 + e for e in range(N)], B, T)
    seeds = soma.seeds_tensor(synth.expert_seeds(N))
    outs = []
    for flags in (0, soma.FLAG_PER_STEP_RECURRENCE):
        ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, mode, pc, flags, probe))
        ctx.set_phase_timing(True)
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, seeds, 2, eps, lr, torch.from_numpy(data).cuda(), losses)
        launches = ctx.phase_times()["rec_launches"]
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy(), launches))
    (t0, l0, n0), (t1, l1, n1) = outs
    chunks = (P + (pc or P) - 1) // (pc or P)
    assert n1 == L * (T - 1) * chunks
    assert n0 == L * chunks      # one persistent launch per layer and chunk
    print(f"{name}: recurrence launches persistent={n0} per-step={n1}")
    assert np.all(np.isfinite(l0))
    rel = np.abs(l0.astype(np.float64) - l1) / np.abs(l1)
    print(f"{name} law {probe}: persistent vs per-step loss rel {rel.max():.2e}")
    assert rel.max() <= 1e-5, rel.max()
    assert_theta_close(t0, t1)


@pytest.mark.parametrize("name,probe", [("h96_b70", 2), ("h96_b24", 1)])
def test_split_and_fp32_per_step_recurrence_agree(name, probe):
    """Where the shape rules out the persistent recurrence (H % 64 != 0, or
    B > 64) the per-step launches form their products on the
    fp16 matrix cores from split operands; the per-step flag keeps fp32
    products.  Same launches, per-pair mean losses within 1e-5, the updated
    weights to the parity tolerance (each path is also held to the oracle)."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name]
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = synth.expert_batches([100 + e for e in range(N)], B, T)
    seeds = soma.seeds_tensor(synth.expert_seeds(N))
    outs = []
    for flags in (0, soma.FLAG_PER_STEP_RECURRENCE):
        ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, mode, pc, flags, probe))
        ctx.set_phase_timing(True)
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, seeds, 2, eps, lr, torch.from_numpy(data).cuda(), losses)
        launches = ctx.phase_times()["rec_launches"]
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy(), launches))
    (t0, l0, n0), (t1, l1, n1) = outs
    chunks = (P + (pc or P) - 1) // (pc or P)
    assert n0 == n1 == L * (T - 1) * chunks
    assert np.all(np.isfinite(l0))
    rel = np.abs(l0.astype(np.float64) - l1) / np.abs(l1)
    print(f"{name} law {probe}: split vs fp32 per-step loss rel {rel.max():.2e}")
    assert rel.max() <= 1e-5, rel.max()
    assert_theta_close(t0, t1)


@pytest.mark.parametrize("name,probe", [("tiny", 0), ("h512_short", 0), ("b64_h128", 0), ("b40_h384", 0),
                                        ("h512_short", 1), ("b40_h384", 2), ("h704_b12", 1)])
def test_streaming_and_tiled_weights_agree(name, probe):
    """The streaming projection and head (weights resident in registers,
    probes drawn once per 128 weight rows, products on the fp16 matrix cores
    from split operands) against the tiled kernels (probes regenerated per row
    tile, fp32 products).  The two product paths differ by the split's
    rounding (about 2^-21 per operand), so the per-pair mean losses agree to
    1e-5 relative and the updated weights to the parity tolerance; each path
    is held to the oracle by the parity tests.  The cases cover a ragged last
    row tile (R = 80, 320) and slot counts that are and are not a multiple of
    8 (the two block-to-job mappings)."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name]
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = synth.expert_batches([100 + e for e in range(N)], B, T)
    seeds = soma.seeds_tensor(synth.expert_seeds(N))
    outs = []
    for flags in (0, soma.FLAG_TILED_WEIGHTS):
        ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, mode, pc, flags, probe))
        th = torch.from_numpy(theta.copy()).cuda()
        losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
        ctx.spsa_step(th, seeds, 3, eps, lr, torch.from_numpy(data).cuda(), losses)
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), losses.cpu().numpy()))
    (t0, l0), (t1, l1) = outs
    assert np.all(np.isfinite(l0))
    rel = np.abs(l0.astype(np.float64) - l1) / np.abs(l1)
    print(f"{name} law {probe}: streaming vs tiled loss rel {rel.max():.2e}")
    assert rel.max() <= 1e-5, rel.max()
    assert_theta_close(t0, t1)


def seeded_moments(ghat, seed=7):
    """Adam moments for a whole-step comparison: m ~ N(0, rms(g_hat)/10),
    v ~ U(0.5, 1.5) 30 mean(g_hat^2) (as after earlier, larger estimates).
    With v above g_hat^2 the update lr m_hat / (sqrt(v_hat) + delta) is smooth
    in g_hat (unlike the first step from zero moments, lr sign(g)), so the
    GPU's estimate, which differs from the oracle's by the fp32 noise in
    L+ - L-, gives theta' within the parity bar of the oracle's own step
    (checked on the CPU: coefficients off by 2e-2 of their largest value move
    theta' by at most 8e-5 of the bar's scale), while the update itself is
    about 3e-3 of theta, 30 times the bar."""
    rng = np.random.default_rng(seed)
    g2 = float(np.mean(ghat ** 2))
    m = (rng.standard_normal(ghat.shape) * 0.1 * np.sqrt(g2)).astype(np.float32)
    v = (rng.uniform(0.5, 1.5, ghat.shape) * 30.0 * g2).astype(np.float32)
    return m, v


def adam_oracle_step(oracle_mod, cfg, theta, seeds, step, eps, lr, data, m0, v0, t, adam):
    """The oracle's whole Adam step: its own forwards and coefficients, then
    its Adam update from (m0, v0) -- nothing from the GPU."""
    o = oracle_mod.spsa_step(cfg, theta, seeds, step, eps, lr, data)
    hp = dict(beta1=float(adam.beta1), beta2=float(adam.beta2), delta=float(adam.delta),
              weight_decay=float(adam.weight_decay))
    outs = [oracle_mod.apply_adam(cfg, theta[e], m0[e], v0[e], t, int(seeds[e]), step,
                                  float(np.float32(np.broadcast_to(lr, (len(seeds),))[e])), o["coef"][e], **hp)
            for e in range(len(seeds))]
    return o, [np.stack([x[i] for x in outs]) for i in range(3)]


def assert_moments_close(got, ref, scale, rtol=2e-2):
    """Adam moments carry the estimate itself, whose GPU-vs-oracle difference
    is the fp32 forward noise in L+ - L- (coefficients agree to ~1e-3..2e-2 of
    their largest value), so they are held to that bar relative to the
    moment's scale; theta' is held to the 1e-4 parity bar."""
    err = np.abs(np.asarray(got, np.float64) - ref).max() / scale
    assert err <= rtol, err
    return err


@pytest.mark.parametrize("name,probe", [("ragged_l2", 1), ("b64_h128", 0), ("tiny", 0)])
def test_adam_step_matches_oracle(oracle_mod, name, probe):
    """A whole step with the Adam-style update (update number 3, seeded
    moments) against the oracle's whole step: losses, coefficients and theta'
    at the parity bar, the moments at the coefficients' bar."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES[name]
    shape = soma.Shape(N, L, E, H, B, T, P, mode, pc, probe=probe)
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = synth.expert_batches([100 + e for e in range(N)], B, T)
    seeds = synth.expert_seeds(N)
    cfg = oracle_mod.cfg_from(shape)
    ghat = oracle_mod.spsa_step(cfg, theta, seeds, 0, eps, lr, data, want_ghat=True)["ghat"]
    m0, v0 = seeded_moments(ghat)
    adam = soma.Adam()
    ctx = soma.Context(shape)
    th = torch.from_numpy(theta.copy()).cuda()
    m = torch.from_numpy(m0.copy()).cuda()
    v = torch.from_numpy(v0.copy()).cuda()
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step_adam(th, m, v, 3, adam, soma.seeds_tensor(seeds), 0, eps, lr, torch.from_numpy(data).cuda(),
                       losses)
    coef = torch.zeros((N, P), dtype=torch.float32, device="cuda")
    ctx.coefficients(coef)
    torch.cuda.synchronize()
    o, (to, mo, vo) = adam_oracle_step(oracle_mod, cfg, theta, seeds, 0, eps, lr, data, m0, v0, 3, adam)
    assert_losses_close(losses.cpu().numpy(), o["losses"])
    cerr = np.abs(coef.cpu().numpy() - o["coef"]).max() / np.abs(o["coef"]).max()
    assert cerr <= 2e-2
    terr = assert_theta_close(th.cpu().numpy(), to)
    uerr = update_rel_error(theta, th.cpu().numpy(), to)
    assert uerr <= 5e-2        # the Adam update vector itself, at the coefficients' bar
    merr = assert_moments_close(m.cpu().numpy(), mo, np.abs(mo).max())
    verr = assert_moments_close(v.cpu().numpy(), vo, np.abs(vo).max())
    print(f"{name} law {probe}: coef rel {cerr:.2e}  theta rel {terr:.2e}  update rel {uerr:.2e}  "
          f"m rel {merr:.2e}  v rel {verr:.2e}")
    assert not np.array_equal(th.cpu().numpy(), theta)
    ctx.close()


@pytest.mark.parametrize("name,A,pc", [("ragged_l2", 3, 2), ("b64_h128", 2, 0), ("tiny", 2, 3)])
def test_accumulated_step_matches_oracle(oracle_mod, name, A, pc):
    """Accumulation over A independently sampled batches (direction j on
    batch j / P): the persistent and streaming kernels (b64_h128), the tiled
    ones (ragged_l2, H = 32), and direction chunks that straddle batches
    (P = 3 with chunks of 2; P = 4 with chunks of 3)."""
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, _ = CASES[name]
    shape = soma.Shape(N, L, E, H, B, T, P, mode, pc, accum=A)
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = np.stack([synth.expert_batches([100 + e for e in range(N)], B, T, data_seed=a) for a in range(A)])
    seeds = synth.expert_seeds(N)
    ctx = soma.Context(shape)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((N, A * P, 2), dtype=torch.float32, device="cuda")
    ctx.spsa_step(th, soma.seeds_tensor(seeds), 0, eps, lr, torch.from_numpy(data).cuda(), losses)
    torch.cuda.synchronize()
    cfg = oracle_mod.cfg_from(shape)
    o = oracle_mod.spsa_step(cfg, theta, seeds, 0, eps, lr, data)
    assert_losses_close(losses.cpu().numpy(), o["losses"])
    assert_theta_close(th.cpu().numpy(), o["theta"])
    # the batches differ, so the accumulated losses are not one batch's repeated
    lg = losses.cpu().numpy()
    assert not np.array_equal(lg[:, :P], lg[:, P:2 * P])


def test_persistent_barrier_timeout_aborts_the_step():
    """A persistent recurrence whose group barrier gives up (a spin limit of
    one poll, forced from the host) aborts the whole step: every block leaves
    through its own bounded wait, the losses read NaN and theta is left as it
    was.  The next step on the same context, with the default limit, runs
    normally (the abort flag is cleared per step).  This runs the staged
    kernel, which waits at every step: the pipelined exchange kernel reads
    the flags it needs two sub-steps ahead and almost never waits, so a tiny
    limit does not force its timeout; its drain after an abort is covered by
    the split-range abort (b64_h128 runs it)."""
    flags = soma.FLAG_STAGED_RECURRENCE
    torch = require_gpu()
    N, L, E, H, B, T, P, eps, lr, mode, pc = CASES["b64_h128"]
    theta = synth.init_theta(N, L, E, H, init_seed=1, distinct=True)
    data = torch.from_numpy(synth.expert_batches([100 + e for e in range(N)], B, T)).cuda()
    seeds = soma.seeds_tensor(synth.expert_seeds(N))
    ctx = soma.Context(soma.Shape(N, L, E, H, B, T, P, mode, pc, flags))
    ctx.set_phase_timing(True)
    th = torch.from_numpy(theta.copy()).cuda()
    losses = torch.zeros((N, P, 2), dtype=torch.float32, device="cuda")
    ctx.set_spin_limit(1)
    ctx.spsa_step(th, seeds, 0, eps, lr, data, losses)
    torch.cuda.synchronize()
    chunks = (P + pc - 1) // pc
    pt = ctx.phase_times()
    assert pt["rec_launches"] == L * chunks and pt["xchg_launches"] == 0   # the staged persistent path ran
    assert torch.isnan(losses).all()
    assert np.array_equal(th.cpu().numpy(), theta)
    ctx.set_spin_limit(0)
    ctx.spsa_step(th, seeds, 0, eps, lr, data, losses)
    torch.cuda.synchronize()
    assert torch.isfinite(losses).all()
    assert not np.array_equal(th.cpu().numpy(), theta)
