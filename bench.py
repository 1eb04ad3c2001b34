#!/usr/bin/env python3
"""Benchmark of the SOMA SPSA step (one GPU).

A step is one pass of the whole hot path for every expert: 2P antithetic
perturbed forwards on the expert's own batch (probes regenerated in the weight
tiles), the cross entropies, the loss reduction, the coefficients and the
regenerate-and-update of every parameter.  Inputs (weights, byte batches,
seeds) are resident in device memory before the timed region starts.

Prints ONE JSON line.  ``value`` is the whole-job perturbed-token rate,
N * 2P * B * (T - 1) / seconds per step; ``steps_per_sec`` is 1 / seconds per
step.  ``roofline`` reports the dominant kernel's algorithmic FLOP rate,
measured with HIP events recorded by the library between its launches on the
step's stream, against the fp32 MFMA peak.  ``cpu_baseline`` times the CPU
oracle on a bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "perturbed forward tokens/sec (expert×pert×token) + SPSA steps/sec, 1 GPU"
PEAK_FP32_MFMA_TFLOPS = 157.3   # MI355X dense fp32 matrix peak
PEAK_FP16_MFMA_TFLOPS = 2500.0  # MI355X dense fp16 matrix peak
# Kernels whose products run on the fp16 matrix cores from split fp32
# operands (three fp16 products per fp32 product, fp32 accumulation).
SPLIT_F16_KERNELS = ("k_rec_xchg", "k_rec_persist", "k_rec_local", "k_rec_step_split", "k_proj_stream", "k_proj_dma",
                     "k_head_stream",
                     "k_head_fused", "k_body", "k_wide_mm")
PEAK_HBM_GBS = 8000.0
PROBE_LAWS = {"gaussian": 0, "sparse": 1, "dense": 2}


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="soma_n2_l2_h512")
    ap.add_argument("--pairs", type=int, default=0, help="override the workload's directions per expert")
    ap.add_argument("--pair-chunk", type=int, default=0)
    ap.add_argument("--optimizer", choices=("sgd", "adam"), default="sgd",
                    help="update: the plain step on the estimate, or the paper's Adam-style update "
                         "(beta 0.9/0.999, delta 1e-8, coupled decay 1e-4) with fp32 moments")
    ap.add_argument("--probe", choices=sorted(PROBE_LAWS), default=None,
                    help="probe law (default: the workload's own): gaussian, sparse (the paper's "
                         "training law: 0 w.p. 1/2, +-1 w.p. 1/4) or dense (+-1)")
    ap.add_argument("--loss-mode", choices=("independent", "summed"), default=None,
                    help="coefficients from each expert's own loss (Section 4) or from the summed loss "
                         "(Appendix J); default: the workload's own")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="per-kernel HBM bytes from rocprofv3 counter runs (JSON), if present")
    ap.add_argument("--workers", type=int, default=0,
                    help="processes drawing the synthetic data (0: one per core, up to 16; "
                         "use 1 under a profiler that initialises the GPU before the program)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of 1 GiB (the reference kernel whose "
                         "FETCH_SIZE / WRITE_SIZE scale the HBM traffic counters)")
    return ap.parse_args()


KERNEL_SOURCES = ("paper_2609_37899_amd/csrc/soma_kernels.hpp", "paper_2609_37899_amd/csrc/soma_rng.hpp")
BODY_SOURCES = KERNEL_SOURCES + ("paper_2609_37899_amd/csrc/soma_body.hpp",)
WIDE_SOURCES = BODY_SOURCES + ("paper_2609_37899_amd/csrc/soma_wide.hpp",)


def kernel_source_hash(kernel: str = "") -> str:
    """Hash of a kernel's sources: stored traffic figures apply only to these."""
    import hashlib
    from paper_2609_37899_amd.build import HIPCC_FLAGS
    h = hashlib.sha256()
    h.update(" ".join(HIPCC_FLAGS).encode())
    srcs = BODY_SOURCES if kernel == "k_body" else (WIDE_SOURCES if kernel.startswith("k_wide") else KERNEL_SOURCES)
    for f in srcs:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


def calibrate_copy():
    import torch
    n = 1 << 28                                   # 2^28 fp32 = 1 GiB per buffer
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read_per_copy": 4 * n,
                      "bytes_written_per_copy": 4 * n, "copies": 3}), flush=True)


def kernel_flops(w):
    """Algorithmic contraction FLOPs per step, by kernel class."""
    N, P, B, T, E, H, L = (w.n_experts, w.n_pairs, w.batch, w.seq_len, w.embed, w.hidden,
                           w.n_layers)
    fwd = N * 2 * P                  # perturbed forwards
    tok = B * (T - 1)                # target tokens per forward
    if w.arch == 1:                  # the paper's body: one fused kernel does every product
        return {"rec": fwd * tok * w.flops_per_token, "proj": 0, "fold": 0, "head": 0}
    if w.arch == 2:                  # the wide body: recurrence; A, U, V products; projections + decoder
        return {"rec": fwd * tok * L * 2 * H * 4 * H, "proj": fwd * tok * L * 3 * 2 * H * 4 * H,
                "fold": fwd * tok * 2 * E * H, "head": fwd * tok * 2 * (H * E + E * 256)}
    rec = fwd * tok * L * 2 * H * 4 * H
    proj = fwd * tok * (L - 1) * 2 * H * 4 * H
    emb_in = fwd * tok * 2 * E * 4 * H     # layer-1 input contraction (executed once per byte value)
    head = fwd * tok * 2 * H * 256
    return {"rec": rec, "proj": proj, "fold": emb_in, "head": head}


def cfg_batch(oracle, w, batch, probe, tied_head):
    """The oracle's configuration of workload w with `batch` sequences."""
    return oracle.make_cfg(w.n_experts, w.n_layers, w.embed, w.hidden, batch, w.seq_len, w.n_pairs,
                           w.loss_mode, probe, arch=w.arch, tied_head=tied_head)


def cpu_baseline(w, theta, data, seeds, probe=0, tied_head=None):
    """Time the oracle on a bounded sample of the workload."""
    import oracle
    cfg = oracle.make_cfg(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, w.n_pairs,
                          w.loss_mode, probe, arch=w.arch, tied_head=tied_head)
    threads = oracle.num_threads()
    seq_flops = 2 * (w.seq_len - 1) * w.flops_per_token      # one sequence, both signs
    if w.batch * seq_flops > 4e11:
        # One perturbed forward (direction 0, + sign) of expert 0 on its first
        # b sequences, b sized to about 10 s of oracle work.
        t0 = time.perf_counter()
        oracle.perturbed_loss(cfg_batch(oracle, w, 1, probe, tied_head), theta[0], int(seeds[0]), 0, 0, 1,
                              w.eps, data[0][:1])
        one = time.perf_counter() - t0
        b = int(max(1, min(w.batch, 10.0 // max(one, 1e-3))))
        t0 = time.perf_counter()
        oracle.perturbed_loss(cfg_batch(oracle, w, b, probe, tied_head), theta[0], int(seeds[0]), 0, 0, 1,
                              w.eps, data[0][:b])
        dt = time.perf_counter() - t0
        tokens = b * (w.seq_len - 1)
        sample = (f"expert 0, direction 0, + sign, its first {b} of {w.batch} sequences at T={w.seq_len} "
                  f"({tokens} perturbed tokens of {w.perturbed_tokens} per step; "
                  f"full step extrapolates to {dt * w.perturbed_tokens / tokens:.0f} s)")
        return {"value": tokens / dt, "unit": "perturbed tokens/s", "cores": threads, "kind": "oracle",
                "sample": sample, "seconds": dt}
    if w.perturbed_tokens * w.flops_per_token < 2e10:
        t0 = time.perf_counter()
        oracle.spsa_step(cfg, theta, seeds, 0, w.eps, w.lr, data)
        dt = time.perf_counter() - t0
        tokens = w.perturbed_tokens
        sample = f"full step of {w.name}"
    else:
        # Directions 0, 1, ... of expert 0 (both signs each) until 10 s of
        # oracle work, at most 8.
        t0 = time.perf_counter()
        n = 0
        while n < min(8, w.n_pairs) and (n == 0 or time.perf_counter() - t0 < 10.0):
            for s in (+1, -1):
                oracle.perturbed_loss(cfg, theta[0], int(seeds[0]), 0, n, s, w.eps, data[0])
            n += 1
        dt = time.perf_counter() - t0
        tokens = n * 2 * w.batch * (w.seq_len - 1)
        sample = (f"expert 0, directions 0..{n - 1}, both signs, at full B={w.batch}, T={w.seq_len} "
                  f"({tokens} perturbed tokens of {w.perturbed_tokens} per step; "
                  f"full step extrapolates to {dt * w.perturbed_tokens / tokens:.0f} s)")
    return {"value": tokens / dt, "unit": "perturbed tokens/s", "cores": threads, "kind": "oracle",
            "sample": sample, "seconds": dt}


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; "
                                   f"--gpus {args.gpus} is not supported (experts would shard "
                                   "across GPUs with no communication between them)"}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_37899_amd import soma, synth, workloads

    w = workloads.ALL[args.workload]
    if args.pairs:
        w = w.with_(n_pairs=args.pairs)
    if args.loss_mode:
        w = w.with_(loss_mode=1 if args.loss_mode == "summed" else 0)
    # Inputs are drawn (with a worker pool) before anything touches the GPU.
    tied = None
    if w.arch == 1:   # the paper's width-32 recipe: one frozen tied E shared by every expert
        theta0 = synth.init_body(w.n_experts, w.n_layers, w.hidden, w.init_seed)
        tied = synth.init_tied_head(w.hidden, init_seed=1)
    elif w.arch == 2:  # the wide controls: every expert its own tied E
        theta0 = synth.init_wide(w.n_experts, w.n_layers, w.hidden, w.embed, w.init_seed)
        tied = synth.init_tied_head(w.embed, init_seed=1, n_experts=w.n_experts)
    else:
        theta0 = synth.init_theta(w.n_experts, w.n_layers, w.embed, w.hidden, w.init_seed)
    nb = max(1, min(args.steps + args.warmup, 3))
    batches = [synth.expert_batches(w.cluster_seeds, w.batch, w.seq_len, data_seed=i,
                                    pool=w.pool_clusters,
                                    workers=args.workers or synth.default_workers())
               for i in range(nb)]
    seeds_np = synth.expert_seeds(w.n_experts)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    probe = PROBE_LAWS[args.probe] if args.probe else w.probe
    probe_name = {v: k for k, v in PROBE_LAWS.items()}[probe]
    shape = soma.Shape(w.n_experts, w.n_layers, w.embed, w.hidden, w.batch, w.seq_len, w.n_pairs,
                       w.loss_mode, args.pair_chunk, probe=probe, arch=w.arch)

    ctx = soma.Context(shape, device=dev)
    if tied is not None:
        dtied = torch.from_numpy(tied).to(dev)
        ctx.set_tied_head(dtied, per_expert=w.arch == 2)
    theta = torch.from_numpy(theta0.copy()).to(dev)
    seeds = soma.seeds_tensor(seeds_np, dev)
    dbatches = [torch.from_numpy(b).to(dev) for b in batches]
    losses = torch.zeros((w.n_experts, w.n_pairs, 2), dtype=torch.float32, device=dev)
    if args.optimizer == "adam":
        m_state = torch.zeros_like(theta)
        v_state = torch.zeros_like(theta)
        adam = soma.Adam()

    def one_step(i):
        if args.optimizer == "adam":
            ctx.spsa_step_adam(theta, m_state, v_state, i + 1, adam, seeds, i, w.eps, w.lr,
                               dbatches[i % nb], losses)
        else:
            ctx.spsa_step(theta, seeds, i, w.eps, w.lr, dbatches[i % nb], losses)
    torch.cuda.synchronize()

    for i in range(args.warmup):
        one_step(i)
    torch.cuda.synchronize()

    ctx.set_phase_timing(True)
    phases = {}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        one_step(args.warmup + i)
        pt = ctx.phase_times()          # waits for this step's last event
        for k, v in pt.items():
            phases[k] = phases.get(k, 0) + v
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ctx.set_phase_timing(False)
    sec = (t1 - t0) / args.steps
    lv = losses.cpu().numpy()
    # The unperturbed evaluation (the validation loss the plateau schedule
    # reads), timed apart from the step.
    eval_loss = torch.zeros(w.n_experts, dtype=torch.float32, device=dev)
    ctx.eval_loss(theta, dbatches[0], eval_loss)
    torch.cuda.synchronize()
    te = time.perf_counter()
    for _ in range(3):
        ctx.eval_loss(theta, dbatches[0], eval_loss)
    torch.cuda.synchronize()
    eval_ms = (time.perf_counter() - te) / 3 * 1e3
    assert np.all(np.isfinite(lv)), "non-finite losses"

    # Dominant kernel and its roofline.
    fl = kernel_flops(w)
    # At H = 64 with E = 32 or 64 and B T <= 16 KiB the recurrence block
    # forms layer 1's input product itself (no fold launch).
    local_rec = (w.arch == 0 and w.hidden == 64 and w.batch <= 64
                 and (w.seq_len - 1) * w.batch * 4 * w.hidden * 4 < 2 ** 31)
    if local_rec and w.embed in (32, 64) and w.batch * w.seq_len <= 16384:
        fl["rec"] += fl["fold"]
        fl["fold"] = 0
        if w.n_layers == 1:          # and the head and cross entropy too (no head launch)
            fl["rec"] += fl["head"]
            fl["head"] = 0
    K = args.steps
    ms = {"rec": phases["rec_ms"] / K, "proj": phases["proj_ms"] / K, "fold": phases["fold_ms"] / K,
          "head": phases["head_ms"] / K, "reduce": phases["reduce_ms"] / K,
          "update": phases["update_ms"] / K}
    launches = {"rec": phases["rec_launches"] / K, "proj": max(phases["proj_launches"] / K, 1),
                "fold": 1, "head": 1}
    dom = max(("rec", "proj", "fold", "head"), key=lambda k: ms[k])
    per_launch_flops = fl[dom] / launches[dom]
    avg_launch_s = ms[dom] / 1e3 / launches[dom]
    achieved = per_launch_flops / avg_launch_s / 1e12
    traffic = None
    # The kernels the library picks for this shape (see soma_api.hip):
    # streaming projection and head where H % 64 == 0, H <= 704 and one
    # slot's gate inputs stay under 2^31 bytes (the projection from the
    # pre-split sequence after the exchange recurrence in fragment order with
    # B = 64); the recurrence one block per job at H = 64, else persistent (one
    # launch per layer and chunk) unless it ran per time step (split fp16
    # products where H % 32 == 0).
    streams = (w.hidden % 64 == 0 and w.hidden <= 704
               and (w.seq_len - 1) * w.batch * 4 * w.hidden * 4 < 2 ** 31)
    presplit = (streams and phases.get("xchg_launches", 0) > 0 and w.batch == 64
                and w.hidden in (128, 256, 512))
    kname = {"rec": "k_rec_step_split" if w.hidden % 32 == 0 else "k_rec_step",
             "proj": ("k_proj_dma" if presplit else "k_proj_stream") if streams else "k_proj", "fold": "k_fold",
             "head": ("k_head_fused" if w.hidden <= 128 else "k_head_stream") if streams else "k_head_ce"}[dom]
    if w.arch == 1:
        kname = "k_body"          # the whole perturbed forward, one launch per direction chunk
    elif w.arch == 2:
        kname = {"rec": "k_rec_persist", "proj": "k_wide_mm", "fold": "k_wide_form", "head": "k_wide_head"}[dom]
    elif dom == "rec" and launches["rec"] < w.n_layers * (w.seq_len - 1):
        kname = ("k_rec_local" if local_rec else
                 "k_rec_xchg" if phases.get("xchg_launches", 0) > 0 else "k_rec_persist")
    if os.path.exists(args.traffic):
        try:
            ent = json.load(open(args.traffic)).get(w.name, {}).get(kname)
            if ent and ent.get("source_hash") == kernel_source_hash(kname):
                traffic = ent["hbm_bytes_per_launch"]
        except (OSError, ValueError, KeyError):
            traffic = None
    split = kname in SPLIT_F16_KERNELS
    peak = PEAK_FP16_MFMA_TFLOPS if split else PEAK_FP32_MFMA_TFLOPS
    roof = {"bound": "mfma", "kernel": kname, "achieved": round(achieved, 3),
            "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": traffic,
            "matmul_dtype": "f16 (fp32 operands split hi+lo, three products, fp32 accumulate)" if split else "f32",
            "flops_per_launch": per_launch_flops, "avg_launch_ms": round(avg_launch_s * 1e3, 4),
            "launches_per_step": launches[dom], "kernel_source_hash": kernel_source_hash(kname)}
    if split:
        roof["executed_f16_tflops"] = round(3 * achieved, 3)
        roof["vs_fp32_mfma_peak"] = round(achieved / PEAK_FP32_MFMA_TFLOPS, 4)
    total_flops = w.perturbed_tokens * w.flops_per_token
    out = {
        "metric": METRIC,
        "value": round(w.perturbed_tokens / sec, 1),
        "unit": "perturbed tokens/s",
        "steps_per_sec": round(1.0 / sec, 4),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(sec * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("f32 (matrix products as three fp16 products of split fp32 operands, fp32 accumulation)"
                  if split else "f32"),
        "data": "synthetic: order-2 Markov byte chains, Dirichlet(0.1) rows, one chain per expert",
        "config": {"workload": w.name, "n_experts": w.n_experts, "n_layers": w.n_layers,
                   "embed": w.embed, "hidden": w.hidden, "batch": w.batch, "seq_len": w.seq_len,
                   "n_pairs": w.n_pairs, "forwards_per_expert": 2 * w.n_pairs,
                   "params_per_expert": w.params_per_expert, "eps": w.eps, "lr": w.lr,
                   "loss_mode": "summed" if w.loss_mode else "independent",
                   "probe": probe_name, "optimizer": args.optimizer,
                   "architecture": {1: "paper body (pre-norm residual LSTM + GELU MLP, frozen tied E)",
                                    2: "wide control body (residual LSTM + GELU MLP at d_t with input/output "
                                       "projections to d_E, per-expert tied E)"}.get(w.arch, "stacked LSTM, untied head"),
                   "parallelism": "single GPU, all experts and directions in each launch"},
        "algorithmic_tflops": round(total_flops / sec / 1e12, 3),
        "phase_ms": {k: round(v, 3) for k, v in ms.items()},
        "eval_ms": round(eval_ms, 3),
        "roofline": roof,
        "mean_loss": float(np.mean(lv)),
    }
    # Deterministic teardown: the context's events and the device buffers are
    # released while the runtime is alive, not by the interpreter's exit.
    torch.cuda.synchronize()
    ctx.close()
    del ctx, theta, dbatches, losses
    torch.cuda.synchronize()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, theta0, batches[0], seeds_np, probe, tied)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
