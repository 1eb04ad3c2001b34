"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This module holds no arithmetic of the method itself (no perturbations, no
forward pass, no estimator): only the data and the initial weights that both
the HIP path and the CPU oracle receive.

* Byte batches stand in for the paper's FineWeb-Edu windows (Section 4;
  Appendix D).  Each expert's data cluster is an order-2 Markov chain over the
  256 byte values.  The transition row of context (a, b) in the cluster with
  seed ``cs`` is a Dirichlet(0.1 * 1_256) draw made lazily, the first time the
  context is visited, from numpy's Philox bit generator keyed by
  (cs, 256 a + b), so a row never depends on the order of visits.  The first
  two bytes of a sequence are uniform.  A batch for (cs, data_seed, step)
  draws its uniforms from ``SeedSequence([data_seed, cs, step])``.
* Initial weights are U(-1/sqrt(H), 1/sqrt(H)) from ``SeedSequence([init_seed])``,
  drawn in float64 and rounded to float32; every expert starts from the same
  body (the paper's experts begin as copies of one seed body, Section 4)
  unless ``distinct`` is set.
"""
from __future__ import annotations

import argparse
import os
import subprocess
import sys
import tempfile

import numpy as np

VOCAB = 256
ALPHA = 0.1


class MarkovCluster:
    """One order-2 Markov byte source with lazily drawn Dirichlet(0.1) rows."""

    def __init__(self, cluster_seed: int):
        self.cluster_seed = int(cluster_seed)
        self._index: dict[int, int] = {}
        self._cdf = np.empty((0, VOCAB), dtype=np.float64)

    def _rows(self, ctx: np.ndarray) -> np.ndarray:
        """Row indices (into self._cdf) of the contexts ctx = 256 a + b."""
        new = [int(c) for c in np.unique(ctx) if int(c) not in self._index]
        if new:
            rows = np.empty((len(new), VOCAB), dtype=np.float64)
            for i, c in enumerate(new):
                g = np.random.Generator(np.random.Philox(
                    key=np.array([self.cluster_seed, c], dtype=np.uint64)))
                rows[i] = np.cumsum(g.dirichlet(np.full(VOCAB, ALPHA)))
            rows[:, -1] = 1.0
            base = self._cdf.shape[0]
            self._cdf = np.concatenate([self._cdf, rows])
            for i, c in enumerate(new):
                self._index[c] = base + i
        return np.fromiter((self._index[int(c)] for c in ctx), dtype=np.int64, count=ctx.size)

    def batch(self, batch: int, seq_len: int, data_seed: int = 0, step: int = 0) -> np.ndarray:
        g = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([int(data_seed), self.cluster_seed, int(step)])))
        x = np.empty((batch, seq_len), dtype=np.uint8)
        x[:, : min(2, seq_len)] = g.integers(0, VOCAB, size=(batch, min(2, seq_len)), dtype=np.uint8)
        u = g.random((batch, max(seq_len - 2, 0)))
        for t in range(2, seq_len):
            ctx = x[:, t - 2].astype(np.int64) * VOCAB + x[:, t - 1]
            idx = self._rows(ctx)          # may grow self._cdf
            cdf = self._cdf[idx]
            nxt = (cdf <= u[:, t - 2: t - 1]).sum(axis=1)
            x[:, t] = np.minimum(nxt, VOCAB - 1)
        return x


def _cluster_batch(args):
    seed, batch, seq_len, data_seed, step = args
    return MarkovCluster(seed).batch(batch, seq_len, data_seed, step)


def expert_batches(cluster_seeds, batch: int, seq_len: int, data_seed: int = 0,
                   step: int = 0, pool: bool = False, workers: int = 1) -> np.ndarray:
    """[N][B][T] uint8, one cluster per expert.  With ``pool`` the clusters
    are pooled into ONE expert's batch (B / len(cluster_seeds) sequences from
    each), returned as [1][B][T].  ``workers`` > 1 draws clusters in forked
    worker processes; call it only from a process that has not initialised a
    GPU (or use :func:`expert_batches_in_child`)."""
    seeds = [int(s) for s in cluster_seeds]
    if pool:
        per = batch // len(seeds)
        jobs = [(s, per, seq_len, data_seed, step) for s in seeds]
        rest = batch - per * len(seeds)
        if rest:
            jobs.append((seeds[0], rest, seq_len, data_seed + 1, step))
    else:
        jobs = [(s, batch, seq_len, data_seed, step) for s in seeds]
    if workers > 1 and len(jobs) > 1:
        import multiprocessing as mp
        with mp.get_context("fork").Pool(min(workers, len(jobs))) as p:
            parts = p.map(_cluster_batch, jobs, chunksize=max(1, len(jobs) // (4 * workers)))
    else:
        parts = [_cluster_batch(j) for j in jobs]
    if pool:
        return np.concatenate(parts, axis=0)[None]
    return np.stack(parts)


def default_workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def expert_batches_in_child(cluster_seeds, batch: int, seq_len: int, data_seed: int = 0,
                            step: int = 0, pool: bool = False) -> np.ndarray:
    """Same result as :func:`expert_batches`, drawn by a fresh child Python
    process with a worker pool (safe to call after GPU initialisation)."""
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "bytes.npy")
        seeds = ",".join(str(int(s)) for s in cluster_seeds)
        cmd = [sys.executable, "-m", "paper_2609_37899_amd.synth", "--out", out, "--seeds", seeds,
               "--batch", str(batch), "--seq-len", str(seq_len), "--data-seed", str(data_seed),
               "--step", str(step)] + (["--pool"] if pool else [])
        root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
        subprocess.run(cmd, check=True, cwd=root)
        return np.load(out)


def param_count(n_layers: int, embed: int, hidden: int) -> int:
    """Size of one expert's flat parameter vector (embedding, LSTM layers, head)."""
    d = VOCAB * embed
    for l in range(n_layers):
        d += 4 * hidden * ((embed if l == 0 else hidden) + hidden)
    return d + VOCAB * hidden


def init_theta(n_experts: int, n_layers: int, embed: int, hidden: int, init_seed: int = 0,
               distinct: bool = False) -> np.ndarray:
    """[N][d] float32, U(-1/sqrt(H), 1/sqrt(H))."""
    d = param_count(n_layers, embed, hidden)
    a = 1.0 / np.sqrt(hidden)
    rows = []
    for e in range(n_experts if distinct else 1):
        ss = np.random.SeedSequence([int(init_seed), e] if distinct else [int(init_seed)])
        rows.append(np.random.Generator(np.random.PCG64(ss)).uniform(-a, a, size=d).astype(np.float32))
    if not distinct:
        rows = rows * n_experts
    return np.stack(rows)


def body_param_count(n_layers: int, d: int) -> int:
    """Size of one expert's parameter vector under the paper's body: per
    block g1[d], W[4d][2d], g2[d], W1[4d][d], W2[d][4d], then g_f[d]."""
    return n_layers * (16 * d * d + 2 * d) + d


def init_body(n_experts: int, n_layers: int, d: int, init_seed: int = 0, distinct: bool = False) -> np.ndarray:
    """[N][d_e] float32 for the paper's body: gains 1 + 0.1 N(0, 1) (away
    from 1 so that a gain that is skipped shows), matrices U(-a, a) with
    a = 1 / sqrt(fan-in)."""
    rows = []
    for e in range(n_experts if distinct else 1):
        ss = np.random.SeedSequence([int(init_seed), e, 7] if distinct else [int(init_seed), 7])
        g = np.random.Generator(np.random.PCG64(ss))
        parts = []
        for _ in range(n_layers):
            parts += [1.0 + 0.1 * g.standard_normal(d),
                      g.uniform(-1, 1, 8 * d * d) / np.sqrt(2 * d),
                      1.0 + 0.1 * g.standard_normal(d),
                      g.uniform(-1, 1, 4 * d * d) / np.sqrt(d),
                      g.uniform(-1, 1, 4 * d * d) / np.sqrt(4 * d)]
        parts.append(1.0 + 0.1 * g.standard_normal(d))
        rows.append(np.concatenate(parts).astype(np.float32))
    if not distinct:
        rows = rows * n_experts
    return np.stack(rows)


def wide_param_count(n_layers: int, d_t: int, d_e: int) -> int:
    """Size of one expert's perturbed vector for the wide controls' body:
    16 D d_t^2 + (2D + 1) d_t + 2 d_E d_t (the head E is separate)."""
    return 16 * n_layers * d_t * d_t + (2 * n_layers + 1) * d_t + 2 * d_e * d_t


def init_wide(n_experts: int, n_layers: int, d_t: int, d_e: int, init_seed: int = 0,
              distinct: bool = False) -> np.ndarray:
    """[N][params] float32 for the wide controls' body, in its canonical order
    (P_in [d_t][d_E]; per block A, R, U, V [d_t][4 d_t]; P_out [d_t][d_E];
    gains g1, g2 per block and g_f): matrices U(-a, a) with a = 1 / sqrt(fan-in),
    gains 1 + 0.1 N(0, 1)."""
    rows = []
    d4 = 4 * d_t
    for e in range(n_experts if distinct else 1):
        ss = np.random.SeedSequence([int(init_seed), e, 13] if distinct else [int(init_seed), 13])
        g = np.random.Generator(np.random.PCG64(ss))
        parts = [g.uniform(-1, 1, d_t * d_e) / np.sqrt(d_e)]
        for _ in range(n_layers):
            parts += [g.uniform(-1, 1, d_t * d4) / np.sqrt(2 * d_t),     # A (input half of the gates)
                      g.uniform(-1, 1, d_t * d4) / np.sqrt(2 * d_t),     # R (recurrent half)
                      g.uniform(-1, 1, d_t * d4) / np.sqrt(d_t),         # U
                      g.uniform(-1, 1, d_t * d4) / np.sqrt(d4)]          # V
        parts.append(g.uniform(-1, 1, d_t * d_e) / np.sqrt(d_t))
        parts.append(1.0 + 0.1 * g.standard_normal((2 * n_layers + 1) * d_t))
        rows.append(np.concatenate(parts).astype(np.float32))
    if not distinct:
        rows = rows * n_experts
    return np.stack(rows)


def init_tied_head(d: int, init_seed: int = 0, n_experts: int = 0, scale: float = 0.3) -> np.ndarray:
    """The tied matrix E, N(0, scale^2) entries: [V][d] (shared), or
    [n_experts][V][d] (one per expert) when n_experts > 0."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(init_seed), 11])))
    shape = (n_experts, VOCAB, d) if n_experts > 0 else (VOCAB, d)
    return (scale * g.standard_normal(shape)).astype(np.float32)


def expert_seeds(n_experts: int, base: int = 0x50A10000) -> np.ndarray:
    """Per-expert perturbation stream seeds."""
    return np.arange(n_experts, dtype=np.uint64) + np.uint64(base)


def _main():
    ap = argparse.ArgumentParser(description="draw synthetic Markov byte batches to a .npy file")
    ap.add_argument("--out", required=True)
    ap.add_argument("--seeds", required=True, help="comma-separated cluster seeds")
    ap.add_argument("--batch", type=int, required=True)
    ap.add_argument("--seq-len", type=int, required=True)
    ap.add_argument("--data-seed", type=int, default=0)
    ap.add_argument("--step", type=int, default=0)
    ap.add_argument("--pool", action="store_true")
    a = ap.parse_args()
    seeds = [int(s) for s in a.seeds.split(",")]
    x = expert_batches(seeds, a.batch, a.seq_len, a.data_seed, a.step, a.pool,
                       workers=default_workers())
    np.save(a.out, x)


if __name__ == "__main__":
    _main()
