"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This module holds no arithmetic of the method itself (no perturbations, no
forward pass, no estimator): only the data and the initial weights that both
the HIP path and the CPU oracle receive.

* Byte batches stand in for the paper's FineWeb-Edu windows (Section 4;
  Appendix D).  Each expert's data cluster is an order-2 Markov chain over the
  256 byte values whose transition row for context (a, b) is a
  Dirichlet(0.1 * 1_256) draw, generated lazily from
  ``SeedSequence([cluster_seed, a, b])``.  The first two bytes of a sequence
  are uniform.  A batch for (cluster_seed, data_seed, step) draws from
  ``SeedSequence([data_seed, cluster_seed, step])``.
* Initial weights are U(-1/sqrt(H), 1/sqrt(H)) from ``SeedSequence([init_seed])``,
  drawn in float64 and rounded to float32; every expert starts from the same
  body ("branch: copy seed body", Section 4) unless ``distinct`` is set.
"""
from __future__ import annotations

import numpy as np

VOCAB = 256
ALPHA = 0.1


class MarkovCluster:
    """One order-2 Markov byte source with lazily drawn Dirichlet(0.1) rows."""

    def __init__(self, cluster_seed: int):
        self.cluster_seed = int(cluster_seed)
        self._cdf: dict[int, np.ndarray] = {}

    def cdf(self, a: int, b: int) -> np.ndarray:
        key = (a << 8) | b
        row = self._cdf.get(key)
        if row is None:
            g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.cluster_seed, a, b])))
            p = g.dirichlet(np.full(VOCAB, ALPHA))
            row = np.cumsum(p)
            row[-1] = 1.0
            self._cdf[key] = row
        return row

    def batch(self, batch: int, seq_len: int, data_seed: int = 0, step: int = 0) -> np.ndarray:
        g = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([int(data_seed), self.cluster_seed, int(step)])))
        x = np.empty((batch, seq_len), dtype=np.uint8)
        x[:, : min(2, seq_len)] = g.integers(0, VOCAB, size=(batch, min(2, seq_len)), dtype=np.uint8)
        u = g.random((batch, max(seq_len - 2, 0)))
        for t in range(2, seq_len):
            for b in range(batch):
                row = self.cdf(int(x[b, t - 2]), int(x[b, t - 1]))
                x[b, t] = min(int(np.searchsorted(row, u[b, t - 2], side="right")), VOCAB - 1)
        return x


def expert_batches(cluster_seeds, batch: int, seq_len: int, data_seed: int = 0,
                   step: int = 0, pool: bool = False) -> np.ndarray:
    """[N][B][T] uint8.  With ``pool`` the clusters are pooled into ONE expert's
    batch (B/len(cluster_seeds) sequences from each), returned as [1][B][T]."""
    clusters = [MarkovCluster(s) for s in cluster_seeds]
    if pool:
        per = batch // len(clusters)
        parts = [c.batch(per, seq_len, data_seed, step) for c in clusters]
        rest = batch - per * len(clusters)
        if rest:
            parts.append(clusters[0].batch(rest, seq_len, data_seed + 1, step))
        return np.concatenate(parts, axis=0)[None]
    return np.stack([c.batch(batch, seq_len, data_seed, step) for c in clusters])


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
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(init_seed), e] if distinct else [int(init_seed)])))
        rows.append(g.uniform(-a, a, size=d).astype(np.float32))
    if not distinct:
        rows = rows * n_experts
    return np.stack(rows)


def expert_seeds(n_experts: int, base: int = 0x50A10000) -> np.ndarray:
    """Per-expert perturbation stream seeds."""
    return np.arange(n_experts, dtype=np.uint64) + np.uint64(base)
