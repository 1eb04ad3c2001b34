"""The workloads the SPSA step is measured and checked on.

Shapes follow the paper's setting (Section 4: byte vocabulary, antithetic
+-eps directions on one shared batch, n_pert = 64, B = 64; Appendix C for the
recurrent experts) at the sizes below.  ``n_pairs`` counts directions; each is
evaluated at +eps and -eps, so an expert runs 2 * n_pairs perturbed forwards.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

from .synth import body_param_count, param_count, wide_param_count


@dataclass(frozen=True)
class Workload:
    name: str
    n_experts: int
    n_layers: int
    embed: int
    hidden: int
    batch: int
    seq_len: int
    n_pairs: int
    eps: float = 1e-3
    lr: float = 1e-3
    loss_mode: int = 0          # 0 independent per-expert losses, 1 summed
    cluster_seeds: tuple = field(default=())
    pool_clusters: bool = False
    init_seed: int = 0
    arch: int = 0               # 0 stacked LSTM, 1 the paper's body (width embed = hidden),
                                # 2 the wide controls' body (width hidden, head width embed)
    probe: int = 0              # probe law: 0 Gaussian, 1 sparse Rademacher, 2 Rademacher

    @property
    def params_per_expert(self) -> int:
        if self.arch == 1:
            return body_param_count(self.n_layers, self.hidden)
        if self.arch == 2:
            return wide_param_count(self.n_layers, self.hidden, self.embed)
        return param_count(self.n_layers, self.embed, self.hidden)

    @property
    def flops_per_token(self) -> int:
        """Contraction work per target token of one perturbed forward:
        2 * sum_l (in_l + H) * 4H + 2 * H * V for the stacked LSTM,
        2 * (D * 16 d^2 + d * V) for the paper's body (per block the gate
        matrix 8 d^2, W1 4 d^2, W2 4 d^2; the decoder d V), and
        2 * (D * 16 d_t^2 + 2 d_E d_t + d_E V) for the wide controls' body
        (the two projections and the decoder at width d_E); elementwise work
        excluded."""
        if self.arch == 1:
            return 2 * (self.n_layers * 16 * self.hidden * self.hidden + self.hidden * 256)
        if self.arch == 2:
            return 2 * (self.n_layers * 16 * self.hidden * self.hidden + 2 * self.embed * self.hidden
                        + self.embed * 256)
        f = 0
        for l in range(self.n_layers):
            f += 2 * ((self.embed if l == 0 else self.hidden) + self.hidden) * 4 * self.hidden
        return f + 2 * self.hidden * 256

    @property
    def perturbed_tokens(self) -> int:
        """Expert x perturbation x target-token count of one SPSA step."""
        return self.n_experts * 2 * self.n_pairs * self.batch * (self.seq_len - 1)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = Workload("tiny_n1_h64", 1, 1, 32, 64, 8, 64, 4, eps=1e-3, lr=1e-2, cluster_seeds=(1,))
SOMA_N2 = Workload("soma_n2_l2_h512", 2, 2, 512, 512, 64, 256, 32, cluster_seeds=(1000, 1001))
SOMA_N4 = Workload("soma_n4_l2_h384", 4, 2, 384, 384, 32, 512, 32,
                   cluster_seeds=(1000, 1001, 1002, 1003))
MONOLITH = Workload("monolith_l2_h704", 1, 2, 704, 704, 64, 256, 128,
                    cluster_seeds=(1000, 1001), pool_clusters=True)
SOMA_N256 = Workload("soma_n256_l1_h64", 256, 1, 32, 64, 16, 256, 32,
                     cluster_seeds=tuple(1000 + c for c in range(256)))

# The paper's width-32 expert (Appendix C: D = 2 blocks, d_t = 32, frozen
# tied E; Appendix E: sparse Rademacher probes, n_pert = 64 directions, B = 64
# sequences of 1,024 bytes), eight experts on the GPU at once.
PAPER_BODY_N8 = Workload("paper_body_n8_d32", 8, 2, 32, 32, 64, 1024, 64,
                         cluster_seeds=tuple(1000 + c for c in range(8)), arch=1, probe=1)

# The paper's N = 2 wider fixed-size control (Table fixed-parameter-counts:
# d_t = 361, d_E = 32, 4.20M body parameters per expert, its own head;
# Appendix C: D = 2 blocks with input and output projections), trained with
# the width-32 recipe's batch (B = 64 sequences of 1,024 bytes, Appendix E)
# and sparse Rademacher probes, 32 directions = 64 perturbed forwards.
WIDE_N2 = Workload("wide_n2_d361", 2, 2, 32, 361, 64, 1024, 32,
                   cluster_seeds=(1000, 1001), arch=2, probe=1)

ALL = {w.name: w for w in (TINY, SOMA_N2, SOMA_N4, MONOLITH, SOMA_N256, PAPER_BODY_N8, WIDE_N2)}
