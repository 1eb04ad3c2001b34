"""Pin the work accounting used by the benchmark against figures the paper prints.

The paper's training-compute model is C_train = 2 T n_pert B N F_N s
(Appendix H, Eq. training-flops) with F = 81.9k operations per token for a
width-32 expert.  The benchmark's per-token count for the workloads whose
expert costs the same (1-layer LSTM, E = 32, H = 64, 256-way head) must
reproduce F exactly, and the formula must reproduce the printed totals.
"""
import json
import os

from paper_2609_37899_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_compute_accounting.json")


def test_width32_ops_per_token():
    g = json.load(open(GOLDEN))
    assert workloads.TINY.flops_per_token == g["width32_ops_per_token"]["value"]
    assert workloads.SOMA_N256.flops_per_token == g["width32_ops_per_token"]["value"]


def test_training_compute_totals():
    g = json.load(open(GOLDEN))
    F = g["width32_ops_per_token"]["value"]
    for c in g["training_compute_cases"]:
        ops = 2 * c["T"] * c["n_pert"] * c["B"] * c["N"] * F * c["updates"]
        assert abs(ops / c["ops"] - 1) < 0.005, c


def test_perturbed_token_counts():
    # expert x perturbation x target token per step: N * 2P * B * (T - 1)
    assert workloads.SOMA_N2.perturbed_tokens == 2 * 64 * 64 * 255
    assert workloads.SOMA_N2.flops_per_token == 8_650_752
    assert workloads.TINY.perturbed_tokens == 1 * 8 * 8 * 63
