"""Host checks of the benchmark's accounting (no GPU).

The roofline figures divide algorithmic work by measured time, so the work
must be the contraction count of the model: for one perturbed forward of
the stacked LSTM, every target token costs 2 H 4H FLOP per layer in the
recurrence, 2 H 4H per layer >= 2 in the input projection and 2 H 256 in
the head.  These are written out here from the model's shapes."""
import json
import os
import subprocess
import sys

from paper_2609_37899_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_n2_workload_work_per_launch():
    w = workloads.ALL["soma_n2_l2_h512"]
    f = bench.kernel_flops(w)
    slots = 2 * 2 * 32                       # experts x signs x directions
    rows = 64 * 255                          # B (T - 1) targets per forward
    per_layer = 2 * rows * 512 * 2048 * slots
    assert per_layer == 4_380_866_641_920    # one recurrence launch
    assert f["rec"] == 2 * per_layer         # two layers
    assert f["proj"] == per_layer            # layer 2's input contraction
    assert f["head"] == 2 * rows * 512 * 256 * slots
    assert w.perturbed_tokens == slots * rows == 2_088_960


def test_every_workload_counts_each_contraction_once():
    for name, w in workloads.ALL.items():
        if w.arch != 0:
            continue
        f = bench.kernel_flops(w)
        fwd_tokens = w.n_experts * 2 * w.n_pairs * w.batch * (w.seq_len - 1)
        H, E, L = w.hidden, w.embed, w.n_layers
        assert f["rec"] == fwd_tokens * L * 8 * H * H, name
        assert f["proj"] == fwd_tokens * (L - 1) * 8 * H * H, name
        assert f["fold"] == fwd_tokens * 8 * E * H, name
        assert f["head"] == fwd_tokens * 512 * H, name


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]
