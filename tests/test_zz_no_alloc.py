"""soma_spsa_step_noalloc (the step for callers that cannot allocate) against
soma_spsa_step through the C ABI: two calls in a row on one GPU, the second
with a smaller input, each bit for bit equal to the workspace entry point's
result at the same direction chunk (the same kernels), and the shape limit
of the static scratch."""
import numpy as np
import pytest

from gpu_common import require_gpu
from paper_2609_37899_amd import soma, synth

pytestmark = pytest.mark.gpu

# (N, L, E, H, B, T, P, eps, lr): the persistent recurrence at H = 128 (its
# group counters and abort flag live in the scratch), then a smaller shape at
# H = 64 (one block per job).
CALLS = [(2, 2, 64, 128, 16, 12, 3, 1e-3, 1e-2), (1, 1, 32, 64, 4, 32, 2, 1e-3, 1e-2)]


def _inputs(N, L, E, H, B, T, seed):
    theta = synth.init_theta(N, L, E, H, init_seed=seed, distinct=True)
    data = synth.expert_batches([300 + 10 * seed + e for e in range(N)], B, T)
    return theta, data, synth.expert_seeds(N, base=0x50A10000 + seed)


def test_noalloc_step_matches_the_workspace_step():
    torch = require_gpu()
    for i, (N, L, E, H, B, T, P, eps, lr) in enumerate(CALLS):
        shape = soma.Shape(N, L, E, H, B, T, P)
        theta, data, seeds = _inputs(N, L, E, H, B, T, i)
        dseeds = soma.seeds_tensor(seeds)
        dbytes = torch.from_numpy(data).cuda()
        results = []
        for noalloc in (True, False):
            th = torch.from_numpy(theta.copy()).cuda()
            losses = torch.full((N, P, 2), -1.0, dtype=torch.float32, device="cuda")
            if noalloc:
                soma.spsa_step_noalloc(shape, th, dseeds, 5, eps, lr, dbytes, losses)
            else:
                ctx = soma.Context(shape)
                ctx.spsa_step(th, dseeds, 5, eps, lr, dbytes, losses)
            torch.cuda.synchronize()
            results.append((th.cpu().numpy(), losses.cpu().numpy()))
            if not noalloc:
                ctx.close()
        (t0, l0), (t1, l1) = results
        print(f"call {i} (N={N} H={H} B={B} T={T} P={P}): losses {l0.mean():.6f}")
        assert np.all(np.isfinite(l0)) and np.all(l0 > 0)
        assert np.array_equal(l0, l1)
        assert np.array_equal(t0, t1)
        assert not np.array_equal(t0, theta)


def test_noalloc_rejects_shapes_beyond_its_scratch():
    torch = require_gpu()
    shape = soma.Shape(2, 2, 512, 512, 64, 256, 32)   # ~600 MB of workspace per direction
    th = torch.zeros((2, soma.param_count(shape)), dtype=torch.float32, device="cuda")
    losses = torch.zeros((2, 32, 2), dtype=torch.float32, device="cuda")
    with pytest.raises(soma.SomaError) as e:
        soma.spsa_step_noalloc(shape, th, soma.seeds_tensor(synth.expert_seeds(2)), 0, 1e-3, 1e-3,
                               torch.zeros((2, 64, 256), dtype=torch.uint8, device="cuda"), losses)
    assert e.value.code == soma.SOMA_ESHAPE
    assert torch.all(th == 0)
