"""Shared helpers of the GPU parity tests (tolerances and device set-up)."""
import numpy as np
import pytest

LOSS_RTOL = 1e-4      # per-perturbation losses: |dL| <= 1e-4 |L_oracle|
THETA_RTOL = 1e-4     # updated weights: |dtheta| <= 1e-4 max(|theta_oracle|, rms(theta_oracle))


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2609_37899_amd import soma
    soma.load()   # raises if the HIP library is missing: no fallback
    return torch


def assert_losses_close(gpu, ref, rtol=LOSS_RTOL):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(gpu - ref) / np.abs(ref)
    assert err.max() <= rtol, f"max rel loss error {err.max():.3e}"
    return err.max()


def assert_theta_close(gpu, ref, rtol=THETA_RTOL):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    floor = np.sqrt(np.mean(ref ** 2))
    err = np.abs(gpu - ref) / np.maximum(np.abs(ref), floor)
    assert err.max() <= rtol, f"max rel theta error {err.max():.3e}"
    return err.max()


def update_rel_error(theta0, gpu, ref):
    """||dtheta_gpu - dtheta_oracle|| / ||dtheta_oracle|| (reported, not gated)."""
    d_g = np.asarray(gpu, np.float64) - np.asarray(theta0, np.float64)
    d_o = np.asarray(ref, np.float64) - np.asarray(theta0, np.float64)
    return float(np.linalg.norm(d_g - d_o) / max(np.linalg.norm(d_o), 1e-300))
