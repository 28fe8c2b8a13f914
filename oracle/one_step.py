"""fp64 CPU oracle for FastVR's one-step latent update (Sec. 3.2, Eq. 9).

TEST INFRASTRUCTURE ONLY: used by tests/ and the benchmark's baseline leg; the
HIP library never imports, links or calls it.

Inference (Sec. 4.1) and Stage II training (Sec. 3.2) restore the latent with a
single update from the LQ endpoint at t = tau:

    z_hat = z_LQ - sigma_tau * v

where v is the velocity the DiT predicts at (z_LQ, tau) and sigma_tau the noise
level of tau.  The paper does not give sigma_tau numerically (it names the point
of a shifted schedule closest to timestep 399), so sigma is an input.
"""
from __future__ import annotations

import numpy as np


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):
        import torch
        return x.detach().to("cpu", torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def one_step_update(z_lq, v, sigma: float) -> np.ndarray:
    """Eq. 9 element by element in float64: z_lq - sigma * v (same shape)."""
    z = _f64(z_lq)
    vv = _f64(v)
    if z.shape != vv.shape:
        raise ValueError(f"shape mismatch: z_lq {z.shape} v {vv.shape}")
    return z - float(sigma) * vv


def target_velocity(z_lq, z_hq, sigma: float) -> np.ndarray:
    """Eq. 4: the velocity of the linear LQ-to-HQ trajectory (Eq. 3) with respect
    to sigma, (z_LQ - z_HQ) / sigma_tau, in float64."""
    return (_f64(z_lq) - _f64(z_hq)) / float(sigma)
