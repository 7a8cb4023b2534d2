"""Noise schedule, classifier-free guidance and the deterministic DDIM update.

Test infrastructure only (see the package docstring).

The paper fixes N = 50 denoising iterations (Sec. 4.7, Sec. 5.1) and describes
AC as resuming the iteration from step K for the remaining N-K steps
(Sec. 2.1). It does not name the sampler; the workload this oracle checks uses
DDIM with eta = 0 (Song et al. 2021, Eq. 12 with sigma = 0) on a linear beta
schedule over 1000 training steps, and classifier-free guidance
(Ho & Salimans 2022, Eq. 6).
"""

import numpy as np

LINEAR = 0
SCALED_LINEAR = 1


def betas(n_train_steps=1000, beta_start=0.00085, beta_end=0.012, kind=LINEAR):
    """Per-step noise variances beta_i, fp64.

    linear:        beta_i = beta_start + (beta_end - beta_start) * i / (T - 1)
    scaled_linear: beta_i = (sqrt(beta_start) + (sqrt(beta_end) - sqrt(beta_start)) * i / (T - 1))^2
    """
    if kind == LINEAR:
        return np.linspace(beta_start, beta_end, n_train_steps, dtype=np.float64)
    if kind == SCALED_LINEAR:
        return np.linspace(beta_start ** 0.5, beta_end ** 0.5, n_train_steps, dtype=np.float64) ** 2
    raise ValueError(f"unknown beta schedule {kind}")


def alphas_cumprod(b):
    """abar_t = prod_{i <= t} (1 - beta_i), fp64 (DDPM notation, Ho et al. 2020)."""
    return np.cumprod(1.0 - np.asarray(b, dtype=np.float64))


def abar_at(abar, t):
    """abar for timestep t; the sentinel t = -1 means 'clean' (abar = 1)."""
    return 1.0 if t < 0 else float(abar[t])


def default_timesteps(n_steps, n_train_steps=1000):
    """Evenly spaced descending timesteps ("leading" spacing with offset 1),
    followed by the clean sentinel -1: for N = 10 this is [901, 801, ..., 1, -1].
    Only a default: the denoiser takes the timestep list as an input."""
    stride = n_train_steps // n_steps
    ts = [(n_steps - 1 - j) * stride + 1 for j in range(n_steps)]
    return np.array(ts + [-1], dtype=np.int32)


def cfg(eps_uncond, eps_cond, scale):
    """Classifier-free guidance: eps = eps_u + s * (eps_c - eps_u)."""
    return eps_uncond + np.float32(scale) * (eps_cond - eps_uncond)


def ddim_step(x, eps, abar_t, abar_prev):
    """One deterministic DDIM step (eta = 0), written as the two textbook stages.

    x0   = (x - sqrt(1 - abar_t) * eps) / sqrt(abar_t)        (predicted clean sample)
    x'   = sqrt(abar_prev) * x0 + sqrt(1 - abar_prev) * eps    (direction pointing to x_t)

    The coefficients are formed in fp64 and applied in the array's precision.
    """
    dt = x.dtype
    x0 = (x - np.asarray(np.sqrt(1.0 - abar_t), dtype=dt) * eps) / np.asarray(np.sqrt(abar_t), dtype=dt)
    return np.asarray(np.sqrt(abar_prev), dtype=dt) * x0 + np.asarray(np.sqrt(1.0 - abar_prev), dtype=dt) * eps
