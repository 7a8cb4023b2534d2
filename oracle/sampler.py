"""The denoise loop with classifier-free guidance and DDIM, resumable at step k.

Test infrastructure only (see the package docstring).

Approximate caching (Sec. 2.1; worker behaviour in Sec. 4.5 and Sec. 4.7) takes
the intermediate latent of a cached prompt at iteration K and runs the
remaining N-K iterations conditioned on the new prompt. Here that is
``denoise(..., start_step=K, n_steps=N-K)``: the latent passed in is x at
``timesteps[K]``, and iteration i (K <= i < K+n) maps x at ``timesteps[i]`` to
x at ``timesteps[i+1]`` (the sentinel -1 stands for the clean sample).
"""

import numpy as np

from . import schedule as S
from .unet import forward


def abar_table(cfg):
    return S.alphas_cumprod(S.betas(cfg.n_train_steps, cfg.beta_start, cfg.beta_end, cfg.beta_schedule))


def step(cfg, W, x, ctx, t, t_prev, cfg_scale, abar=None, ff_act=None):
    """One guided DDIM iteration for a batch of B latents.

    x [B, c, H, W] fp32; ctx [2B, L, D] = B unconditional then B conditional rows.
    The UNet runs once on [x; x] (effective batch 2B). Returns
    (eps_raw [2B, c, H, W], eps_guided [B, c, H, W], x_next [B, c, H, W]). ff_act: the
    quantized variant's rounding of the feed-forward inputs (unet.transformer)."""
    if abar is None:
        abar = abar_table(cfg)
    b = x.shape[0]
    eps_raw = forward(cfg, W, np.concatenate([x, x], axis=0), t, ctx, ff_act)
    eps = S.cfg(eps_raw[:b], eps_raw[b:], cfg_scale)
    x_next = S.ddim_step(x, eps, S.abar_at(abar, t), S.abar_at(abar, t_prev))
    return eps_raw, eps, x_next.astype(np.float32)


def denoise(cfg, W, x, ctx, timesteps, start_step, n_steps, cfg_scale, trace=None):
    """Run iterations start_step .. start_step + n_steps - 1; returns the final latent.
    If ``trace`` is a list, the latent after every iteration is appended to it."""
    ts = np.asarray(timesteps)
    if start_step < 0 or n_steps < 0 or start_step + n_steps + 1 > ts.size:
        raise ValueError("timesteps too short for start_step + n_steps")
    abar = abar_table(cfg)
    x = np.asarray(x, dtype=np.float32).copy()
    for i in range(start_step, start_step + n_steps):
        _, _, x = step(cfg, W, x, ctx, int(ts[i]), int(ts[i + 1]), cfg_scale, abar)
        if trace is not None:
            trace.append(x.copy())
    return x


def bf16_round(x):
    """fp32 -> bf16 -> fp32 with round-to-nearest, ties to even: keep the upper 16
    bits of the IEEE single after adding half a unit of the kept part (0x7fff) plus
    the kept part's lowest bit (which breaks a tie towards the even neighbour).
    Finite inputs only."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
    return b.astype(np.uint32).view(np.float32)


def denoise_capture(cfg, W, x, ctx, timesteps, start_step, n_steps, cfg_scale, capture_at):
    """The cache write of Sec. 4.7 (a prompt's run stores its intermediate states at
    K): runs `denoise` and returns (final latent, [bf16_round(latent after K
    iterations) for K in capture_at]); K = start_step is the input latent."""
    for k in capture_at:
        if not start_step <= k <= start_step + n_steps:
            raise ValueError("capture iteration outside [start_step, start_step + n_steps]")
    trace = [np.asarray(x, dtype=np.float32).copy()]
    final = denoise(cfg, W, x, ctx, timesteps, start_step, n_steps, cfg_scale, trace=trace)
    return final, [bf16_round(trace[k - start_step]) for k in capture_at]
