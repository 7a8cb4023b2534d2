"""Named workloads and seeded synthetic inputs.

This module holds shapes, sizes and seeded random draws only: none of the
denoiser's arithmetic. The test suite and the benchmark use it to feed the
same inputs to the HIP library and to the CPU oracle.

Inputs are synthetic stand-ins for what the paper's worker consumes (Sec. 4.5,
Sec. 4.7): a text-encoder context (77 tokens) per prompt, a prompt embedding
for the cache lookup, and cached intermediate latents. The paper's prompts
(DiffusionDB) and trained weights are not used: weights are random with
variance 1/fan_in, and the context, latents and embeddings are standard normal.
"""

from dataclasses import dataclass, field, replace

import numpy as np

DN_FP32 = 0
DN_BF16 = 1
DN_FP8 = 2


@dataclass
class DnConfig:
    """Mirror of the C ``dn_config`` struct (one UNet model + its sampler schedule)."""
    dtype: int = DN_BF16
    batch: int = 1                      # images; the UNet runs 2*batch (CFG)
    latent_c: int = 4
    latent_h: int = 128
    latent_w: int = 128
    model_channels: int = 320           # C0: sinusoid width; the time embedding is 4*C0
    levels: tuple = ((320, 0, 5, 64), (640, 2, 10, 64), (1280, 10, 20, 64))  # (C, depth, heads, head_dim)
    layers_per_block: int = 2
    mid_depth: int = 10                 # -1: no middle block; 0: Res, Res; >0: Res, Transformer, Res
    tiny_topology: int = 0
    ctx_len: int = 77
    ctx_dim: int = 2048
    ff_mult: int = 4
    gn_groups: int = 32
    gn_eps: float = 1e-5
    tx_gn_eps: float = 1e-6
    ln_eps: float = 1e-5
    n_train_steps: int = 1000
    beta_start: float = 0.00085
    beta_end: float = 0.012
    beta_schedule: int = 0              # 0 linear, 1 scaled_linear

    def with_(self, **kw):
        return replace(self, **kw)


def tiny(dtype=DN_FP32):
    """Tiny denoiser: latent 1x4x16x16, C=64, one ResBlock and one transformer
    block (4 heads x 16, context 77x128), 10 DDIM steps."""
    return DnConfig(dtype=dtype, batch=1, latent_h=16, latent_w=16, model_channels=64,
                    levels=((64, 1, 4, 16),), layers_per_block=1, mid_depth=-1,
                    tiny_topology=1, ctx_dim=128)


def sd15_level(dtype=DN_BF16):
    """SD-1.5-shaped two-level UNet: 64x64 latent, C=320 (8 heads x 40) then C=640 at
    32x32 (10 heads x 64), one transformer per attention stage, context 77x768."""
    return DnConfig(dtype=dtype, batch=1, latent_h=64, latent_w=64, model_channels=320,
                    levels=((320, 1, 8, 40), (640, 1, 10, 64)), layers_per_block=2,
                    mid_depth=1, ctx_dim=768)


def sdxl(dtype=DN_BF16, batch=1):
    """SD-XL-shaped UNet: 128x128 latent; C=320 ResNet-only, C=640 with 2 transformer
    blocks (10 x 64), C=1280 with 10 (20 x 64); context 77x2048; time embedding 1280."""
    return DnConfig(dtype=dtype, batch=batch)


def sdxl_small(dtype=DN_BF16, batch=1):
    """Smaller SD-XL variant: 1 transformer block per 64x64 stage, 4 per 32x32 stage."""
    return DnConfig(dtype=dtype, batch=batch,
                    levels=((320, 0, 5, 64), (640, 1, 10, 64), (1280, 4, 20, 64)), mid_depth=4)


@dataclass
class VaeConfig:
    """Mirror of the C ``dn_vae_config`` struct: the latent decoder run once per image
    after the denoise loop (Table 3's VAE Decoder)."""
    dtype: int = DN_BF16
    batch: int = 1
    latent_c: int = 4
    latent_h: int = 128
    latent_w: int = 128
    block_channels: tuple = (128, 256, 512, 512)   # level widths, slowest-resolution last
    layers_per_block: int = 2                       # the up path runs layers_per_block + 1 ResBlocks per level
    gn_groups: int = 32
    gn_eps: float = 1e-6
    scaling_factor: float = 0.13025                 # the latent is divided by it before decoding
    out_c: int = 3

    def with_(self, **kw):
        return replace(self, **kw)


def sd_vae(dtype=DN_BF16, latent=128, batch=1):
    """The SD / SD-XL latent decoder: widths 128, 256, 512, 512, three ResBlocks per up
    level, one-head attention in the middle block; latent x latent -> 8x larger RGB image
    (128 -> 1024 x 1024 for SD-XL; 64 -> 512 x 512, the size Table 3 counts)."""
    return VaeConfig(dtype=dtype, batch=batch, latent_h=latent, latent_w=latent)


def tiny_vae(dtype=DN_FP32):
    """A two-level decoder (widths 64, 128, one ResBlock pair per level): 8x8 latent ->
    16x16 image. Same module types as the full decoder, small enough for exact checks."""
    return VaeConfig(dtype=dtype, batch=1, latent_h=8, latent_w=8, block_channels=(64, 128), layers_per_block=1)


def sd20_shape():
    """SD 2.0 UNet topology (4 levels, linear projections, context 1024). Used only
    for the parameter / FLOP pins of Table 3; not a benchmark workload."""
    return DnConfig(dtype=DN_BF16, batch=1, latent_h=64, latent_w=64, model_channels=320,
                    levels=((320, 1, 5, 64), (640, 1, 10, 64), (1280, 1, 20, 64), (1280, 0, 20, 64)),
                    layers_per_block=2, mid_depth=1, ctx_dim=1024)


# ----------------------------------------------------------------------------- seeded draws

def weight_blob(table, seed):
    """Flat fp32 weight blob for a weight table [(numel, fan_in, kind)] in canonical
    order, drawn tensor by tensor from one numpy Generator(seed):
    weights and biases ~ N(0, 1/fan_in); norm scales 1 + 0.1 N(0,1); norm shifts 0.1 N(0,1)."""
    rng = np.random.default_rng(seed)
    total = int(sum(int(r[0]) for r in table))
    out = np.empty(total, dtype=np.float32)
    off = 0
    for numel, fan_in, kind in table:
        numel = int(numel)
        z = rng.standard_normal(numel, dtype=np.float32)
        if kind in ("w", "b", 0, 1):
            z *= np.float32(1.0 / np.sqrt(fan_in))
        elif kind in ("g", 2):
            z = np.float32(1.0) + np.float32(0.1) * z
        elif kind in ("beta", 3):
            z *= np.float32(0.1)
        else:
            raise ValueError(kind)
        out[off:off + numel] = z
        off += numel
    return out


def weight_blob_device(table, seed, device):
    """The same recipe as ``weight_blob`` drawn by torch's generator on a GPU (the
    2.56 B-parameter SD-XL blob in about a second instead of half a minute): a flat fp32
    CUDA tensor. A different stream of numbers than ``weight_blob`` for the same seed;
    the tests copy it to the host for the oracle."""
    import torch
    g = torch.Generator(device=device).manual_seed(seed)
    total = int(sum(int(r[0]) for r in table))
    out = torch.empty(total, device=device, dtype=torch.float32)
    off = 0
    for numel, fan_in, kind in table:
        numel = int(numel)
        v = out[off:off + numel]
        if kind in ("w", "b", 0, 1):
            v.normal_(0.0, float(fan_in) ** -0.5, generator=g)
        elif kind in ("g", 2):
            v.normal_(1.0, 0.1, generator=g)
        elif kind in ("beta", 3):
            v.normal_(0.0, 0.1, generator=g)
        else:
            raise ValueError(kind)
        off += numel
    return out


def normal(shape, seed, dtype=np.float32):
    """Standard-normal array from numpy Generator(seed)."""
    return np.random.default_rng(seed).standard_normal(shape, dtype=np.float32).astype(dtype)


def latent(cfg, seed=0):
    """Initial latent [B, C, H, W] fp32 ~ N(0, 1)."""
    return normal((cfg.batch, cfg.latent_c, cfg.latent_h, cfg.latent_w), seed)


def text_ctx(cfg, seed_uncond=1, seed_cond=2):
    """Context [2B, ctx_len, ctx_dim] fp32 ~ N(0, 1): B unconditional rows, then B conditional."""
    u = normal((cfg.batch, cfg.ctx_len, cfg.ctx_dim), seed_uncond)
    c = normal((cfg.batch, cfg.ctx_len, cfg.ctx_dim), seed_cond)
    return np.concatenate([u, c], axis=0)


def cache_embeddings(n, dim, seed=7):
    """Cache of n prompt embeddings [n, dim] fp16: N(0, I) rows normalised to unit
    length in fp32, then rounded to fp16."""
    rng = np.random.default_rng(seed)
    out = np.empty((n, dim), dtype=np.float16)
    step = 1 << 16
    for s in range(0, n, step):
        z = rng.standard_normal((min(step, n - s), dim), dtype=np.float32)
        z /= np.linalg.norm(z, axis=1, keepdims=True)
        out[s:s + z.shape[0]] = z.astype(np.float16)
    return out


def planted_queries(cache, count, seed=9, cos_lo=0.8, cos_hi=0.95):
    """Queries [count, dim] fp16, each q = cos(th) c_j + sin(th) u with c_j a random
    cache row (as fp32), u a random unit vector orthogonal to it and cos(th) ~ U(lo, hi).
    Returns (queries, planted row indices)."""
    rng = np.random.default_rng(seed)
    n, dim = cache.shape
    rows = rng.integers(0, n, size=count)
    qs = np.empty((count, dim), dtype=np.float16)
    for i, j in enumerate(rows):
        c = cache[j].astype(np.float32)
        c = c / np.linalg.norm(c)
        u = rng.standard_normal(dim, dtype=np.float32)
        u -= (u @ c) * c
        u /= np.linalg.norm(u)
        ct = rng.uniform(cos_lo, cos_hi)
        qs[i] = (ct * c + np.sqrt(1.0 - ct * ct) * u).astype(np.float16)
    return qs, rows
