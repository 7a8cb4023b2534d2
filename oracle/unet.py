"""One evaluation of the latent-diffusion UNet denoiser eps_theta(x_t, t, ctx), NCHW fp32.

Test infrastructure only (see the package docstring).

The module sequence is ``topology.walk``; the weights come from the canonical
fp32 blob (``topology.tensor_table`` order). Block definitions follow the
latent-diffusion UNet (Rombach et al. 2022) as configured for SD-XL
(Podell et al. 2023) — the model the paper serves in AC mode (Sec. 5.1):

ResBlock(x, temb):   h = conv1(SiLU(GN1(x))) + Linear(SiLU(temb))[:, :, None, None]
                     h = conv2(SiLU(GN2(h)));  out = skip(x) + h   (skip = 1x1 conv if Cin != Cout)
Transformer(x, ctx): h = proj_in(tokens(GN(x)));  per block:
                         h += SelfAttn(LN1(h)); h += CrossAttn(LN2(h), ctx); h += GEGLU-FF(LN3(h))
                     out = x + image(proj_out(h))
Downsample: conv3x3 stride 2, pad 1.   Upsample: nearest x2, then conv3x3.
"""

import numpy as np

from . import layers as L
from .topology import tensor_table, walk


def unpack(cfg, blob):
    """Split the flat blob into named fp32 arrays (views), checking its length."""
    table = tensor_table(cfg)
    total = sum(int(np.prod(s)) for _, s, _, _ in table)
    blob = np.asarray(blob, dtype=np.float32)
    if blob.size != total:
        raise ValueError(f"weight blob has {blob.size} floats, topology needs {total}")
    out = {}
    off = 0
    for name, shape, _, _ in table:
        n = int(np.prod(shape))
        out[name] = blob[off:off + n].reshape(shape)
        off += n
    return out


def bf16_model_weights(W):
    """The parameters of the model in bf16 mode: every convolution and linear weight
    matrix of the UNet body rounded to bf16 (nearest, ties to even; the values stay
    fp32 arrays, exactly representable); biases, norm scales and shifts, the time MLP
    (``time.lin*.w``) and the ResBlocks' time projections (``*.temb.w``) are the time
    embedding's and the norms' parameters, which bf16 mode keeps in fp32. Returns a
    new dict; W is not modified."""
    from .sampler import bf16_round
    out = {}
    for k, v in W.items():
        if k.endswith(".w") and not k.startswith("time.") and not k.endswith(".temb.w"):
            out[k] = bf16_round(v).reshape(v.shape)
        else:
            out[k] = v
    return out


def time_embedding(cfg, W, t):
    """temb = lin2(SiLU(lin1(sinusoid(t, C0)))) -> [4 C0]."""
    e = L.timestep_sinusoid(t, cfg.model_channels)
    h = L.linear(e, W["time.lin1.w"], W["time.lin1.b"])
    return L.linear(L.silu(h), W["time.lin2.w"], W["time.lin2.b"])


def resblock(cfg, W, p, x, temb):
    g = cfg.gn_groups
    h = L.silu(L.group_norm(x, g, W[p + ".gn1.g"], W[p + ".gn1.b"], cfg.gn_eps))
    h = L.conv2d(h, W[p + ".conv1.w"], W[p + ".conv1.b"])
    h = h + L.linear(L.silu(temb), W[p + ".temb.w"], W[p + ".temb.b"])[:, :, None, None]
    h = L.silu(L.group_norm(h, g, W[p + ".gn2.g"], W[p + ".gn2.b"], cfg.gn_eps))
    h = L.conv2d(h, W[p + ".conv2.w"], W[p + ".conv2.b"])
    if p + ".skip.w" in W:
        x = L.conv2d(x, W[p + ".skip.w"], W[p + ".skip.b"], pad=0)
    return x + h


def transformer(cfg, W, p, x, ctx, depth, heads, ff_act=None):
    """ff_act: None, or the rounding the quantized variant applies to the feed-forward's
    two inputs (the third LayerNorm's output and the GEGLU output)."""
    n, c, hh, ww = x.shape
    h = L.group_norm(x, cfg.gn_groups, W[p + ".gn.g"], W[p + ".gn.b"], cfg.tx_gn_eps)
    h = h.reshape(n, c, hh * ww).transpose(0, 2, 1)          # tokens in row-major (y, x) order
    h = L.linear(h, W[p + ".proj_in.w"], W[p + ".proj_in.b"])
    for k in range(depth):
        b = f"{p}.blk{k}"
        a = L.layer_norm(h, W[b + ".ln1.g"], W[b + ".ln1.b"], cfg.ln_eps)
        h = h + L.attention(a, a, W[b + ".attn1.q.w"], W[b + ".attn1.k.w"], W[b + ".attn1.v.w"],
                            W[b + ".attn1.o.w"], W[b + ".attn1.o.b"], heads)
        a = L.layer_norm(h, W[b + ".ln2.g"], W[b + ".ln2.b"], cfg.ln_eps)
        h = h + L.attention(a, ctx, W[b + ".attn2.q.w"], W[b + ".attn2.k.w"], W[b + ".attn2.v.w"],
                            W[b + ".attn2.o.w"], W[b + ".attn2.o.b"], heads)
        a = L.layer_norm(h, W[b + ".ln3.g"], W[b + ".ln3.b"], cfg.ln_eps)
        if ff_act is None:
            h = h + L.geglu_ff(a, W[b + ".ff1.w"], W[b + ".ff1.b"], W[b + ".ff2.w"], W[b + ".ff2.b"])
        else:
            u = L.linear(ff_act(a), W[b + ".ff1.w"], W[b + ".ff1.b"])
            half = u.shape[-1] // 2
            g = ff_act(u[..., :half] * L.gelu(u[..., half:]))
            h = h + L.linear(g, W[b + ".ff2.w"], W[b + ".ff2.b"])
    h = L.linear(h, W[p + ".proj_out.w"], W[p + ".proj_out.b"])
    return x + h.transpose(0, 2, 1).reshape(n, c, hh, ww)


def forward(cfg, W, x, t, ctx, ff_act=None):
    """eps_theta for a batch: x [n, latent_c, H, W] fp32, scalar timestep t,
    ctx [n, ctx_len, ctx_dim] fp32 -> [n, latent_c, H, W] fp32. W from ``unpack``;
    ff_act as in ``transformer``."""
    x = np.asarray(x, dtype=np.float32)
    ctx = np.asarray(ctx, dtype=np.float32)
    temb = None
    h = None
    skips = []
    for op in walk(cfg):
        kind = op[0]
        if kind == "time":
            temb = time_embedding(cfg, W, t)[None, :].repeat(x.shape[0], axis=0)
        elif kind == "conv_in":
            h = L.conv2d(x, W["conv_in.w"], W["conv_in.b"])
        elif kind == "push":
            skips.append(h)
        elif kind == "pop_concat":
            h = np.concatenate([h, skips.pop()], axis=1)
        elif kind == "res":
            h = resblock(cfg, W, op[1], h, temb)
        elif kind == "tx":
            _, p, _, depth, heads = op
            h = transformer(cfg, W, p, h, ctx, depth, heads, ff_act)
        elif kind == "down":
            h = L.conv2d(h, W[op[1] + ".w"], W[op[1] + ".b"], stride=2)
        elif kind == "up":
            h = L.conv2d(L.upsample_nearest2x(h), W[op[1] + ".w"], W[op[1] + ".b"])
        elif kind == "out":
            h = L.silu(L.group_norm(h, cfg.gn_groups, W["out.gn.g"], W["out.gn.b"], cfg.gn_eps))
            h = L.conv2d(h, W["conv_out.w"], W["conv_out.b"])
    return h.astype(np.float32)
