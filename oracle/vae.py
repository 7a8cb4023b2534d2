"""The latent decoder that turns the final denoised latent into the image (the VAE
Decoder component of Table 3, run once after the denoise loop), NCHW fp32.

Test infrastructure only (see the package docstring).

Structure (the KL-autoencoder decoder of latent diffusion, Rombach et al. 2022):
  z / scaling_factor -> post_quant 1x1 conv -> conv_in 3x3 (latent_c -> C_top)
  -> mid: ResBlock, self-attention (one head over all C channels), ResBlock
  -> up levels l = L-1 .. 0 at width C_l: (layers_per_block + 1) ResBlocks, then for
     l > 0 a nearest-x2 upsample followed by a 3x3 conv
  -> GroupNorm, SiLU, conv_out 3x3 (C_0 -> out_c).
ResBlock(x) = skip(x) + conv2(SiLU(GN2(conv1(SiLU(GN1(x)))))) with no time input; skip
is a 1x1 conv when the width changes. Attention(x) = x + proj(softmax(Q K^T / sqrt(C)) V)
over the H*W positions of GN(x), with Q, K, V, proj linear layers with bias.
"""

import numpy as np

from . import layers as L


def tensor_table(cfg):
    """[(name, shape, kind, fan_in)] in the canonical blob order (kind: w, b, g, beta)."""
    t = []

    def wb(name, shape):
        fan = int(np.prod(shape[1:]))
        t.append((name + ".w", tuple(shape), "w", fan))
        t.append((name + ".b", (shape[0],), "b", fan))

    def norm(name, c):
        t.append((name + ".g", (c,), "g", 0))
        t.append((name + ".b", (c,), "beta", 0))

    def res(p, cin, cout):
        norm(p + ".gn1", cin)
        wb(p + ".conv1", (cout, cin, 3, 3))
        norm(p + ".gn2", cout)
        wb(p + ".conv2", (cout, cout, 3, 3))
        if cin != cout:
            wb(p + ".skip", (cout, cin, 1, 1))

    ch = cfg.block_channels
    top = ch[-1]
    wb("post_quant", (cfg.latent_c, cfg.latent_c, 1, 1))
    wb("conv_in", (top, cfg.latent_c, 3, 3))
    res("mid.res0", top, top)
    norm("mid.attn.gn", top)
    for p in ("q", "k", "v", "o"):
        wb("mid.attn." + p, (top, top))
    res("mid.res1", top, top)
    prev = top
    for l in range(len(ch) - 1, -1, -1):
        for j in range(cfg.layers_per_block + 1):
            res(f"up{l}.{j}", prev, ch[l])
            prev = ch[l]
        if l > 0:
            wb(f"up{l}.up", (ch[l], ch[l], 3, 3))
    norm("out.gn", ch[0])
    wb("conv_out", (cfg.out_c, ch[0], 3, 3))
    return t


def unpack(cfg, blob):
    table = tensor_table(cfg)
    total = sum(int(np.prod(s)) for _, s, _, _ in table)
    blob = np.asarray(blob, dtype=np.float32)
    if blob.size != total:
        raise ValueError(f"VAE blob has {blob.size} floats, the decoder needs {total}")
    out, off = {}, 0
    for name, shape, _, _ in table:
        n = int(np.prod(shape))
        out[name] = blob[off:off + n].reshape(shape)
        off += n
    return out


def param_count(cfg):
    return sum(int(np.prod(s)) for _, s, _, _ in tensor_table(cfg))


def flop_count(cfg, batch, h, w):
    """(conv + linear FLOPs, attention-product FLOPs) of one decode of `batch` latents
    of h x w, 2 FLOPs per multiply-add."""
    lin = 0
    att = 0
    ch = cfg.block_channels
    top = ch[-1]

    def conv(cin, cout, hw, k=9):
        return 2 * batch * hw * cout * cin * k

    def res(cin, cout, hw):
        f = conv(cin, cout, hw) + conv(cout, cout, hw)
        return f + (conv(cin, cout, hw, 1) if cin != cout else 0)

    hw = h * w
    lin += conv(cfg.latent_c, cfg.latent_c, hw, 1) + conv(cfg.latent_c, top, hw)
    lin += 2 * res(top, top, hw) + 4 * 2 * batch * hw * top * top
    att += 2 * 2 * batch * hw * hw * top
    prev = top
    for l in range(len(ch) - 1, -1, -1):
        for _ in range(cfg.layers_per_block + 1):
            lin += res(prev, ch[l], hw)
            prev = ch[l]
        if l > 0:
            hw *= 4
            lin += conv(ch[l], ch[l], hw)
    lin += conv(ch[0], cfg.out_c, hw)
    return lin, att


def resblock(cfg, W, p, x):
    g = cfg.gn_groups
    h = L.silu(L.group_norm(x, g, W[p + ".gn1.g"], W[p + ".gn1.b"], cfg.gn_eps))
    h = L.conv2d(h, W[p + ".conv1.w"], W[p + ".conv1.b"])
    h = L.silu(L.group_norm(h, g, W[p + ".gn2.g"], W[p + ".gn2.b"], cfg.gn_eps))
    h = L.conv2d(h, W[p + ".conv2.w"], W[p + ".conv2.b"])
    if p + ".skip.w" in W:
        x = L.conv2d(x, W[p + ".skip.w"], W[p + ".skip.b"], pad=0)
    return x + h


def mid_attention(cfg, W, x):
    n, c, hh, ww = x.shape
    h = L.group_norm(x, cfg.gn_groups, W["mid.attn.gn.g"], W["mid.attn.gn.b"], cfg.gn_eps)
    tok = h.reshape(n, c, hh * ww).transpose(0, 2, 1)           # positions in row-major (y, x) order
    q = L.linear(tok, W["mid.attn.q.w"], W["mid.attn.q.b"])
    k = L.linear(tok, W["mid.attn.k.w"], W["mid.attn.k.b"])
    v = L.linear(tok, W["mid.attn.v.w"], W["mid.attn.v.b"])
    o = np.empty_like(q)
    scale = np.asarray(1.0 / np.sqrt(c), dtype=q.dtype)
    for b in range(n):
        o[b] = L.softmax((q[b] @ k[b].T) * scale) @ v[b]
    o = L.linear(o, W["mid.attn.o.w"], W["mid.attn.o.b"])
    return x + o.transpose(0, 2, 1).reshape(n, c, hh, ww)


def decode(cfg, W, z):
    """Image [B, out_c, 2^(L-1) H, 2^(L-1) W] fp32 from latents z [B, latent_c, H, W]."""
    x = np.asarray(z, dtype=np.float32) / np.float32(cfg.scaling_factor)
    x = L.conv2d(x, W["post_quant.w"], W["post_quant.b"], pad=0)
    x = L.conv2d(x, W["conv_in.w"], W["conv_in.b"])
    x = resblock(cfg, W, "mid.res0", x)
    x = mid_attention(cfg, W, x)
    x = resblock(cfg, W, "mid.res1", x)
    ch = cfg.block_channels
    for l in range(len(ch) - 1, -1, -1):
        for j in range(cfg.layers_per_block + 1):
            x = resblock(cfg, W, f"up{l}.{j}", x)
        if l > 0:
            x = L.conv2d(L.upsample_nearest2x(x), W[f"up{l}.up.w"], W[f"up{l}.up.b"])
    x = L.silu(L.group_norm(x, cfg.gn_groups, W["out.gn.g"], W["out.gn.b"], cfg.gn_eps))
    return L.conv2d(x, W["conv_out.w"], W["conv_out.b"]).astype(np.float32)


def bf16_model_weights(W):
    """The decoder's parameters in bf16 mode: every convolution and linear weight matrix
    rounded to bf16 (nearest, ties to even), except the 1x1 post-quantisation conv,
    which bf16 mode applies in fp32 with the latent; biases and norm parameters stay
    fp32. Returns a new dict."""
    from .sampler import bf16_round
    return {k: (bf16_round(v).reshape(v.shape) if k.endswith(".w") and not k.startswith("post_quant") else v)
            for k, v in W.items()}
