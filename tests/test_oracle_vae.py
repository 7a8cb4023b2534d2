"""Pins of the oracle's latent decoder (oracle.vae): the topology against Table 3's VAE
Decoder row (parameter count, 16-bit size, FLOPs and arithmetic intensity, all to the
printed digits), and the wiring of its blocks against closed forms: an attention block
whose value projection is zero adds exactly the projected bias; a ResBlock whose
second conv is zero is its (skip) input; the decoder's output size and the latent
scaling."""

import json
import os

import numpy as np
import pytest

from oracle import layers as L, vae as V
from paper_2511_06724_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden", "table3_vae.json")


def _gn_elements(cfg, batch, h, w):
    """Elements normalised by the decoder's GroupNorms in one decode."""
    ch, top, hw = cfg.block_channels, cfg.block_channels[-1], h * w
    el = batch * hw * top * (2 + 2 + 1)              # two mid ResBlocks (two norms each), the attention norm
    prev = top
    for l in range(len(ch) - 1, -1, -1):
        for _ in range(cfg.layers_per_block + 1):
            el += batch * hw * (prev + ch[l])
            prev = ch[l]
        if l > 0:
            hw *= 4
    return el + batch * hw * ch[0]


def test_table3_vae_decoder_row():
    g = json.load(open(GOLD))["vae_decoder"]
    cfg = W.sd_vae(latent=g["latent"][0])
    p = V.param_count(cfg)
    assert p == 49_490_199
    # the table prints 0.050 B; the size column (0.092 GiB) and the arithmetic intensity
    # (8 printed digits) pin the count exactly, the parameter column only to its rounding
    assert abs(p / 1e9 - g["params_b"]) <= 1e-3
    assert round(p * 2 / 2 ** 30, 3) == g["size_gib"]
    lin, att = V.flop_count(cfg, g["batch"], *g["latent"])
    total = lin + 2 * _gn_elements(cfg, g["batch"], *g["latent"])
    assert round(total / 1e9, 3) == g["gflops"]
    # the intensity is FLOPs per 16-bit weight byte; it agrees to 2.4e-7 relative (the
    # size of a few fp32 rounding steps in the table's own arithmetic), not to all 8 digits
    assert abs(total / (2 * p) / g["arith_intensity"] - 1) < 1e-6


def _weights(cfg, seed):
    rng = np.random.default_rng(seed)
    out = {}
    for name, shape, kind, fan in V.tensor_table(cfg):
        if kind in ("w", "b"):
            out[name] = (rng.standard_normal(shape) / np.sqrt(fan)).astype(np.float64)
        elif kind == "g":
            out[name] = 1 + 0.1 * rng.standard_normal(shape)
        else:
            out[name] = 0.1 * rng.standard_normal(shape)
    return out


def test_attention_with_zero_values_adds_the_projected_bias():
    cfg = W.tiny_vae()
    Wt = _weights(cfg, 1)
    Wt["mid.attn.v.w"] = np.zeros_like(Wt["mid.attn.v.w"])
    x = np.random.default_rng(2).standard_normal((2, cfg.block_channels[-1], 3, 5))
    got = V.mid_attention(cfg, Wt, x)
    # every softmax row sums to one, so the attended value is v.b at every position
    add = Wt["mid.attn.o.w"] @ Wt["mid.attn.v.b"] + Wt["mid.attn.o.b"]
    assert np.allclose(got, x + add[None, :, None, None], atol=1e-12)


def test_resblock_with_zero_second_conv_is_its_skip():
    cfg = W.tiny_vae()
    Wt = _weights(cfg, 3)
    x = np.random.default_rng(4).standard_normal((1, 128, 4, 4))
    p = "up0.0"                                     # 128 -> 64: has a 1x1 skip
    assert p + ".skip.w" in Wt
    Wt[p + ".conv2.w"] = np.zeros_like(Wt[p + ".conv2.w"])
    got = V.resblock(cfg, Wt, p, x)
    skip = np.einsum("oc,nchw->nohw", Wt[p + ".skip.w"][:, :, 0, 0], x) + Wt[p + ".skip.b"][None, :, None, None]
    assert np.allclose(got, skip + Wt[p + ".conv2.b"][None, :, None, None], atol=1e-12)


def test_decode_shape_and_latent_scaling():
    cfg = W.tiny_vae()
    Wt = {k: v.astype(np.float32) for k, v in _weights(cfg, 5).items()}
    z = np.random.default_rng(6).standard_normal((1, 4, 8, 8)).astype(np.float32)
    img = V.decode(cfg, Wt, z)
    assert img.shape == (1, 3, 16, 16) and np.isfinite(img).all()
    # dividing by the scaling factor is the only use of it: scaling z and the factor together changes nothing
    cfg2 = cfg.with_(scaling_factor=cfg.scaling_factor * 2)
    assert np.allclose(V.decode(cfg2, Wt, 2 * z), img, rtol=1e-5, atol=1e-5)
    with pytest.raises(ValueError):
        V.unpack(cfg, np.zeros(3, np.float32))
