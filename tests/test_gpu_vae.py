"""Latent decoder parity on the GPU (dn_vae_create / dn_vae_decode) against the oracle
(oracle.vae.decode) on the same seeded weights and latents.

Bars (relative L2 over the whole image): fp32 mode 1e-4; bf16 mode 2e-2, taken against
the oracle on the bf16 decoder's weights (the seeded draws rounded to bf16, as
dn_vae_create stores them), with the distance to the unrounded weights reported and
bounded at 3e-2. The decode is deterministic (bitwise equal reruns)."""

import numpy as np
import pytest
import torch

from oracle import vae as OV
from paper_2511_06724_amd import dn, workloads as W
from tests.gpu_util import DEV, announce, f32_dev, rel_l2

pytestmark = pytest.mark.gpu


def _decode(cfg, blob, z, twice=False):
    dec = dn.Decoder(cfg, blob)
    s = 1 << (len(cfg.block_channels) - 1)
    img = torch.empty((cfg.batch, cfg.out_c, cfg.latent_h * s, cfg.latent_w * s), device=DEV)
    zd = f32_dev(z)
    dec.decode(zd, img)
    out = [img.clone()]
    if twice:
        dec.decode(zd, img)
        out.append(img.clone())
    torch.cuda.synchronize()
    dec.close()
    return [o.cpu().numpy() for o in out]


@pytest.mark.parametrize("batch", [1, 2])
def test_tiny_decoder_fp32(batch):
    announce(f"vae tiny fp32 batch={batch}")
    cfg = W.tiny_vae(W.DN_FP32).with_(batch=batch)
    blob = W.weight_blob(dn.vae_weight_table(cfg), 21)
    z = W.normal((batch, 4, 8, 8), 22)
    got = _decode(cfg, blob, z)[0]
    ref = OV.decode(cfg, OV.unpack(cfg, blob), z)
    e = rel_l2(got, ref)
    announce(f"  rel-L2 {e:.3e}")
    assert got.shape == (batch, 3, 16, 16)
    assert e <= 1e-4


def _bf16_case(cfg, seed, blob=None):
    blob = W.weight_blob(dn.vae_weight_table(cfg), seed) if blob is None else blob
    z = W.normal((cfg.batch, cfg.latent_c, cfg.latent_h, cfg.latent_w), seed + 1)
    got, again = _decode(cfg, blob, z, twice=True)
    assert np.array_equal(got, again)
    Wt = OV.unpack(cfg, blob)
    ref16 = OV.decode(cfg, OV.bf16_model_weights(Wt), z)
    e16 = rel_l2(got, ref16)
    announce(f"  vs oracle on the bf16 decoder: rel-L2 {e16:.3e}")
    ref32 = OV.decode(cfg, Wt, z)
    e32 = rel_l2(got, ref32)
    announce(f"  vs oracle on the unrounded weights: {e32:.3e} (weight rounding alone {rel_l2(ref16, ref32):.3e})")
    assert np.isfinite(got).all()
    assert e16 <= 2e-2 and e32 <= 3e-2


def test_tiny_decoder_bf16():
    announce("vae tiny bf16")
    _bf16_case(W.tiny_vae(W.DN_BF16), 31)


def test_sd_decoder_512_bf16():
    """Table 3's configuration: the 49.5 M-parameter decoder, 64x64 latent -> 512x512
    image (2.48 TFLOP; attention over 4096 positions)."""
    announce("vae sd 64x64 -> 512x512 bf16 (oracle ~2.5 TFLOP on the host)")
    _bf16_case(W.sd_vae(W.DN_BF16, latent=64), 41)


@pytest.mark.timeout(900)
def test_sdxl_decoder_1024_bf16():
    """The SD-XL image size: 128x128 latent -> 1024x1024 image (9.9 TFLOP; one 512-wide
    attention head over 16384 positions, a 16384 x 16384 score matrix)."""
    announce("vae 128x128 -> 1024x1024 bf16 (oracle ~10.5 TFLOP on the host)")
    cfg = W.sd_vae(W.DN_BF16, latent=128)
    blob = W.weight_blob_device(dn.vae_weight_table(cfg), 51, DEV).cpu().numpy()
    _bf16_case(cfg, 51, blob)


def test_decoder_config_errors():
    announce("vae config errors")
    base = W.tiny_vae(W.DN_BF16)
    for bad in (base.with_(latent_h=7), base.with_(block_channels=(64, 96)), base.with_(scaling_factor=0.0),
                base.with_(batch=0), base.with_(block_channels=(64, 64, 64, 64, 64))):
        with pytest.raises((dn.DnError, IndexError)):
            dn.vae_weight_table(bad)
    n = sum(t[0] for t in dn.vae_weight_table(base))
    with pytest.raises(dn.DnError):
        dn.Decoder(base, np.zeros(n - 1, np.float32))
