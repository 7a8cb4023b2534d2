"""Pins of the oracle's fp8 quantisation (oracle.quant): the E4M3 rounding against the
format's 256 codes decoded from its definition (every value a fixed point, midpoints to
the even code, saturation at 448), against torch's float8_e4m3fn conversion, and the
per-row weight quantisation's scale and error bound."""

import numpy as np
import torch

from oracle import quant as Q, topology as T, unet as U
from paper_2511_06724_amd import workloads as Wk


def _decode(code):
    s = -1.0 if code & 0x80 else 1.0
    e, m = (code >> 3) & 0xF, code & 7
    if e == 0xF and m == 7:
        return None                                 # NaN codes
    return s * (m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7))


def test_fp8_round_fixed_points_midpoints_saturation():
    vals = sorted({_decode(c) for c in range(256) if _decode(c) is not None})
    assert len(vals) == 253 and max(vals) == 448.0 and min(vals) == -448.0   # +-0 are one value
    v = np.array(vals)
    assert np.array_equal(Q.fp8_round(v), v.astype(np.float32))
    pos = v[v >= 0]
    codes = {val: c for c in range(128) if (val := _decode(c)) is not None}
    for a, b in zip(pos[:-1], pos[1:]):
        mid = (a + b) / 2
        even = a if codes[a] % 2 == 0 else b
        assert Q.fp8_round(mid) == even and Q.fp8_round(-mid) == -even
        assert Q.fp8_round(np.nextafter(mid, 0)) == a and Q.fp8_round(np.nextafter(mid, 1e9)) == b
    assert list(Q.fp8_round([448.0, 464.0, 1e6, -1e6])) == [448.0, 448.0, 448.0, -448.0]


def test_fp8_round_matches_torch():
    x = np.random.default_rng(1).standard_normal(200_000).astype(np.float32) * np.float32(30.0)
    x = x[np.abs(x) <= 448]
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).float().numpy()
    assert np.array_equal(Q.fp8_round(x), t)


def test_quantize_rows_scale_and_error():
    rng = np.random.default_rng(2)
    w = (rng.standard_normal((64, 300)) * rng.uniform(0.01, 3.0, (64, 1))).astype(np.float32)
    w[5] = 0.0
    dq, s = Q.quantize_rows(w)
    m = np.abs(w).max(axis=1)
    assert np.array_equal(s[m > 0], (m[m > 0] / np.float32(448)).astype(np.float32)) and s[5] == 1.0
    assert np.all(dq[5] == 0)
    # the largest entry of each row is exactly +-448 codes
    assert np.allclose(np.abs(dq).max(axis=1)[m > 0], m[m > 0], rtol=1e-6)
    # error bound: half an E4M3 quantum of the scaled value (relative 2^-4 for normal codes)
    scaled = np.abs(w) / s[:, None]
    q = np.where(scaled >= 2.0 ** -6, 2.0 ** (np.floor(np.log2(np.maximum(scaled, 2.0 ** -6))) - 3), 2.0 ** -9)
    assert np.all(np.abs(dq - w) <= 0.5 * q * s[:, None] * (1 + 1e-6) + 1e-30)


def test_fp8_model_weights_touch_only_the_feed_forward():
    cfg = Wk.tiny()
    blob = Wk.weight_blob([(int(np.prod(s)), f, k) for _, s, k, f in T.tensor_table(cfg)], 4)
    W = U.unpack(cfg, blob)
    W8, W16 = Q.fp8_model_weights(W), U.bf16_model_weights(W)
    ff = [k for k in W if k.endswith(".ff1.w") or k.endswith(".ff2.w")]
    assert len(ff) == 2
    for k in W:
        if k in ff:
            assert np.array_equal(W8[k], Q.quantize_rows(W[k])[0])
        else:
            assert np.array_equal(W8[k], W16[k])


def test_ff_act_hook_identity_and_effect():
    """With the identity as the feed-forward rounding the UNet is unchanged; with E4M3
    rounding it moves by roughly the format's relative precision."""
    from oracle import sampler
    cfg = Wk.tiny()
    blob = Wk.weight_blob([(int(np.prod(s)), f, k) for _, s, k, f in T.tensor_table(cfg)], 5)
    W = U.unpack(cfg, blob)
    x, ctx = Wk.latent(cfg, 0), Wk.text_ctx(cfg)
    ref = U.forward(cfg, W, np.concatenate([x, x]), 901, ctx)
    same = U.forward(cfg, W, np.concatenate([x, x]), 901, ctx, ff_act=lambda a: a)
    assert np.array_equal(ref, same)
    q = sampler.step(cfg, W, x, ctx, 901, 801, 7.5, ff_act=Q.fp8_round)[0]
    d = np.linalg.norm(q - ref) / np.linalg.norm(ref)
    assert 1e-4 < d < 5e-2
