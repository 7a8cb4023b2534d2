"""fp8 quantisation of the quantized UNet variant (an approximation level, Sec. 4.2:
quantized models count as approximation levels next to smaller models and skipped
iterations).

Test infrastructure only (see the package docstring).

Format: OCP 8-bit floating point E4M3 (1 sign bit, 4 exponent bits with bias 7, 3
mantissa bits; no infinities; largest finite magnitude 448; subnormal quantum 2^-9).
Rounding: to nearest, ties to even, saturating at +-448.

Scheme of the variant: the GEGLU feed-forward's two matrices are stored as E4M3 codes
with one fp32 scale per output row (scale = max_k |w[n][k]| / 448, code = round(w / scale)),
and their inputs (the LayerNorm output and the GEGLU output) are rounded to E4M3 at
scale 1 (both are normalised or products of normalised values, far inside +-448).
"""

import numpy as np

E4M3_MAX = 448.0


def fp8_round(x):
    """x rounded to the nearest E4M3 value (ties to even), saturating at +-448, as fp32."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    # quantum: 2^(e - 3) for a normal magnitude in [2^e, 2^(e+1)), 2^-9 below 2^-6
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -6)))
    q = 2.0 ** (e - 3)
    r = np.rint(a / q) * q            # rint: ties to the even multiple, i.e. the even code
    return (np.sign(x) * np.minimum(r, E4M3_MAX)).astype(np.float32)


def quantize_rows(w):
    """Per-output-row E4M3 quantisation of a weight matrix w [N][K] (fp32): returns
    (the dequantised matrix code * scale [N][K] fp32, scales [N] fp32). The scale and the
    division are fp32 operations, as the library computes them."""
    w = np.asarray(w, dtype=np.float32)
    m = np.abs(w).max(axis=1).astype(np.float32)
    s = (m / np.float32(E4M3_MAX)).astype(np.float32)
    s = np.where(s > 0, s, np.float32(1.0)).astype(np.float32)
    codes = fp8_round((w / s[:, None]).astype(np.float32))
    return (codes * s[:, None]).astype(np.float32), s


def fp8_model_weights(W):
    """The quantized variant's parameters: the bf16 model's (every conv and linear
    matrix of the UNet body rounded to bf16) except the feed-forward matrices, which are
    quantised per row to E4M3 from the fp32 draws (dequantised values)."""
    from .unet import bf16_model_weights
    out = bf16_model_weights(W)
    for k, v in W.items():
        if k.endswith(".ff1.w") or k.endswith(".ff2.w"):
            out[k] = quantize_rows(v)[0]
    return out
