"""Plain NumPy layers of the latent-diffusion UNet (NCHW, PyTorch weight layouts).

Test infrastructure only (see the package docstring).

Every function is the textbook definition of its layer; a matmul is the only
library primitive used for contractions. Tensors are kept in the dtype they
arrive in (fp32 for the UNet; the tests feed fp64 to the brute-force pins).
"""

import numpy as np
from scipy.special import erf


def silu(x):
    """SiLU(x) = x * sigmoid(x) = x / (1 + exp(-x))."""
    return x / (1.0 + np.exp(-x))


def gelu(x):
    """Exact GELU: x * Phi(x) = 0.5 x (1 + erf(x / sqrt(2)))."""
    return (0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))).astype(x.dtype, copy=False)


def linear(x, w, b=None):
    """y = x W^T + b with W stored [out, in] (PyTorch nn.Linear layout)."""
    y = x @ w.T
    if b is not None:
        y = y + b
    return y


def conv2d(x, w, b, stride=1, pad=1):
    """2-D cross-correlation (no kernel flip) with zero padding.

    x [N, Cin, H, W], w [Cout, Cin, kh, kw], b [Cout] -> [N, Cout, Ho, Wo],
    Ho = (H + 2 pad - kh) // stride + 1. Written as a sum over kernel taps of
    one matmul per tap (the contraction over Cin).
    """
    n, cin, h, wd = x.shape
    cout, cin_w, kh, kw = w.shape
    assert cin == cin_w, (cin, cin_w)
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    xp = np.ascontiguousarray(xp.transpose(0, 2, 3, 1))  # [N, Hp, Wp, Cin]
    out = np.zeros((n, ho, wo, cout), dtype=x.dtype)
    for i in range(kh):
        for j in range(kw):
            patch = xp[:, i:i + stride * (ho - 1) + 1:stride, j:j + stride * (wo - 1) + 1:stride, :]
            w_tap = np.ascontiguousarray(w[:, :, i, j].T)  # [Cin, Cout]
            out += (patch.reshape(-1, cin) @ w_tap).reshape(n, ho, wo, cout)
    out += b
    return np.ascontiguousarray(out.transpose(0, 3, 1, 2))


def upsample_nearest2x(x):
    """Nearest-neighbour x2: out[.., y, x] = in[.., y // 2, x // 2]."""
    return x.repeat(2, axis=2).repeat(2, axis=3)


def group_norm(x, groups, gamma, beta, eps):
    """GroupNorm (Wu & He 2018): per sample and group of C/G channels, normalise
    over (C/G, H, W) with the biased variance, then apply the per-channel affine.
    The statistics are taken in fp64 and the result is cast back."""
    n, c, h, w = x.shape
    xg = x.reshape(n, groups, -1).astype(np.float64)
    mu = xg.mean(axis=2, keepdims=True)
    var = ((xg - mu) ** 2).mean(axis=2, keepdims=True)
    y = ((xg - mu) / np.sqrt(var + eps)).reshape(n, c, h, w).astype(x.dtype)
    return y * gamma[None, :, None, None] + beta[None, :, None, None]


def layer_norm(x, gamma, beta, eps):
    """LayerNorm over the last axis (biased variance, fp64 statistics), then affine."""
    x64 = x.astype(np.float64)
    mu = x64.mean(axis=-1, keepdims=True)
    var = ((x64 - mu) ** 2).mean(axis=-1, keepdims=True)
    y = ((x64 - mu) / np.sqrt(var + eps)).astype(x.dtype)
    return y * gamma + beta


def timestep_sinusoid(t, dim):
    """Sinusoidal timestep features of the latent-diffusion UNet: with half = dim/2
    and f_j = exp(-ln(10000) j / half), emb = [cos(t f_j) for j] ++ [sin(t f_j) for j]."""
    half = dim // 2
    j = np.arange(half, dtype=np.float64)
    f = np.exp(-np.log(10000.0) * j / half)
    a = float(t) * f
    return np.concatenate([np.cos(a), np.sin(a)]).astype(np.float32)


def softmax(s, axis=-1):
    """Max-subtracted softmax."""
    m = s.max(axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=axis, keepdims=True)


def attention(xq, xkv, wq, wk, wv, wo, bo, heads):
    """Multi-head scaled dot-product attention (Vaswani et al. 2017) as used in the
    UNet's transformer blocks: Q = xq Wq^T, K = xkv Wk^T, V = xkv Wv^T (no bias),
    heads are contiguous d-wide channel slices, O_h = softmax(Q_h K_h^T / sqrt(d)) V_h,
    out = concat_h(O_h) Wo^T + bo.

    xq [N, Sq, Cq], xkv [N, Skv, Ckv] -> [N, Sq, C]. Loops over (sample, head) so that
    the score matrix of one head is the largest temporary.
    """
    q = linear(xq, wq)
    k = linear(xkv, wk)
    v = linear(xkv, wv)
    n, sq, inner = q.shape
    d = inner // heads
    scale = np.asarray(1.0 / np.sqrt(d), dtype=q.dtype)
    o = np.empty_like(q)
    for b in range(n):
        for h in range(heads):
            sl = slice(h * d, (h + 1) * d)
            p = softmax((q[b, :, sl] @ k[b, :, sl].T) * scale)
            o[b, :, sl] = p @ v[b, :, sl]
    return linear(o, wo, bo)


def geglu_ff(x, w1, b1, w2, b2):
    """GEGLU feed-forward (Shazeer 2020): [a, g] = split(x W1^T + b1) into the first
    and second halves of the projection, h = a * GELU(g), out = h W2^T + b2."""
    u = linear(x, w1, b1)
    half = u.shape[-1] // 2
    return linear(u[..., :half] * gelu(u[..., half:]), w2, b2)
