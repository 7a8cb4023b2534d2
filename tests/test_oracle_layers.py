"""Pins of the oracle's layer primitives against brute force, closed forms and invariants.

Each brute-force reference here is an explicit loop over the definition, on inputs
small enough for pure Python, in fp64.
"""

import math

import numpy as np
import pytest

from oracle import layers as L


def _direct_conv(x, w, b, stride, pad):
    n, cin, h, wd = x.shape
    cout, _, kh, kw = w.shape
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    out = np.zeros((n, cout, ho, wo))
    for s in range(n):
        for o in range(cout):
            for y in range(ho):
                for xx in range(wo):
                    acc = b[o]
                    for c in range(cin):
                        for i in range(kh):
                            for j in range(kw):
                                iy = y * stride + i - pad
                                ix = xx * stride + j - pad
                                if 0 <= iy < h and 0 <= ix < wd:
                                    acc += x[s, c, iy, ix] * w[o, c, i, j]
                    out[s, o, y, xx] = acc
    return out


@pytest.mark.parametrize("shape,cout,stride,k", [
    ((2, 3, 5, 6), 4, 1, 3), ((1, 5, 7, 7), 3, 2, 3), ((2, 2, 6, 4), 5, 2, 3), ((1, 4, 3, 3), 2, 1, 1)])
def test_conv_matches_direct_sum(shape, cout, stride, k):
    rng = np.random.default_rng(1)
    x = rng.standard_normal(shape)
    w = rng.standard_normal((cout, shape[1], k, k))
    b = rng.standard_normal(cout)
    pad = k // 2
    got = L.conv2d(x, w, b, stride=stride, pad=pad)
    np.testing.assert_allclose(got, _direct_conv(x, w, b, stride, pad), rtol=1e-12, atol=1e-12)


def test_conv_of_upsampled_input_matches_direct_sum():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((1, 3, 3, 4))
    up = L.upsample_nearest2x(x)
    for y in range(6):
        for xx in range(8):
            assert np.array_equal(up[:, :, y, xx], x[:, :, y // 2, xx // 2])
    w = rng.standard_normal((2, 3, 3, 3))
    b = rng.standard_normal(2)
    np.testing.assert_allclose(L.conv2d(up, w, b), _direct_conv(up, w, b, 1, 1), rtol=1e-12, atol=1e-12)


def test_conv_special_cases():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 4, 5, 5))
    # centre-tap identity kernel returns the input
    w = np.zeros((4, 4, 3, 3))
    for c in range(4):
        w[c, c, 1, 1] = 1.0
    np.testing.assert_array_equal(L.conv2d(x, w, np.zeros(4)), x)
    # a 1x1 conv is a matmul over channels
    w1 = rng.standard_normal((3, 4, 1, 1))
    ref = np.einsum("nchw,oc->nohw", x, w1[:, :, 0, 0])
    np.testing.assert_allclose(L.conv2d(x, w1, np.zeros(3), pad=0), ref, rtol=1e-12, atol=1e-12)
    # cross-correlation, not convolution: a kernel with a single off-centre tap shifts the input
    ws = np.zeros((1, 1, 3, 3))
    ws[0, 0, 0, 0] = 1.0  # reads (y-1, x-1)
    xs = rng.standard_normal((1, 1, 4, 4))
    got = L.conv2d(xs, ws, np.zeros(1))
    assert got[0, 0, 2, 3] == xs[0, 0, 1, 2]
    assert got[0, 0, 0, 1] == 0.0


def test_group_norm_moments_and_constant_input():
    rng = np.random.default_rng(4)
    x = (3.0 + 2.0 * rng.standard_normal((2, 8, 5, 3))).astype(np.float32)
    y = L.group_norm(x, 4, np.ones(8, np.float32), np.zeros(8, np.float32), 1e-5)
    yg = y.reshape(2, 4, -1).astype(np.float64)
    np.testing.assert_allclose(yg.mean(axis=2), 0.0, atol=1e-6)
    np.testing.assert_allclose(yg.var(axis=2), 1.0, atol=1e-4)
    # affine is per channel
    g = rng.standard_normal(8).astype(np.float32)
    be = rng.standard_normal(8).astype(np.float32)
    y2 = L.group_norm(x, 4, g, be, 1e-5)
    np.testing.assert_allclose(y2, y * g[None, :, None, None] + be[None, :, None, None], rtol=1e-6, atol=1e-6)
    # constant input -> beta
    c = np.full((1, 8, 2, 2), 5.0, np.float32)
    np.testing.assert_allclose(L.group_norm(c, 4, g, be, 1e-5), np.broadcast_to(be[None, :, None, None], c.shape),
                               atol=1e-6)
    # brute-force one group
    xs = x[1, 2:4].astype(np.float64).ravel()
    mu = sum(xs) / len(xs)
    var = sum((v - mu) ** 2 for v in xs) / len(xs)
    ref = (x[1, 2:4].astype(np.float64) - mu) / math.sqrt(var + 1e-5)
    np.testing.assert_allclose(y[1, 2:4], ref, rtol=1e-5, atol=1e-5)


def test_layer_norm_moments():
    rng = np.random.default_rng(5)
    x = (1.0 + rng.standard_normal((3, 7, 16))).astype(np.float32)
    y = L.layer_norm(x, np.ones(16, np.float32), np.zeros(16, np.float32), 1e-5).astype(np.float64)
    np.testing.assert_allclose(y.mean(-1), 0.0, atol=1e-6)
    np.testing.assert_allclose(y.var(-1), 1.0, atol=1e-4)
    c = np.full((2, 16), -2.0, np.float32)
    be = rng.standard_normal(16).astype(np.float32)
    np.testing.assert_allclose(L.layer_norm(c, np.ones(16, np.float32), be, 1e-5), np.broadcast_to(be, c.shape),
                               atol=1e-6)


def _naive_attention(xq, xkv, wq, wk, wv, wo, bo, heads):
    n, sq, _ = xq.shape
    skv = xkv.shape[1]
    c = wq.shape[0]
    d = c // heads
    out = np.zeros((n, sq, wo.shape[0]))
    for b in range(n):
        q = [[sum(xq[b, i, k] * wq[o, k] for k in range(xq.shape[2])) for o in range(c)] for i in range(sq)]
        kk = [[sum(xkv[b, j, k] * wk[o, k] for k in range(xkv.shape[2])) for o in range(c)] for j in range(skv)]
        vv = [[sum(xkv[b, j, k] * wv[o, k] for k in range(xkv.shape[2])) for o in range(c)] for j in range(skv)]
        for i in range(sq):
            cat = [0.0] * c
            for h in range(heads):
                s = [sum(q[i][h * d + e] * kk[j][h * d + e] for e in range(d)) / math.sqrt(d) for j in range(skv)]
                m = max(s)
                p = [math.exp(v - m) for v in s]
                z = sum(p)
                for e in range(d):
                    cat[h * d + e] = sum(p[j] / z * vv[j][h * d + e] for j in range(skv))
            for o in range(wo.shape[0]):
                out[b, i, o] = bo[o] + sum(cat[k] * wo[o, k] for k in range(c))
    return out


def test_attention_matches_naive_softmax():
    rng = np.random.default_rng(6)
    n, sq, skv, cq, ckv, c, heads = 2, 5, 7, 6, 3, 8, 2
    xq = rng.standard_normal((n, sq, cq))
    xkv = rng.standard_normal((n, skv, ckv))
    wq, wk, wv = rng.standard_normal((c, cq)), rng.standard_normal((c, ckv)), rng.standard_normal((c, ckv))
    wo, bo = rng.standard_normal((4, c)), rng.standard_normal(4)
    got = L.attention(xq, xkv, wq, wk, wv, wo, bo, heads)
    np.testing.assert_allclose(got, _naive_attention(xq, xkv, wq, wk, wv, wo, bo, heads), rtol=1e-10, atol=1e-10)


def test_attention_special_cases():
    rng = np.random.default_rng(7)
    c = 4
    eye = np.eye(c)
    xq = rng.standard_normal((1, 3, c))
    # one key -> every query returns that key's value
    xkv = rng.standard_normal((1, 1, c))
    got = L.attention(xq, xkv, eye, eye, eye, eye, np.zeros(c), heads=2)
    np.testing.assert_allclose(got, np.broadcast_to(xkv, got.shape), rtol=1e-12)
    # identical keys -> mean of the values
    keys = np.repeat(rng.standard_normal((1, 1, c)), 5, axis=1)
    wv = rng.standard_normal((c, c))
    v = keys @ wv.T
    vals = rng.standard_normal((1, 5, c))
    # make V differ while K is identical: K from xkv, V from a separate projection of other rows
    xkv2 = np.concatenate([keys, vals], axis=2)  # [1, 5, 2c]
    wk2 = np.concatenate([eye, np.zeros((c, c))], axis=1)
    wv2 = np.concatenate([np.zeros((c, c)), eye], axis=1)
    got = L.attention(xq, xkv2, eye, wk2, wv2, eye, np.zeros(c), heads=1)
    np.testing.assert_allclose(got, np.broadcast_to(vals.mean(axis=1, keepdims=True), got.shape), rtol=1e-12)
    del v
    # zero queries -> uniform weights -> mean of values
    got = L.attention(np.zeros((1, 2, c)), vals, eye, eye, eye, eye, np.zeros(c), heads=2)
    np.testing.assert_allclose(got, np.broadcast_to(vals.mean(axis=1, keepdims=True), got.shape), rtol=1e-12)


def test_activation_closed_forms():
    assert L.gelu(np.array([0.0]))[0] == 0.0
    assert L.silu(np.array([0.0]))[0] == 0.0
    big = np.array([30.0, -30.0])
    np.testing.assert_allclose(L.gelu(big), [30.0, 0.0], atol=1e-12)
    np.testing.assert_allclose(L.silu(big), [30.0, 0.0], atol=1e-10)
    # GELU(x) = x Phi(x): compare with the normal CDF by trapezoid integration of the density
    for xv in (-1.3, 0.4, 2.2):
        grid = np.linspace(-12.0, xv, 200001)
        dens = np.exp(-grid ** 2 / 2) / math.sqrt(2 * math.pi)
        phi = float(np.sum((dens[1:] + dens[:-1]) * 0.5 * np.diff(grid)))
        assert abs(L.gelu(np.array([xv]))[0] - xv * phi) < 1e-8
    # SiLU(x) = x sigmoid(x)
    assert abs(L.silu(np.array([1.5]))[0] - 1.5 / (1 + math.exp(-1.5))) < 1e-12


def test_geglu_halves():
    rng = np.random.default_rng(8)
    x = rng.standard_normal((3, 4))
    w1 = rng.standard_normal((6, 4))
    b1 = rng.standard_normal(6)
    w2 = rng.standard_normal((2, 3))
    b2 = rng.standard_normal(2)
    u = x @ w1.T + b1
    a, g = u[:, :3], u[:, 3:]
    h = np.array([[a[i, j] * 0.5 * g[i, j] * (1 + math.erf(g[i, j] / math.sqrt(2))) for j in range(3)]
                  for i in range(3)])
    np.testing.assert_allclose(L.geglu_ff(x, w1, b1, w2, b2), h @ w2.T + b2, rtol=1e-12)


def test_sinusoid():
    e0 = L.timestep_sinusoid(0, 8)
    np.testing.assert_array_equal(e0, [1, 1, 1, 1, 0, 0, 0, 0])
    t, dim = 37, 10
    e = L.timestep_sinusoid(t, dim)
    for j in range(5):
        f = 10000.0 ** (-j / 5)
        assert abs(e[j] - math.cos(t * f)) < 1e-6
        assert abs(e[5 + j] - math.sin(t * f)) < 1e-6
