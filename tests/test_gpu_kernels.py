"""Kernel parity on the GPU: each single-kernel entry point of the C ABI against the
oracle's layer on the same seeded inputs (the inputs the kernel sees, i.e. after
rounding to the kernel dtype, are what the oracle receives, in fp64).

Tolerances (relative L2 over the whole output):
* fp32 kernels: 1e-5 (fp32 accumulation over K <= 23040 terms, different order);
* bf16 kernels: 8e-3 — fp32 accumulation, but the output itself is rounded to
  bf16 (relative error <= 2^-9 = 2e-3 per element) and attention rounds P to bf16;
  fp32 outputs of bf16 kernels: 2e-3.
Shapes span several tiles with ragged M, N and sequence tails; the last tests run
the SD-XL shapes of the benchmark in the same launch configuration and compare
sampled outputs computed one by one.
"""

import math

import numpy as np
import pytest
import torch

from oracle import layers as L
from paper_2511_06724_amd import dn
from tests.gpu_util import DEV, announce, f32_dev, host, rel_l2, tdtype, to_dev

pytestmark = pytest.mark.gpu

TOL = {dn.DN_FP32: 1e-5, dn.DN_BF16: 8e-3}
DT = [dn.DN_FP32, dn.DN_BF16]


def _rng(seed):
    return np.random.default_rng(seed)


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("M,N,K", [(300, 200, 128), (512, 384, 640), (1000, 1280, 64), (64, 64, 1280),
                                   (2048, 2048, 128), (8192, 512, 256), (300, 1280, 2560), (77, 96, 1920),
                                   (1000, 640, 5120), (129, 256, 704), (2000, 1248, 1280), (8000, 608, 2560),
                                   (8192, 200, 256), (16384, 640, 1280), (2048, 10240, 1280), (16300, 608, 1280)])
def test_linear(dtype, M, N, K):
    """Shapes cover every tile plan: in fp32 the register-staged 64 x 64 / 128 x 128
    tiles; in bf16 the row-major kernels for N % 32 != 0 (N = 200) and the fragment-B
    kernel with 128 x 128 and 128 x 256 tiles, with and without split-K (few tiles and
    long K: 300 x 1280 x 2560, 1000 x 640 x 5120), the five-wave 64 x 160 and 128 x 160
    tiles (2000 x 1248 x 1280, 8000 x 608 x 2560: one tile per CU, ragged last row tile
    and column tile), ragged M and N tails; a tall row-major case (8192 x 200 x 256); the
    four-wave 128 x 160 tiles, two per CU, that linear layers with more 160-column tiles
    than CUs take (16384 x 640 x 1280, 2048 x 10240 x 1280; 16300 x 608 x 1280 with a ragged
    last row tile and column tile). Outputs: bf16 / fp32 without residual, fp32
    with an fp32 residual, and the op's dtype with a residual in that dtype."""
    announce(f"linear dtype={dtype} M={M} N={N} K={K}")
    r = _rng(M + N + K)
    x, xh = to_dev(r.standard_normal((M, K)), dtype)
    w, wh = to_dev(r.standard_normal((N, K)) / math.sqrt(K), dtype)
    b = r.standard_normal(N).astype(np.float32)
    res = r.standard_normal((M, N)).astype(np.float32)
    y = torch.empty((M, N), device=DEV, dtype=tdtype(dtype))
    wp = dn.pack_weight(dtype, w, N, K)
    dn.op_linear(dtype, x, wp, f32_dev(b), y, M, N, K)
    yr = torch.empty((M, N), device=DEV, dtype=torch.float32)
    dn.op_linear(dtype, x, wp, f32_dev(b), yr, M, N, K, resid=f32_dev(res), resid_f32=True, y_f32=True)
    resd, resh = to_dev(res, dtype)
    yd = torch.empty((M, N), device=DEV, dtype=tdtype(dtype))
    dn.op_linear(dtype, x, wp, f32_dev(b), yd, M, N, K, resid=resd)
    torch.cuda.synchronize()
    ref = L.linear(xh, wh, b.astype(np.float64))
    assert rel_l2(host(y), ref) < TOL[dtype]
    assert rel_l2(host(yr), ref + res) < (1e-5 if dtype == dn.DN_FP32 else 2e-3)
    assert rel_l2(host(yd), ref + resh) < TOL[dtype]


def _interleave(w1, n):
    """GEGLU packed layout: 32-row blocks alternate value rows and gate rows."""
    out = np.empty_like(w1)
    for j in range(n // 32):
        out[64 * j:64 * j + 32] = w1[32 * j:32 * j + 32]
        out[64 * j + 32:64 * j + 64] = w1[n + 32 * j:n + 32 * j + 32]
    return out


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("M,N,K", [(300, 96, 128), (512, 1280, 320), (2048, 5120, 1280), (2000, 5120, 1280)])
def test_linear_geglu(dtype, M, N, K):
    """Ragged small shapes and SD-XL's FF-in at full size, whole output: in bf16 its 640
    128 x 256 tiles leave a quarter round, whose column bands run as 64-row tiles (with a
    ragged last row tile of both kinds at 2000 rows)."""
    announce(f"geglu dtype={dtype} M={M} N={N} K={K}")
    r = _rng(7 * M + N)
    x, xh = to_dev(r.standard_normal((M, K)), dtype)
    w1 = (r.standard_normal((2 * N, K)) / math.sqrt(K)).astype(np.float32)
    b1 = r.standard_normal(2 * N).astype(np.float32)
    wp = dn.pack_weight(dtype, to_dev(_interleave(w1, N), dtype)[0], 2 * N, K)
    w1h = host(to_dev(w1, dtype)[0])
    bp = _interleave(b1[:, None], N)[:, 0].copy()
    y = torch.empty((M, N), device=DEV, dtype=tdtype(dtype))
    dn.op_linear(dtype, x, wp, f32_dev(bp), y, M, N, K, geglu=True)
    torch.cuda.synchronize()
    u = L.linear(xh, w1h, b1.astype(np.float64))
    ref = u[:, :N] * L.gelu(u[:, N:])
    assert rel_l2(host(y), ref) < TOL[dtype]


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("n,H,W,Cin,Cout,up,stride", [
    (2, 9, 7, 64, 96, 0, 1), (2, 9, 7, 64, 96, 0, 2), (1, 5, 6, 128, 64, 1, 1), (2, 16, 16, 128, 320, 0, 1),
    (2, 128, 128, 320, 320, 0, 1), (2, 128, 128, 640, 320, 0, 1), (1, 64, 64, 640, 640, 1, 1),
    (2, 100, 100, 320, 320, 0, 1)])
def test_conv3x3(dtype, n, H, W, Cin, Cout, up, stride):
    """Small shapes with ragged tiles, and the SD-XL convolutions at full size, whole
    output against the oracle: the 128x128-level ResBlock convolutions (32768 rows, 320
    channels from 320 and from a 640-channel input) and the nearest-x2 upsampling
    convolution into that level (640 channels): in bf16 these run on the four-wave
    160-column tiles, two workgroups per CU; 2 x 100 x 100 has a ragged last row tile."""
    announce(f"conv dtype={dtype} n={n} H={H} W={W} Cin={Cin} Cout={Cout} up={up} stride={stride}")
    r = _rng(n * H * W + Cin + Cout + up + stride)
    x, xh = to_dev(r.standard_normal((n, H, W, Cin)), dtype)
    wt = (r.standard_normal((Cout, Cin, 3, 3)) / math.sqrt(9 * Cin)).astype(np.float32)
    wd, _ = to_dev(wt.transpose(0, 2, 3, 1), dtype)
    wh = host(to_dev(wt, dtype)[0])
    b = r.standard_normal(Cout).astype(np.float32)
    temb = r.standard_normal((n, Cout)).astype(np.float32)
    xin = xh.transpose(0, 3, 1, 2)
    if up:
        xin = L.upsample_nearest2x(xin)
    ref = L.conv2d(xin, wh, b.astype(np.float64), stride=stride)          # NCHW
    ho, wo = ref.shape[2], ref.shape[3]
    res = r.standard_normal((n, ho, wo, Cout)).astype(np.float32)
    resd, resh = to_dev(res, dtype)
    y = torch.empty((n, ho, wo, Cout), device=DEV, dtype=tdtype(dtype))
    wp = dn.pack_weight(dtype, wd, Cout, 9 * Cin)
    dn.op_conv3x3(dtype, x, n, H, W, Cin, wp, f32_dev(b), y, Cout, up=up, stride=stride, temb=f32_dev(temb),
                  resid=resd)
    torch.cuda.synchronize()
    full = ref.transpose(0, 2, 3, 1) + temb[:, None, None, :] + resh
    assert rel_l2(host(y), full) < TOL[dtype]


def _pad_heads(a, heads, d, dp):
    """[.., heads*d] -> [.., heads*dp] with zeros in each head's padding columns."""
    out = np.zeros(a.shape[:-1] + (heads * dp,), dtype=a.dtype)
    for h in range(heads):
        out[..., h * dp:h * dp + d] = a[..., h * d:(h + 1) * d]
    return out


def _vt_layout(v, heads, dp, ld):
    """[B, S, heads*dp] -> V^T [B, heads, dp, ld] (zeros past S)."""
    B, S, _ = v.shape
    out = np.zeros((B, heads, dp, ld), dtype=v.dtype)
    out[..., :S] = v.reshape(B, S, heads, dp).transpose(0, 2, 3, 1)
    return out


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("B,heads,Sq,Skv,d", [(2, 3, 200, 77, 64), (1, 2, 256, 300, 64), (2, 2, 130, 96, 40),
                                              (2, 4, 256, 256, 16), (1, 1, 5, 1, 64), (2, 20, 1024, 1024, 64),
                                              (1, 3, 2100, 333, 64), (2, 1, 70, 257, 64)])
def test_attention(dtype, B, heads, Sq, Skv, d):
    announce(f"attention dtype={dtype} B={B} heads={heads} Sq={Sq} Skv={Skv} d={d}")
    r = _rng(B * heads + Sq + Skv + d)
    dp = 32 if d <= 32 else 64
    ld = (Skv + 63) // 64 * 64
    q = r.standard_normal((B, Sq, heads * d)).astype(np.float32)
    k = r.standard_normal((B, Skv, heads * d)).astype(np.float32)
    v = r.standard_normal((B, Skv, heads * d)).astype(np.float32)
    qd, qh = to_dev(_pad_heads(q, heads, d, dp), dtype)
    kd, kh = to_dev(_pad_heads(k, heads, d, dp), dtype)
    vtd, vth = to_dev(_vt_layout(_pad_heads(v, heads, d, dp), heads, dp, ld), dtype)
    o = torch.zeros((B, Sq, heads * dp), device=DEV, dtype=tdtype(dtype))
    P = heads * dp
    dn.op_attention(dtype, qd, P, kd, P, vtd, ld, o, P, B, heads, Sq, Skv, dp, 1.0 / math.sqrt(d))
    torch.cuda.synchronize()
    # oracle: multi-head attention with identity projections on the unpadded heads
    strip = lambda a: np.concatenate([a[..., h * dp:h * dp + d] for h in range(heads)], axis=-1)
    vh = vth[..., :Skv].transpose(0, 3, 1, 2).reshape(B, Skv, P)            # back to [B, Skv, heads*dp]
    c = heads * d
    eye, zero = np.eye(c), np.zeros((c, c))
    xkv = np.concatenate([strip(kh), strip(vh)], axis=-1)          # K and V from one [.., 2c] input
    ref = L.attention(strip(qh), xkv, eye, np.hstack([eye, zero]), np.hstack([zero, eye]), eye, np.zeros(c), heads)
    got = host(o)
    assert rel_l2(strip(got), ref) < TOL[dtype]
    # padding columns of o are zero (v's padding is zero)
    if dp != d:
        assert np.all(got[..., d:dp] == 0)


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("M,seq,heads,dp,K", [(300, 150, 3, 64, 128), (512, 256, 4, 32, 64), (8192, 4096, 10, 64, 640),
                                              (2048, 1024, 20, 64, 1280)])
def test_linear_vt(dtype, M, seq, heads, dp, K):
    """Attention input projection: Q, K columns to y, V columns transposed per head
    into vt[sample][head][d][token] (the last two shapes are the SD-XL QKV projections
    at the 64x64 and 32x32 levels, on the fragment-B kernel)."""
    announce(f"linear_vt dtype={dtype} M={M} seq={seq} heads={heads} dp={dp} K={K}")
    P = heads * dp
    N = 3 * P
    r = _rng(M + K + dp)
    x, xh = to_dev(r.standard_normal((M, K)), dtype)
    w, wh = to_dev(r.standard_normal((N, K)) / math.sqrt(K), dtype)
    b = r.standard_normal(N).astype(np.float32)
    ld = (seq + 63) // 64 * 64
    y = torch.empty((M, 2 * P), device=DEV, dtype=tdtype(dtype))
    vt = torch.zeros((M // seq, heads, dp, ld), device=DEV, dtype=tdtype(dtype))
    dn.op_linear_vt(dtype, x, dn.pack_weight(dtype, w, N, K), f32_dev(b), y, M, N, K, 2 * P, vt, heads, dp, seq, ld)
    torch.cuda.synchronize()
    ref = L.linear(xh, wh, b.astype(np.float64))
    assert rel_l2(host(y), ref[:, :2 * P]) < TOL[dtype]
    ref_vt = ref[:, 2 * P:].reshape(M // seq, seq, heads, dp).transpose(0, 2, 3, 1)
    got = host(vt)
    assert rel_l2(got[..., :seq], ref_vt) < TOL[dtype]
    assert np.all(got[..., seq:] == 0)


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("n,HW,C,G,silu", [(2, 300, 320, 32, 1), (2, 64, 64, 32, 0), (1, 1000, 1920, 32, 1),
                                            (2, 1024, 1280, 32, 1), (2, 4096, 640, 32, 0), (1, 16384, 320, 32, 1),
                                            (2, 200, 96, 32, 1), (2, 1024, 2560, 32, 1)])
def test_groupnorm(dtype, n, HW, C, G, silu):
    """Includes the SD-XL shapes (40, 20 and 10 channels per group at 32x32, 64x64 and
    128x128, and the 2560-channel concatenation at 32x32), an odd channel count per group
    (96 / 32 = 3), and both apply mappings: one channel vector per thread (at most 256
    16-byte vectors per pixel) and (pixel, vector) pairs (fp32 from 1280 channels, bf16 at
    2560)."""
    announce(f"groupnorm dtype={dtype} n={n} HW={HW} C={C} silu={silu}")
    r = _rng(n + HW + C)
    x, xh = to_dev(0.5 + 2.0 * r.standard_normal((n, HW, C)), dtype)
    g = (1 + 0.1 * r.standard_normal(C)).astype(np.float32)
    b = (0.1 * r.standard_normal(C)).astype(np.float32)
    y = torch.empty((n, HW, C), device=DEV, dtype=tdtype(dtype))
    dn.op_groupnorm(dtype, x, y, n, HW, C, G, f32_dev(g), f32_dev(b), 1e-5, silu)
    torch.cuda.synchronize()
    ref = L.group_norm(xh.transpose(0, 2, 1)[..., None], G, g.astype(np.float64), b.astype(np.float64), 1e-5)
    ref = ref[..., 0].transpose(0, 2, 1)
    if silu:
        ref = L.silu(ref)
    assert rel_l2(host(y), ref) < (2e-6 if dtype == dn.DN_FP32 else TOL[dtype])


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("M,C", [(300, 1280), (77, 64), (2048, 640)])
def test_layernorm(dtype, M, C):
    announce(f"layernorm dtype={dtype} M={M} C={C}")
    r = _rng(M + C)
    x = (1.0 + 3.0 * r.standard_normal((M, C))).astype(np.float32)
    g = (1 + 0.1 * r.standard_normal(C)).astype(np.float32)
    b = (0.1 * r.standard_normal(C)).astype(np.float32)
    y = torch.empty((M, C), device=DEV, dtype=tdtype(dtype))
    dn.op_layernorm(dtype, f32_dev(x), y, M, C, f32_dev(g), f32_dev(b), 1e-5)
    torch.cuda.synchronize()
    ref = L.layer_norm(x.astype(np.float64), g.astype(np.float64), b.astype(np.float64), 1e-5)
    assert rel_l2(host(y), ref) < (2e-6 if dtype == dn.DN_FP32 else TOL[dtype])


@pytest.mark.parametrize("dtype", DT)
@pytest.mark.parametrize("M,C,nsplit,bias,resid", [(2048, 1280, 3, True, True), (2048, 1280, 2, True, False),
                                                   (8192, 640, 4, True, True), (301, 320, 1, False, True),
                                                   (77, 2048, 8, True, True)])
def test_layernorm_slabs(dtype, M, C, nsplit, bias, resid):
    """The LayerNorm that completes a split-K residual update: x <- (x if resid) + bias +
    sum of the fp32 slabs, written back, then normalised. 2048 x 1280 with three slabs is
    the FF-out of a 32x32 SD-XL block feeding the next block's first LayerNorm; two
    slabs without residual is proj_in; the widest row (C = 2048) with eight slabs."""
    announce(f"layernorm slabs dtype={dtype} M={M} C={C} nsplit={nsplit} bias={bias} resid={resid}")
    r = _rng(M + C + nsplit)
    x = (0.5 + 2.0 * r.standard_normal((M, C))).astype(np.float32)
    slabs = r.standard_normal((nsplit, M, C)).astype(np.float32)
    bv = r.standard_normal(C).astype(np.float32)
    g = (1 + 0.1 * r.standard_normal(C)).astype(np.float32)
    b = (0.1 * r.standard_normal(C)).astype(np.float32)
    xd = f32_dev(x)
    y = torch.empty((M, C), device=DEV, dtype=tdtype(dtype))
    dn.op_layernorm_slabs(dtype, xd, y, M, C, f32_dev(g), f32_dev(b), 1e-5, f32_dev(slabs), nsplit,
                          f32_dev(bv) if bias else None, resid)
    torch.cuda.synchronize()
    full = (x.astype(np.float64) if resid else 0.0) + slabs.astype(np.float64).sum(axis=0)
    if bias:
        full = full + bv
    # the rebuilt residual row: fp32 sums of at most 10 terms of size ~3
    assert rel_l2(host(xd), full) < 1e-6
    ref = L.layer_norm(full, g.astype(np.float64), b.astype(np.float64), 1e-5)
    assert rel_l2(host(y), ref) < (2e-6 if dtype == dn.DN_FP32 else TOL[dtype])


def test_probe_mfma_rate():
    """The matrix-core probe the bench reports beside the published peak: a rate and a
    clock in the range the device can reach (at most the published 2.5 PFLOP/s at 2.4 GHz),
    and an argument error for an iteration count out of range."""
    announce("probe mfma rate")
    tf, ghz = dn.probe_mfma_rate(2000)
    assert 500.0 < tf <= 2600.0
    assert 0.5 < ghz <= 2.6
    # 32x32x16 MFMAs at one per 32 cycles per SIMD: the rate follows from the clock
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert tf <= cus * 4 * 32768 / 32 * ghz * 1e9 / 1e12 * 1.05
    with pytest.raises(dn.DnError):
        dn.probe_mfma_rate(0)


def test_layernorm_slabs_argument_errors():
    x = torch.zeros((4, 64), device=DEV)
    y = torch.zeros((4, 64), device=DEV)
    g = torch.ones(64, device=DEV)
    for ns in (0, 9):
        with pytest.raises(dn.DnError):
            dn.op_layernorm_slabs(dn.DN_FP32, x, y, 4, 64, g, g, 1e-5, x, ns)
    with pytest.raises(dn.DnError):
        dn.op_layernorm_slabs(dn.DN_FP32, x, y, 4, 64, g, g, 1e-5, None, 1)


# ----------------------------------------------------------------------------- SD-XL shapes, sampled

def _sample_idx(r, shape, count):
    return tuple(r.integers(0, s, size=count) for s in shape)


def test_sdxl_ff_in_geglu_sampled():
    """FF-in of a 32x32 SD-XL transformer block: 2048 x (2 x 5120) x 1280, bf16, GEGLU epilogue."""
    announce("sdxl ff-in geglu 2048x10240x1280")
    M, N, K = 2048, 5120, 1280
    g = torch.Generator(device=DEV).manual_seed(3)
    x = torch.randn((M, K), device=DEV, generator=g).to(torch.bfloat16)
    w = (torch.randn((2 * N, K), device=DEV, generator=g) / math.sqrt(K)).to(torch.bfloat16)
    b = torch.randn(2 * N, device=DEV, generator=g)
    y = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    dn.op_linear(dn.DN_BF16, x, dn.pack_weight(dn.DN_BF16, w, 2 * N, K), b, y, M, N, K, geglu=True)
    torch.cuda.synchronize()
    r = _rng(5)
    ms, ns = _sample_idx(r, (M, N), 512)
    xh, wh, bh, yh = host(x), host(w), host(b), host(y)
    for m, n in zip(ms, ns):
        blk, c = n // 32, n % 32
        rv, rg = 64 * blk + c, 64 * blk + 32 + c
        a = float(xh[m] @ wh[rv] + bh[rv])
        gg = float(xh[m] @ wh[rg] + bh[rg])
        ref = a * 0.5 * gg * (1 + math.erf(gg / math.sqrt(2)))
        assert abs(yh[m, n] - ref) <= 1e-2 * max(1.0, abs(ref)), (m, n, yh[m, n], ref)


def test_sdxl_conv_top_level_sampled():
    """3x3 conv at the SD-XL top level: 2 x 128 x 128 x 320 -> 320 (M = 32768, K = 2880), bf16."""
    announce("sdxl conv 32768x320x2880")
    n, H, W, C = 2, 128, 128, 320
    g = torch.Generator(device=DEV).manual_seed(4)
    x = torch.randn((n, H, W, C), device=DEV, generator=g).to(torch.bfloat16)
    w = (torch.randn((C, 3, 3, C), device=DEV, generator=g) / math.sqrt(9 * C)).to(torch.bfloat16)
    b = torch.randn(C, device=DEV, generator=g)
    y = torch.empty((n, H, W, C), device=DEV, dtype=torch.bfloat16)
    dn.op_conv3x3(dn.DN_BF16, x, n, H, W, C, dn.pack_weight(dn.DN_BF16, w, C, 9 * C), b, y, C)
    torch.cuda.synchronize()
    r = _rng(6)
    xh, wh, bh, yh = host(x), host(w), host(b), host(y)
    for s, yy, xx, co in zip(*_sample_idx(r, (n, H, W, C), 256)):
        acc = bh[co]
        for ky in range(3):
            for kx in range(3):
                iy, ix = yy + ky - 1, xx + kx - 1
                if 0 <= iy < H and 0 <= ix < W:
                    acc += float(xh[s, iy, ix] @ wh[co, ky, kx])
        assert abs(yh[s, yy, xx, co] - acc) <= 1e-2 * max(1.0, abs(acc)), (s, yy, xx, co)


def test_sdxl_self_attention_sampled():
    """Self-attention at the SD-XL 64x64 level: 2 samples x 10 heads, S = 4096, d = 64, bf16."""
    announce("sdxl attention S=4096 10x64")
    B, heads, S, d = 2, 10, 4096, 64
    P = heads * d
    g = torch.Generator(device=DEV).manual_seed(5)
    qk = torch.randn((B, S, 2 * P), device=DEV, generator=g).to(torch.bfloat16)
    vt = torch.randn((B, heads, d, S), device=DEV, generator=g).to(torch.bfloat16)
    o = torch.empty((B, S, P), device=DEV, dtype=torch.bfloat16)
    q, k = qk[..., :P], qk[..., P:]
    dn.lib.dn_op_attention(dn.DN_BF16, q.data_ptr(), 2 * P, k.data_ptr(), 2 * P, vt.data_ptr(), S, o.data_ptr(),
                           P, B, heads, S, S, 64, 1.0 / 8.0, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    r = _rng(7)
    qh = host(qk)
    vh = host(vt)
    oh = host(o)
    for b, h in [(0, 0), (1, 9), (0, 5)]:
        rows = r.integers(0, S, size=16)
        K_ = qh[b, :, P + h * d:P + (h + 1) * d]
        V_ = vh[b, h].T                                   # [S, d]
        for i in rows:
            s = K_ @ qh[b, i, h * d:(h + 1) * d] / 8.0
            p = np.exp(s - s.max())
            ref = (p / p.sum()) @ V_
            assert rel_l2(oh[b, i, h * d:(h + 1) * d], ref) < 1e-2, (b, h, i)


@pytest.mark.parametrize("M,N,K", [(2048, 1280, 5120), (2048, 1280, 1280), (2048, 3840, 1280), (154, 2560, 2048)])
def test_sdxl_linear_shapes_sampled_and_deterministic(M, N, K):
    """The M = 2048 projections of the SD-XL 32x32 blocks (FF-out, attention out, QKV)
    and the context K/V projection, in the launch configuration the denoiser uses
    (split-K where the planner picks it): sampled outputs against fp64 dot products,
    and two launches bitwise equal (the split-K reduction order is fixed)."""
    announce(f"sdxl linear {M}x{N}x{K}")
    g = torch.Generator(device=DEV).manual_seed(M + N + K)
    x = torch.randn((M, K), device=DEV, generator=g).to(torch.bfloat16)
    w = (torch.randn((N, K), device=DEV, generator=g) / math.sqrt(K)).to(torch.bfloat16)
    b = torch.randn(N, device=DEV, generator=g)
    res = torch.randn((M, N), device=DEV, generator=g)
    y1 = torch.empty((M, N), device=DEV)
    y2 = torch.empty((M, N), device=DEV)
    wp = dn.pack_weight(dn.DN_BF16, w, N, K)
    dn.op_linear(dn.DN_BF16, x, wp, b, y1, M, N, K, resid=res, resid_f32=True, y_f32=True)
    dn.op_linear(dn.DN_BF16, x, wp, b, y2, M, N, K, resid=res, resid_f32=True, y_f32=True)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    r = _rng(M + K)
    xh, wh, bh, rh, yh = host(x), host(w), host(b), host(res), host(y1)
    for m, n in zip(*_sample_idx(r, (M, N), 400)):
        ref = float(xh[m] @ wh[n] + bh[n] + rh[m, n])
        assert abs(yh[m, n] - ref) <= 2e-3 * max(1.0, abs(ref)), (m, n, yh[m, n], ref)


# ----------------------------------------------------------------------------- fp8 (E4M3) quantized variant

def _fp8_offsets(N, K):
    """Byte offset of (n, k) in the fp8 fragment order (pack_fp8)."""
    n = np.arange(N)[:, None]
    k = np.arange(K)[None, :]
    return ((n // 32) * (K // 64) + k // 64) * 2048 + ((n % 32) + 32 * ((k % 64) // 32)) * 32 + (k % 32)


def _fp8_values(codes_u8):
    return torch.from_numpy(np.ascontiguousarray(codes_u8)).view(torch.float8_e4m3fn).float().numpy()


def _to_fp8_dev(x):
    """fp32 values -> (device E4M3 codes, the values they hold)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).to(DEV), t.float().numpy().astype(np.float64)


@pytest.mark.parametrize("N,K", [(64, 128), (1280, 5120), (640, 256)])
def test_fp8_pack_matches_oracle_quantization(N, K):
    """dn_pack_weight(DN_FP8): every row scale bitwise the oracle's, every code the
    oracle's quantised value."""
    from oracle import quant as Q
    announce(f"fp8 pack N={N} K={K}")
    r = _rng(N + K)
    w = (r.standard_normal((N, K)) * r.uniform(0.01, 2.0, (N, 1))).astype(np.float32)
    w[3] = 0.0
    packed = dn.pack_weight(dn.DN_FP8, torch.from_numpy(w).to(DEV), N, K).cpu().numpy()
    scales = packed[N * K:].view(np.float32)
    deq, s = Q.quantize_rows(w)
    assert np.array_equal(scales.view(np.uint32), s.view(np.uint32))
    vals = _fp8_values(packed[:N * K][_fp8_offsets(N, K)])
    assert np.array_equal((vals * s[:, None]).astype(np.float32), deq)


@pytest.mark.parametrize("M,N,K,geglu,resid", [(300, 256, 256, False, False), (2048, 1280, 5120, False, True),
                                               (1000, 640, 1280, False, True), (300, 256, 128, True, False),
                                               (2048, 5120, 1280, True, False), (2000, 5120, 1280, True, False)])
def test_fp8_linear(M, N, K, geglu, resid):
    """The fp8 GEMM against the oracle on the quantised operands: fp32 output within
    1e-5 (products exact, fp32 sums in another order); the GEGLU output in E4M3 against
    the oracle's E4M3 rounding of the exact result (at least 99 % identical codes, the
    rest one quantum off at rounding boundaries)."""
    from oracle import quant as Q
    announce(f"fp8 linear M={M} N={N} K={K} geglu={geglu} resid={resid}")
    r = _rng(3 * M + N + K)
    Nw = 2 * N if geglu else N
    x8, xh = _to_fp8_dev(r.standard_normal((M, K)))
    w = (r.standard_normal((Nw, K)) / math.sqrt(K)).astype(np.float32)
    b = r.standard_normal(Nw).astype(np.float32)
    wi = _interleave(w, N) if geglu else w
    bi = _interleave(b[:, None], N)[:, 0].copy() if geglu else b
    wp = dn.pack_weight(dn.DN_FP8, torch.from_numpy(wi).to(DEV), Nw, K)
    wq = Q.quantize_rows(w)[0].astype(np.float64)      # the same quantisation row by row
    u = xh @ wq.T + b.astype(np.float64)
    if geglu:
        y = torch.empty((M, N), device=DEV, dtype=torch.uint8)
        dn.op_linear(dn.DN_FP8, x8, wp, f32_dev(bi), y, M, N, K, geglu=True)
        torch.cuda.synchronize()
        ref = u[:, :N] * L.gelu(u[:, N:])
        got = _fp8_values(y.cpu().numpy())
        want = Q.fp8_round(ref)
        assert rel_l2(got, ref) < 4e-2
        assert np.mean(got == want) >= 0.99
        return
    res = r.standard_normal((M, N)).astype(np.float32) if resid else None
    y = torch.empty((M, N), device=DEV)
    dn.op_linear(dn.DN_FP8, x8, wp, f32_dev(b), y, M, N, K, resid=f32_dev(res) if resid else None, resid_f32=True,
                 y_f32=True)
    yb = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    dn.op_linear(dn.DN_FP8, x8, wp, f32_dev(b), yb, M, N, K)
    torch.cuda.synchronize()
    ref = u + (res if resid else 0.0)
    assert rel_l2(host(y), ref) < 1e-5
    assert rel_l2(host(yb), u) < 8e-3


def test_fp8_layernorm():
    """LayerNorm with E4M3 output: codes identical to the oracle's rounding of the exact
    normalised values except at rounding boundaries."""
    from oracle import quant as Q
    announce("fp8 layernorm 2048x1280")
    M, C = 2048, 1280
    r = _rng(99)
    x = (1.0 + 3.0 * r.standard_normal((M, C))).astype(np.float32)
    g = (1 + 0.1 * r.standard_normal(C)).astype(np.float32)
    b = (0.1 * r.standard_normal(C)).astype(np.float32)
    y = torch.empty((M, C), device=DEV, dtype=torch.uint8)
    dn.op_layernorm(dn.DN_FP8, f32_dev(x), y, M, C, f32_dev(g), f32_dev(b), 1e-5)
    torch.cuda.synchronize()
    ref = L.layer_norm(x.astype(np.float64), g.astype(np.float64), b.astype(np.float64), 1e-5)
    got = _fp8_values(y.cpu().numpy())
    assert np.mean(got == Q.fp8_round(ref)) >= 0.999
    assert rel_l2(got, ref) < 4e-2
