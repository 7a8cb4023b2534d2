// Latent decoder (the VAE Decoder of Table 3): the final denoised latent -> the RGB
// image, once per image after the loop. Same kernels as the UNet (implicit-GEMM
// convolutions with the nearest-x2 upsample folded into the loader, GroupNorm + SiLU,
// linear layers) plus the middle block's single-head self-attention over all positions,
// which at SD-XL size is one 512-wide head over 16384 positions: scores by a GEMM
// (fp32), a row softmax kernel, then P V by a GEMM.
#include <algorithm>
#include <cmath>

#include "model.h"

namespace dn {

namespace {

constexpr int kVaeCinPad = 64;

// ---------------------------------------------------------------- kernels

// Decoder input: x[b][p][c] = sum_k pq_w[c][k] z[b][k][p] / scale + pq_b[c] for
// c < latent_c (the 1x1 post-quantisation conv), zero in the padding channels.
template <typename T>
__global__ void vae_input_kernel(const float* z, const float* pq_w, const float* pq_b, float inv_scale, T* x, int B,
                                 int C, int HW) {
  const long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (i >= (long long)B * HW) return;
  const int b = (int)(i / HW), p = (int)(i - (long long)b * HW);
  float zin[kVaeCinPad];
  for (int k = 0; k < C; ++k) zin[k] = z[((long long)b * C + k) * HW + p] * inv_scale;
  T* row = x + i * kVaeCinPad;
  for (int c = 0; c < kVaeCinPad; ++c) {
    float v = 0.f;
    if (c < C) {
      v = pq_b[c];
      for (int k = 0; k < C; ++k) v += pq_w[c * C + k] * zin[k];
    }
    row[c] = from_f32<T>(v);
  }
}

// NHWC fp32 [B][HW][C] -> NCHW fp32 [B][C][HW].
__global__ void vae_output_kernel(const float* src, float* img, int B, int C, int HW) {
  const long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (i >= (long long)B * C * HW) return;
  const int p = (int)(i % HW);
  const long long bc = i / HW;
  const int c = (int)(bc % C), b = (int)(bc / C);
  img[i] = src[((long long)b * HW + p) * C + c];
}

__device__ __forceinline__ void ms_merge(float& m, float& l, float m2, float l2) {
  const float mn = fmaxf(m, m2);
  l = (m == -INFINITY ? 0.f : l * exp2f(m - mn)) + (m2 == -INFINITY ? 0.f : l2 * exp2f(m2 - mn));
  m = mn;
}

// Row softmax of scores S [rows][n] (fp32) with a scale: P = exp(s*scale - max) / sum.
// One workgroup per row; a running (maximum, sum) per thread in log2 units, merged over
// the wave and the workgroup in a fixed order, then a second pass writes P.
template <typename T>
__global__ __launch_bounds__(256) void softmax_rows_kernel(const float* S, T* P, int n, float scale_log2) {
  __shared__ float sm[4], sl[4];
  const long long row = blockIdx.x;
  const float* s = S + row * n;
  float m = -INFINITY, l = 0.f;
  for (int j = threadIdx.x; j < n; j += 256) {
    const float v = s[j] * scale_log2;
    if (v > m) {
      l = (m == -INFINITY ? 0.f : l * exp2f(m - v)) + 1.f;
      m = v;
    } else {
      l += exp2f(v - m);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(l, o, 64);
    ms_merge(m, l, m2, l2);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sm[w] = m;
    sl[w] = l;
  }
  __syncthreads();
  m = sm[0];
  l = sl[0];
  for (int k = 1; k < 4; ++k) ms_merge(m, l, sm[k], sl[k]);
  const float inv = 1.f / l;
  T* p = P + row * n;
  for (int j = threadIdx.x; j < n; j += 256) p[j] = from_f32<T>(exp2f(s[j] * scale_log2 - m) * inv);
}

int blocks(long long n) { return static_cast<int>((n + 255) / 256); }

// ---------------------------------------------------------------- model

struct VConv {
  void* w = nullptr;  // [cout][taps * cinp] packed
  float* b = nullptr;
  int cin = 0, cinp = 0, cout = 0, taps = 9;
};
struct VRes {
  float *g1 = nullptr, *b1 = nullptr, *g2 = nullptr, *b2 = nullptr;
  VConv c1, c2, skip;
  bool has_skip = false;
  int cin = 0, cout = 0;
};

// One up level: its ResBlocks, then (level > 0) the upsample conv.
struct VLevel {
  std::vector<VRes> res;
  bool up = false;
  VConv up_conv;
  int c = 0;
};

}  // namespace

struct Vae {
  dn_vae_config cfg{};
  bool bf = true;
  size_t esz = 2;
  int cus = 256;
  void* packed = nullptr;
  float* params = nullptr;
  float *pq_w = nullptr, *pq_b = nullptr;
  VConv conv_in, conv_out;
  VRes mid0, mid1;
  float *attn_g = nullptr, *attn_b = nullptr;
  VConv qkv, proj;  // 1x1 layers: qkv [3C][C] (q, k, v rows), proj [C][C]
  std::vector<VLevel> levels;  // from the coarsest level (L - 1) to level 0
  float *out_g = nullptr, *out_b = nullptr;
  // workspace
  void* arena = nullptr;
  void *xin = nullptr, *X = nullptr, *Y = nullptr, *G = nullptr, *Hh = nullptr, *Sk = nullptr;
  void *qkvbuf = nullptr, *vt = nullptr, *kpack = nullptr, *vpack = nullptr, *P = nullptr, *o = nullptr;
  float *S = nullptr, *out = nullptr, *gn_partial = nullptr, *gn_stats = nullptr, *split = nullptr;
  size_t split_floats = 0;
  void* zero = nullptr;
};

namespace {

std::vector<TensorSpec> vae_table(const dn_vae_config& c) {
  std::vector<TensorSpec> t;
  int64_t off = 0;
  auto add = [&](const std::string& name, std::vector<int64_t> shape, int kind, int fan) {
    TensorSpec s;
    s.name = name;
    s.shape = shape;
    s.numel = 1;
    for (auto d : shape) s.numel *= d;
    s.offset = off;
    s.kind = kind;
    s.fan_in = fan;
    off += s.numel;
    t.push_back(s);
  };
  auto wb = [&](const std::string& n, std::vector<int64_t> shape) {
    int64_t fan = 1;
    for (size_t i = 1; i < shape.size(); ++i) fan *= shape[i];
    add(n + ".w", shape, 0, (int)fan);
    add(n + ".b", {shape[0]}, 1, (int)fan);
  };
  auto norm = [&](const std::string& n, int64_t ch) {
    add(n + ".g", {ch}, 2, 0);
    add(n + ".b", {ch}, 3, 0);
  };
  auto res = [&](const std::string& p, int64_t cin, int64_t cout) {
    norm(p + ".gn1", cin);
    wb(p + ".conv1", {cout, cin, 3, 3});
    norm(p + ".gn2", cout);
    wb(p + ".conv2", {cout, cout, 3, 3});
    if (cin != cout) wb(p + ".skip", {cout, cin, 1, 1});
  };
  const int L = c.n_levels;
  const int64_t top = c.channels[L - 1];
  wb("post_quant", {c.latent_c, c.latent_c, 1, 1});
  wb("conv_in", {top, c.latent_c, 3, 3});
  res("mid.res0", top, top);
  norm("mid.attn.gn", top);
  for (const char* p : {"q", "k", "v", "o"}) wb(std::string("mid.attn.") + p, {top, top});
  res("mid.res1", top, top);
  int64_t prev = top;
  for (int l = L - 1; l >= 0; --l) {
    for (int j = 0; j <= c.layers_per_block; ++j) {
      res("up" + std::to_string(l) + "." + std::to_string(j), prev, c.channels[l]);
      prev = c.channels[l];
    }
    if (l > 0) wb("up" + std::to_string(l) + ".up", {c.channels[l], c.channels[l], 3, 3});
  }
  norm("out.gn", c.channels[0]);
  wb("conv_out", {c.out_c, c.channels[0], 3, 3});
  return t;
}

struct VPacker {
  Vae* v;
  const float* blob;
  std::map<std::string, const TensorSpec*> idx;
  char* pk = nullptr;
  size_t pk_bytes = 0;
  float* pr = nullptr;
  size_t pr_floats = 0;
  bool dry = true;
  hipStream_t s = nullptr;

  const TensorSpec& t(const std::string& n) {
    auto it = idx.find(n);
    DN_CHECK(it != idx.end(), "internal: missing VAE tensor " + n);
    return *it->second;
  }
  void* alloc_packed(size_t elems) {
    const size_t bytes = (elems * v->esz + 255) / 256 * 256;
    void* p = dry ? nullptr : pk + pk_bytes;
    pk_bytes += bytes;
    return p;
  }
  float* alloc_params(size_t n) {
    float* p = dry ? nullptr : pr + pr_floats;
    pr_floats += (n + 63) / 64 * 64;
    return p;
  }
  float* param(const std::string& n) {
    const TensorSpec& ts = t(n);
    float* d = alloc_params(ts.numel);
    if (!dry) DN_HIP(hipMemcpyAsync(d, blob + ts.offset, ts.numel * 4, hipMemcpyDeviceToDevice, s));
    return d;
  }
  // rows x cols packed matrix from source rows [src_row0, src_row0 + rows) of tensor n
  void mat(void* dst, int rows, int cols, const TensorSpec& src, int col_mode, int src_cols, int cin, int cinp,
           long long src_row0 = 0) {
    if (dry) return;
    PackParams p;
    p.dst = dst;
    p.rows = rows;
    p.cols = cols;
    p.ld_dst = cols;
    p.src = blob + src.offset + src_row0 * src_cols;
    p.row_mode = 0;
    p.col_mode = col_mode;
    p.src_rows = rows;
    p.src_cols = src_cols;
    p.Cin = cin;
    p.Cinp = cinp;
    p.frag = v->bf && gemm_frag_layout(rows, cols);
    if (v->bf)
      pack<bf16>(p, s);
    else
      pack<float>(p, s);
  }
  VConv conv3(const std::string& n, int cin, int cout) {
    VConv c;
    c.cin = cin;
    c.cinp = (cin + kVaeCinPad - 1) / kVaeCinPad * kVaeCinPad;
    c.cout = cout;
    c.taps = 9;
    c.w = alloc_packed((size_t)cout * 9 * c.cinp);
    mat(c.w, cout, 9 * c.cinp, t(n + ".w"), 2, 9 * cin, cin, c.cinp);
    c.b = param(n + ".b");
    return c;
  }
  VConv lin(const std::string& n, int cin, int cout) {
    VConv c;
    c.cin = c.cinp = cin;
    c.cout = cout;
    c.taps = 1;
    c.w = alloc_packed((size_t)cout * cin);
    mat(c.w, cout, cin, t(n + ".w"), 0, cin, 0, 0);
    c.b = param(n + ".b");
    return c;
  }
  VRes res(const std::string& p, int cin, int cout) {
    VRes r;
    r.cin = cin;
    r.cout = cout;
    r.g1 = param(p + ".gn1.g");
    r.b1 = param(p + ".gn1.b");
    r.c1 = conv3(p + ".conv1", cin, cout);
    r.g2 = param(p + ".gn2.g");
    r.b2 = param(p + ".gn2.b");
    r.c2 = conv3(p + ".conv2", cout, cout);
    r.has_skip = cin != cout;
    if (r.has_skip) r.skip = lin(p + ".skip", cin, cout);
    return r;
  }
};

void vae_build(Vae* v, VPacker& pk) {
  const dn_vae_config& c = v->cfg;
  const int L = c.n_levels, top = c.channels[L - 1];
  v->pq_w = pk.param("post_quant.w");
  v->pq_b = pk.param("post_quant.b");
  v->conv_in = pk.conv3("conv_in", c.latent_c, top);
  v->mid0 = pk.res("mid.res0", top, top);
  v->attn_g = pk.param("mid.attn.gn.g");
  v->attn_b = pk.param("mid.attn.gn.b");
  // fused q, k, v: rows [0, C) q, [C, 2C) k, [2C, 3C) v, each packed into its row range
  // (C is a multiple of 32, so a range starts on a whole fragment block); biases likewise
  v->qkv.cin = v->qkv.cinp = top;
  v->qkv.cout = 3 * top;
  v->qkv.taps = 1;
  v->qkv.w = pk.alloc_packed((size_t)3 * top * top);
  v->qkv.b = pk.alloc_params(3 * top);
  const char* qkv_names[3] = {"mid.attn.q", "mid.attn.k", "mid.attn.v"};
  for (int j = 0; j < 3; ++j) {
    if (pk.dry) continue;
    void* dst = static_cast<char*>(v->qkv.w) + (size_t)j * top * top * v->esz;
    pk.mat(dst, top, top, pk.t(std::string(qkv_names[j]) + ".w"), 0, top, 0, 0);
    const TensorSpec& bs = pk.t(std::string(qkv_names[j]) + ".b");
    DN_HIP(hipMemcpyAsync(v->qkv.b + (size_t)j * top, pk.blob + bs.offset, top * 4, hipMemcpyDeviceToDevice, pk.s));
  }
  v->proj = pk.lin("mid.attn.o", top, top);
  v->mid1 = pk.res("mid.res1", top, top);
  v->levels.clear();
  int prev = top;
  for (int l = L - 1; l >= 0; --l) {
    VLevel lv;
    lv.c = c.channels[l];
    for (int j = 0; j <= c.layers_per_block; ++j) {
      lv.res.push_back(pk.res("up" + std::to_string(l) + "." + std::to_string(j), prev, c.channels[l]));
      prev = c.channels[l];
    }
    lv.up = l > 0;
    if (lv.up) lv.up_conv = pk.conv3("up" + std::to_string(l) + ".up", c.channels[l], c.channels[l]);
    v->levels.push_back(lv);
  }
  v->out_g = pk.param("out.gn.g");
  v->out_b = pk.param("out.gn.b");
  v->conv_out = pk.conv3("conv_out", c.channels[0], c.out_c);
}

}  // namespace
}  // namespace dn

namespace dn {
namespace {

// Executor of one decode; with dry = true it only sizes the workspace (largest
// activation, GroupNorm partials, split-K slabs).
template <typename T> struct VaeExec {
  Vae* v;
  hipStream_t s;
  int n;
  bool dry = false;
  size_t act = 0, gnp = 0, gns = 0, split = 0;

  void need_act(long long e) { act = std::max(act, (size_t)e); }

  void gemm_(GemmParams& p) {
    const GemmPlan g = gemm_plan<T>(p.M, p.N, p.K, 0, v->cus, p.vt == nullptr, false, p.taps == 9);
    if (dry) {
      split = std::max(split, gemm_workspace_floats(g, p.M, p.N));
      return;
    }
    p.zero16 = v->zero;
    p.part = v->split;
    p.part_floats = v->split_floats;
    gemm<T>(p, g, s);
  }
  // 3x3 conv (optionally on the nearest-x2 upsampled input) or 1x1 layer over NHWC rows
  void conv(const VConv& w, const void* x, int H, int W, int up, void* out, const void* resid, bool out_f32 = false) {
    const int Ho = up ? 2 * H : H, Wo = up ? 2 * W : W;
    GemmParams p;
    p.a0 = x;
    p.c0 = w.cinp;
    p.lda0 = w.cinp;
    p.taps = w.taps;
    p.in_h = H;
    p.in_w = W;
    p.up = up;
    p.out_h = Ho;
    p.out_w = Wo;
    p.stride = 1;
    p.b = w.w;
    p.ldb = w.taps * w.cinp;
    p.M = n * Ho * Wo;
    p.N = w.cout;
    p.K = w.taps * w.cinp;
    p.bias = w.b;
    p.resid = resid;
    p.ldr = w.cout;
    p.out = out;
    p.ldo = w.cout;
    p.out_f32 = out_f32;
    p.n_store = w.cout;
    need_act((long long)p.M * w.cout);
    gemm_(p);
  }
  void gn(const void* x, int HW, int C, const float* g, const float* b, bool silu, void* y) {
    need_act((long long)n * HW * C);
    if (dry) {
      gnp = std::max(gnp, groupnorm_workspace_floats(n, HW, C, v->cfg.gn_groups));
      gns = std::max(gns, (size_t)2 * n * C);
      return;
    }
    GroupNormParams p;
    p.x0 = x;
    p.c0 = C;
    p.n = n;
    p.HW = HW;
    p.G = v->cfg.gn_groups;
    p.gamma = g;
    p.beta = b;
    p.eps = v->cfg.gn_eps;
    p.silu = silu;
    p.y = y;
    p.partial = v->gn_partial;
    p.stats = v->gn_stats;
    groupnorm<T>(p, s);
  }
  // ResBlock x (in X) -> out: skip(x) + conv2(SiLU(GN2(conv1(SiLU(GN1(x))))))
  void res(const VRes& r, const void* x, int H, int W, void* out) {
    const int HW = H * W;
    gn(x, HW, r.cin, r.g1, r.b1, true, v->G);
    conv(r.c1, v->G, H, W, 0, v->Hh, nullptr);
    gn(v->Hh, HW, r.cout, r.g2, r.b2, true, v->G);
    const void* resid = x;
    if (r.has_skip) {
      conv(r.skip, x, H, W, 0, v->Sk, nullptr);
      resid = v->Sk;
    }
    conv(r.c2, v->G, H, W, 0, out, resid);
  }
  // Middle-block attention x -> out over the HW positions of each sample, one head of C.
  void attention(const void* x, int H, int W, void* out) {
    const int HW = H * W, C = v->qkv.cin;
    const size_t e = sizeof(T);
    gn(x, HW, C, v->attn_g, v->attn_b, false, v->G);
    // Q, K -> qkvbuf [n HW][2C]; V -> vt [n][1][C][HW] (transposed by the epilogue)
    GemmParams p;
    p.a0 = v->G;
    p.c0 = C;
    p.lda0 = C;
    p.b = v->qkv.w;
    p.ldb = C;
    p.M = n * HW;
    p.N = 3 * C;
    p.K = C;
    p.bias = v->qkv.b;
    p.out = v->qkvbuf;
    p.ldo = 2 * C;
    p.n_store = 3 * C;
    p.vt = v->vt;
    p.vt_col0 = 2 * C;
    p.vt_dp = C;
    p.vt_heads = 1;
    p.vt_seq = HW;
    p.vt_ld = HW;
    need_act((long long)n * HW * 2 * C);
    gemm_(p);
    const bool frag_s = sizeof(T) == 2 && gemm_frag_layout(HW, C);
    const bool frag_v = sizeof(T) == 2 && gemm_frag_layout(C, HW);
    for (int b = 0; b < n; ++b) {
      const T* qb = static_cast<const T*>(v->qkvbuf) + (size_t)b * HW * 2 * C;
      const T* vtb = static_cast<const T*>(v->vt) + (size_t)b * C * HW;
      // scores S = Q K^T (fp32)
      GemmParams sp;
      sp.a0 = qb;
      sp.c0 = C;
      sp.lda0 = 2 * C;
      if (frag_s) {
        if (!dry) to_frag(reinterpret_cast<const bf16*>(qb + C), HW, C, 2 * C, static_cast<bf16*>(v->kpack), s);
        sp.b = v->kpack;
        sp.ldb = C;
      } else {
        sp.b = qb + C;
        sp.ldb = 2 * C;
      }
      sp.M = HW;
      sp.N = HW;
      sp.K = C;
      sp.out = v->S;
      sp.ldo = HW;
      sp.out_f32 = 1;
      sp.n_store = HW;
      gemm_(sp);
      if (!dry)
        hipLaunchKernelGGL(softmax_rows_kernel<T>, dim3(HW), dim3(256), 0, s, v->S, static_cast<T*>(v->P), HW,
                           static_cast<float>(1.4426950408889634 / std::sqrt((double)C)));
      // O = P V
      GemmParams op;
      op.a0 = v->P;
      op.c0 = HW;
      op.lda0 = HW;
      if (frag_v) {
        if (!dry) to_frag(reinterpret_cast<const bf16*>(vtb), C, HW, HW, static_cast<bf16*>(v->vpack), s);
        op.b = v->vpack;
      } else {
        op.b = vtb;
      }
      op.ldb = HW;
      op.M = HW;
      op.N = C;
      op.K = HW;
      op.out = static_cast<char*>(v->o) + (size_t)b * HW * C * e;
      op.ldo = C;
      op.n_store = C;
      gemm_(op);
    }
    conv(v->proj, v->o, H, W, 0, out, x);
  }

  void decode(const float* z, float* img) {
    const dn_vae_config& c = v->cfg;
    int H = c.latent_h, W = c.latent_w;
    const int HW0 = H * W;
    if (!dry)
      hipLaunchKernelGGL(vae_input_kernel<T>, dim3(blocks((long long)n * HW0)), dim3(256), 0, s, z, v->pq_w, v->pq_b,
                         1.f / c.scaling_factor, static_cast<T*>(v->xin), n, c.latent_c, HW0);
    conv(v->conv_in, v->xin, H, W, 0, v->X, nullptr);
    res(v->mid0, v->X, H, W, v->Y);
    attention(v->Y, H, W, v->X);
    res(v->mid1, v->X, H, W, v->Y);
    void* cur = v->Y;
    void* other = v->X;
    for (const VLevel& lv : v->levels) {
      for (const VRes& r : lv.res) {
        res(r, cur, H, W, other);
        std::swap(cur, other);
      }
      if (lv.up) {
        conv(lv.up_conv, cur, H, W, 1, other, nullptr);
        std::swap(cur, other);
        H *= 2;
        W *= 2;
      }
    }
    gn(cur, H * W, c.channels[0], v->out_g, v->out_b, true, v->G);
    conv(v->conv_out, v->G, H, W, 0, v->out, nullptr, true);
    if (!dry)
      hipLaunchKernelGGL(vae_output_kernel, dim3(blocks((long long)n * c.out_c * H * W)), dim3(256), 0, s, v->out,
                         img, n, c.out_c, H * W);
    if (!dry) DN_HIP(hipGetLastError());
  }
};

void vae_validate(const dn_vae_config& c) {
  DN_CHECK(c.abi_version == DN_ABI_VERSION, "vae config: abi_version mismatch");
  DN_CHECK(c.dtype == DN_FP32 || c.dtype == DN_BF16, "vae config: dtype must be DN_FP32 or DN_BF16");
  DN_CHECK(c.batch >= 1 && c.batch <= 64, "vae config: batch must be in [1, 64]");
  DN_CHECK(c.latent_c >= 1 && c.latent_c <= kVaeCinPad, "vae config: latent_c must be in [1, 64]");
  DN_CHECK(c.n_levels >= 1 && c.n_levels <= DN_MAX_LEVELS, "vae config: n_levels must be in [1, 4]");
  DN_CHECK(c.layers_per_block >= 0 && c.layers_per_block <= 8, "vae config: layers_per_block must be in [0, 8]");
  DN_CHECK(c.gn_groups >= 1 && c.gn_eps > 0.f, "vae config: gn_groups >= 1 and gn_eps > 0");
  DN_CHECK(std::isfinite(c.scaling_factor) && c.scaling_factor > 0.f, "vae config: scaling_factor must be > 0");
  DN_CHECK(c.out_c >= 1 && c.out_c <= 64, "vae config: out_c must be in [1, 64]");
  for (int l = 0; l < c.n_levels; ++l)
    DN_CHECK(c.channels[l] >= 64 && c.channels[l] % 64 == 0 && c.channels[l] <= 2048 &&
                 c.channels[l] % c.gn_groups == 0,
             "vae config: level widths must be multiples of 64 (<= 2048) divisible by gn_groups");
  const long long hw = (long long)c.latent_h * c.latent_w;
  DN_CHECK(c.latent_h >= 1 && c.latent_w >= 1 && hw % 64 == 0 && hw <= 65536,
           "vae config: latent_h * latent_w must be a multiple of 64, at most 65536");
  DN_CHECK(hw << (2 * (c.n_levels - 1)) <= (1ll << 22), "vae config: image larger than 4 M pixels");
}

template <typename T> void vae_walk(Vae* v, hipStream_t s, bool dry, const float* z, float* img, VaeExec<T>* out) {
  VaeExec<T> ex{v, s, v->cfg.batch};
  ex.dry = dry;
  ex.decode(z, img);
  if (out) *out = ex;
}

}  // namespace

std::vector<TensorSpec> vae_weight_table(const dn_vae_config& cfg) {
  vae_validate(cfg);
  return vae_table(cfg);
}

Vae* vae_create(const dn_vae_config& cfg, const float* weights, size_t n_floats, bool on_device) {
  const std::vector<TensorSpec> table = vae_weight_table(cfg);
  const int64_t total = table.back().offset + table.back().numel;
  DN_CHECK(weights != nullptr, "dn_vae_create: null weights");
  DN_CHECK((int64_t)n_floats == total, "dn_vae_create: weight blob has " + std::to_string(n_floats) +
                                           " floats, the decoder needs " + std::to_string(total));
  int dev = 0;
  DN_HIP(hipGetDevice(&dev));
  hipDeviceProp_t prop;
  DN_HIP(hipGetDeviceProperties(&prop, dev));
  if (std::string(prop.gcnArchName).find("gfx950") == std::string::npos)
    throw Error(DN_EUNSUPPORTED, std::string("dn_vae_create: device is ") + prop.gcnArchName + ", built for gfx950");
  std::unique_ptr<Vae> v(new Vae());
  v->cfg = cfg;
  v->bf = cfg.dtype == DN_BF16;
  v->esz = v->bf ? 2 : 4;
  v->cus = prop.multiProcessorCount;
  float* blob = nullptr;
  bool own = false;
  try {
    if (on_device) {
      blob = const_cast<float*>(weights);
    } else {
      DN_HIP(hipMalloc(&blob, (size_t)total * 4));
      own = true;
      DN_HIP(hipMemcpy(blob, weights, (size_t)total * 4, hipMemcpyHostToDevice));
    }
    VPacker pk;
    pk.v = v.get();
    pk.blob = blob;
    for (const auto& t : table) pk.idx[t.name] = &t;
    pk.dry = true;
    vae_build(v.get(), pk);
    DN_HIP(hipMalloc(&v->packed, pk.pk_bytes));
    DN_HIP(hipMalloc(&v->params, pk.pr_floats * 4));
    pk.pk = static_cast<char*>(v->packed);
    pk.pr = v->params;
    pk.pk_bytes = 0;
    pk.pr_floats = 0;
    pk.dry = false;
    vae_build(v.get(), pk);
    DN_HIP(hipStreamSynchronize(nullptr));
    if (own) {
      DN_HIP(hipFree(blob));
      blob = nullptr;
    }
    // workspace, sized by a dry walk of one decode
    size_t act = 0, gnp = 0, gns = 0, split = 0;
    if (v->bf) {
      VaeExec<bf16> ex{v.get(), nullptr, cfg.batch};
      vae_walk<bf16>(v.get(), nullptr, true, nullptr, nullptr, &ex);
      act = ex.act, gnp = ex.gnp, gns = ex.gns, split = ex.split;
    } else {
      VaeExec<float> ex{v.get(), nullptr, cfg.batch};
      vae_walk<float>(v.get(), nullptr, true, nullptr, nullptr, &ex);
      act = ex.act, gnp = ex.gnp, gns = ex.gns, split = ex.split;
    }
    const int L = cfg.n_levels, C = cfg.channels[L - 1];
    const size_t HW = (size_t)cfg.latent_h * cfg.latent_w, n = cfg.batch, e = v->esz;
    const size_t HWo = HW << (2 * (L - 1));
    std::vector<std::pair<void**, size_t>> want = {
        {&v->xin, n * HW * kVaeCinPad * e},
        {&v->X, act * e},
        {&v->Y, act * e},
        {&v->G, act * e},
        {&v->Hh, act * e},
        {&v->Sk, act * e},
        {&v->qkvbuf, n * HW * 2 * C * e},
        {&v->vt, n * C * HW * e},
        {&v->kpack, HW * C * e},
        {&v->vpack, C * HW * e},
        {&v->P, HW * HW * e},
        {&v->o, n * HW * C * e},
        {reinterpret_cast<void**>(&v->S), HW * HW * 4},
        {reinterpret_cast<void**>(&v->out), n * HWo * cfg.out_c * 4},
        {reinterpret_cast<void**>(&v->gn_partial), std::max<size_t>(gnp, 1) * 4},
        {reinterpret_cast<void**>(&v->gn_stats), std::max<size_t>(gns, 1) * 4},
        {&v->zero, 256}};
    size_t bytes = 0;
    for (auto& w : want) bytes += (w.second + 255) / 256 * 256;
    DN_HIP(hipMalloc(&v->arena, bytes));
    size_t off = 0;
    for (auto& w : want) {
      *w.first = static_cast<char*>(v->arena) + off;
      off += (w.second + 255) / 256 * 256;
    }
    DN_HIP(hipMemset(v->xin, 0, n * HW * kVaeCinPad * e));
    DN_HIP(hipMemset(v->zero, 0, 256));
    v->split_floats = split;
    if (split) DN_HIP(hipMalloc(&v->split, split * 4));
  } catch (...) {
    if (own && blob) (void)hipFree(blob);
    vae_destroy(v.release());
    throw;
  }
  return v.release();
}

void vae_decode(Vae* v, const float* latent, float* image, hipStream_t s) {
  DN_CHECK(v && latent && image, "dn_vae_decode: null pointer");
  if (v->bf)
    vae_walk<bf16>(v, s, false, latent, image, nullptr);
  else
    vae_walk<float>(v, s, false, latent, image, nullptr);
}

void vae_destroy(Vae* v) {
  if (!v) return;
  (void)hipDeviceSynchronize();
  if (v->packed) (void)hipFree(v->packed);
  if (v->params) (void)hipFree(v->params);
  if (v->arena) (void)hipFree(v->arena);
  if (v->split) (void)hipFree(v->split);
  delete v;
}

}  // namespace dn
