// UNet denoiser: topology walk, weight packing, workspace and executor.
//
// The module sequence is the latent-diffusion UNet the paper serves (Table 3
// sizes SD-XL and SD 2.0 with this layout): ResNet blocks, spatial transformers
// (self-attention, cross-attention to the text context, GEGLU feed-forward),
// stride-2 downsamples, a middle block and an up path that concatenates skip
// activations, with nearest-x2 upsampling. Activations are NHWC ("token-major")
// in the configured dtype; the transformer residual stream is fp32.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>

#include "model.h"

namespace dn {

// ============================================================================ topology

namespace {

struct Walker {
  // Module events in forward order.
  enum Kind { TIME, CONV_IN, PUSH, POP_CONCAT, RES, TX, DOWN, UP, OUT };
  struct Ev {
    Kind kind;
    std::string prefix;
    int cin = 0, cout = 0, c = 0, depth = 0, heads = 0, head_dim = 0;
  };
};

std::vector<Walker::Ev> walk(const dn_config& cfg) {
  using W = Walker;
  std::vector<W::Ev> ev;
  const int c0 = cfg.model_channels;
  ev.push_back({W::TIME, "time"});
  ev.push_back({W::CONV_IN, "conv_in", cfg.latent_c, c0});
  int ch = c0;
  auto res = [&](const std::string& p, int cin, int cout) {
    W::Ev e{W::RES, p};
    e.cin = cin;
    e.cout = cout;
    ev.push_back(e);
  };
  auto tx = [&](const std::string& p, const dn_level& lv, int depth) {
    W::Ev e{W::TX, p};
    e.c = lv.channels;
    e.depth = depth;
    e.heads = lv.heads;
    e.head_dim = lv.head_dim;
    ev.push_back(e);
  };
  if (cfg.tiny_topology) {
    const dn_level& lv = cfg.level[0];
    res("down0.0.res", c0, lv.channels);
    if (lv.depth > 0) tx("down0.0.tx", lv, lv.depth);
    W::Ev o{W::OUT, "out"};
    o.cin = lv.channels;
    ev.push_back(o);
    return ev;
  }
  std::vector<int> skips{c0};
  ev.push_back({W::PUSH, ""});
  const int L = cfg.n_levels;
  for (int l = 0; l < L; ++l) {
    const dn_level& lv = cfg.level[l];
    for (int j = 0; j < cfg.layers_per_block; ++j) {
      const std::string p = "down" + std::to_string(l) + "." + std::to_string(j);
      res(p + ".res", ch, lv.channels);
      ch = lv.channels;
      if (lv.depth > 0) tx(p + ".tx", lv, lv.depth);
      ev.push_back({W::PUSH, ""});
      skips.push_back(ch);
    }
    if (l < L - 1) {
      W::Ev d{W::DOWN, "down" + std::to_string(l) + ".down"};
      d.c = lv.channels;
      ev.push_back(d);
      ev.push_back({W::PUSH, ""});
      skips.push_back(ch);
    }
  }
  if (cfg.mid_depth >= 0) {
    const dn_level& lv = cfg.level[L - 1];
    res("mid.res0", ch, lv.channels);
    ch = lv.channels;
    if (cfg.mid_depth > 0) tx("mid.tx", lv, cfg.mid_depth);
    res("mid.res1", ch, ch);
  }
  for (int l = L - 1; l >= 0; --l) {
    const dn_level& lv = cfg.level[l];
    for (int j = 0; j <= cfg.layers_per_block; ++j) {
      const int sk = skips.back();
      skips.pop_back();
      W::Ev pc{W::POP_CONCAT, ""};
      pc.c = sk;
      ev.push_back(pc);
      const std::string p = "up" + std::to_string(l) + "." + std::to_string(j);
      res(p + ".res", ch + sk, lv.channels);
      ch = lv.channels;
      if (lv.depth > 0) tx(p + ".tx", lv, lv.depth);
    }
    if (l > 0) {
      W::Ev u{W::UP, "up" + std::to_string(l) + ".up"};
      u.c = lv.channels;
      ev.push_back(u);
    }
  }
  W::Ev o{W::OUT, "out"};
  o.cin = ch;
  ev.push_back(o);
  return ev;
}

struct TableBuilder {
  std::vector<TensorSpec> t;
  int64_t off = 0;
  void add(const std::string& name, std::vector<int64_t> shape, int kind, int fan_in) {
    TensorSpec s;
    s.name = name;
    s.shape = shape;
    s.numel = 1;
    for (auto d : shape) s.numel *= d;
    s.offset = off;
    s.kind = kind;
    s.fan_in = fan_in;
    off += s.numel;
    t.push_back(s);
  }
  void w(const std::string& n, std::vector<int64_t> shape) {
    int64_t fan = 1;
    for (size_t i = 1; i < shape.size(); ++i) fan *= shape[i];
    add(n + ".w", shape, 0, static_cast<int>(fan));
  }
  void wb(const std::string& n, std::vector<int64_t> shape) {
    w(n, shape);
    add(n + ".b", {shape[0]}, 1, t.back().fan_in);
  }
  void norm(const std::string& n, int64_t c) {
    add(n + ".g", {c}, 2, 0);
    add(n + ".b", {c}, 3, 0);
  }
};

}  // namespace

void validate_config(const dn_config& c) {
  DN_CHECK(c.abi_version == DN_ABI_VERSION, "config: abi_version mismatch");
  DN_CHECK(c.dtype == DN_FP32 || c.dtype == DN_BF16 || c.dtype == DN_FP8,
           "config: dtype must be DN_FP32, DN_BF16 or DN_FP8");
  DN_CHECK(c.batch >= 1 && c.batch <= 64, "config: batch must be in [1, 64]");
  DN_CHECK(c.latent_c >= 1 && c.latent_c <= kCinPad, "config: latent_c must be in [1, 64]");
  DN_CHECK(c.n_levels >= 1 && c.n_levels <= DN_MAX_LEVELS, "config: n_levels must be in [1, 4]");
  DN_CHECK(c.model_channels >= 2 && c.model_channels % kCinPad == 0, "config: model_channels must be a multiple of 64");
  DN_CHECK(c.gn_groups >= 1, "config: gn_groups must be >= 1");
  DN_CHECK(c.model_channels % c.gn_groups == 0, "config: model_channels not divisible by gn_groups");
  DN_CHECK(4 * c.model_channels <= 2048, "config: time embedding wider than 2048");
  DN_CHECK(c.layers_per_block >= 1 && c.layers_per_block <= 8, "config: layers_per_block must be in [1, 8]");
  DN_CHECK(c.mid_depth >= -1 && c.mid_depth <= 64, "config: mid_depth must be in [-1, 64]");
  DN_CHECK(c.tiny_topology == 0 || c.tiny_topology == 1, "config: tiny_topology must be 0 or 1");
  DN_CHECK(!c.tiny_topology || c.n_levels == 1, "config: tiny_topology needs exactly one level");
  DN_CHECK(c.ctx_len >= 1 && c.ctx_len <= 4096, "config: ctx_len must be in [1, 4096]");
  DN_CHECK(c.ctx_dim >= 1 && c.ctx_dim % kCinPad == 0, "config: ctx_dim must be a multiple of 64");
  DN_CHECK(c.ff_mult >= 1 && c.ff_mult <= 8, "config: ff_mult must be in [1, 8]");
  DN_CHECK(c.gn_eps > 0.f && c.tx_gn_eps > 0.f && c.ln_eps > 0.f, "config: epsilons must be positive");
  DN_CHECK(c.n_train_steps >= 1 && c.n_train_steps <= 100000, "config: n_train_steps out of range");
  DN_CHECK(c.beta_schedule == DN_BETA_LINEAR || c.beta_schedule == DN_BETA_SCALED_LINEAR, "config: bad beta_schedule");
  DN_CHECK(c.beta_start > 0.f && c.beta_end > 0.f && c.beta_start < 1.f && c.beta_end < 1.f, "config: betas in (0, 1)");
  const int div = c.tiny_topology ? 1 : (1 << (c.n_levels - 1));
  DN_CHECK(c.latent_h >= div && c.latent_w >= div && c.latent_h % div == 0 && c.latent_w % div == 0,
           "config: latent size must be divisible by 2^(n_levels-1)");
  DN_CHECK((int64_t)c.latent_h * c.latent_w <= (1 << 20), "config: latent too large");
  for (int l = 0; l < c.n_levels; ++l) {
    const dn_level& lv = c.level[l];
    DN_CHECK(lv.channels >= 1 && lv.channels % kCinPad == 0 && lv.channels <= 4096,
             "config: level channels must be a multiple of 64, <= 4096");
    DN_CHECK(lv.channels % c.gn_groups == 0, "config: level channels not divisible by gn_groups");
    DN_CHECK(lv.depth >= 0 && lv.depth <= 64, "config: level depth must be in [0, 64]");
    const bool attn = lv.depth > 0 || (l == c.n_levels - 1 && c.mid_depth > 0);
    if (c.dtype == DN_FP8 && (lv.depth > 0 || (l == c.n_levels - 1 && c.mid_depth > 0)))
      DN_CHECK(lv.channels % 128 == 0, "config: DN_FP8 needs transformer widths that are multiples of 128");
    if (attn) {
      DN_CHECK(lv.heads >= 1 && lv.head_dim >= 1 && lv.head_dim <= 64, "config: heads >= 1, head_dim in [1, 64]");
      DN_CHECK(lv.heads * lv.head_dim == lv.channels, "config: heads * head_dim must equal channels");
      DN_CHECK(lv.channels <= 2048, "config: transformer width must be <= 2048");
    }
  }
}

std::vector<TensorSpec> weight_table(const dn_config& cfg) {
  validate_config(cfg);
  TableBuilder tb;
  const int64_t c0 = cfg.model_channels, temb = 4 * c0;
  for (const auto& e : walk(cfg)) {
    switch (e.kind) {
      case Walker::TIME:
        tb.wb("time.lin1", {temb, c0});
        tb.wb("time.lin2", {temb, temb});
        break;
      case Walker::CONV_IN:
        tb.wb("conv_in", {c0, cfg.latent_c, 3, 3});
        break;
      case Walker::RES:
        tb.norm(e.prefix + ".gn1", e.cin);
        tb.wb(e.prefix + ".conv1", {e.cout, e.cin, 3, 3});
        tb.wb(e.prefix + ".temb", {e.cout, temb});
        tb.norm(e.prefix + ".gn2", e.cout);
        tb.wb(e.prefix + ".conv2", {e.cout, e.cout, 3, 3});
        if (e.cin != e.cout) tb.wb(e.prefix + ".skip", {e.cout, e.cin, 1, 1});
        break;
      case Walker::TX: {
        const int64_t c = e.c;
        tb.norm(e.prefix + ".gn", c);
        tb.wb(e.prefix + ".proj_in", {c, c});
        for (int k = 0; k < e.depth; ++k) {
          const std::string b = e.prefix + ".blk" + std::to_string(k);
          tb.norm(b + ".ln1", c);
          tb.w(b + ".attn1.q", {c, c});
          tb.w(b + ".attn1.k", {c, c});
          tb.w(b + ".attn1.v", {c, c});
          tb.wb(b + ".attn1.o", {c, c});
          tb.norm(b + ".ln2", c);
          tb.w(b + ".attn2.q", {c, c});
          tb.w(b + ".attn2.k", {c, cfg.ctx_dim});
          tb.w(b + ".attn2.v", {c, cfg.ctx_dim});
          tb.wb(b + ".attn2.o", {c, c});
          tb.norm(b + ".ln3", c);
          tb.wb(b + ".ff1", {2 * cfg.ff_mult * c, c});
          tb.wb(b + ".ff2", {c, cfg.ff_mult * c});
        }
        tb.wb(e.prefix + ".proj_out", {c, c});
        break;
      }
      case Walker::DOWN:
      case Walker::UP:
        tb.wb(e.prefix, {e.c, e.c, 3, 3});
        break;
      case Walker::OUT:
        tb.norm("out.gn", e.cin);
        tb.wb("conv_out", {cfg.latent_c, e.cin, 3, 3});
        break;
      default:
        break;
    }
  }
  return tb.t;
}

// ============================================================================ model

namespace {

struct ConvW {
  void* w = nullptr;  // [cout][9 * cinp]
  float* b = nullptr;
  int cin = 0, cinp = 0, cout = 0;
};
struct LinW {
  void* w = nullptr;  // [n][k]
  float* b = nullptr;
  float* scale = nullptr;  // fp8 matrices: per-row scales (w then holds E4M3 codes)
  int n = 0, k = 0;
};
struct Norm {
  float* g = nullptr;
  float* b = nullptr;
};
struct ResL {
  Norm gn1, gn2;
  ConvW conv1, conv2;
  LinW skip;
  bool has_skip = false;
  int cin = 0, cout = 0, temb_off = 0;
};
struct TxBlock {
  Norm ln1, ln2, ln3;
  LinW qkv, o1, q2, kv2, o2, ff1, ff2;
  int kv_slot = 0;
};
struct TxL {
  Norm gn;
  LinW proj_in, proj_out;
  std::vector<TxBlock> blocks;
  int c = 0, heads = 0, D = 0, Dp = 0;
};
struct Layer {
  Walker::Kind kind;
  int res = -1, tx = -1, conv = -1;  // indices into Model vectors
  int skip_c = 0;
};

}  // namespace

struct Model {
  dn_config cfg{};
  int n = 0;         // UNet batch = 2B
  size_t esz = 2;    // element size of activations / packed weights
  bool bf = true;
  bool fp8ff = false;  // the GEGLU feed-forward on E4M3 operands (dtype DN_FP8)
  int temb_dim = 0, temb_total = 0;
  // parameters
  void* packed = nullptr;  // all packed weight matrices
  float* params = nullptr; // fp32 biases, norm parameters, time MLP, temb projections
  float *lin1_w = nullptr, *lin1_b = nullptr, *lin2_w = nullptr, *lin2_b = nullptr;
  float *tproj_w = nullptr, *tproj_b = nullptr;
  ConvW conv_in, conv_out;
  Norm out_gn;
  std::vector<ResL> res;
  std::vector<TxL> tx;
  std::vector<ConvW> convs;  // down / up convs
  std::vector<Layer> layers;
  int n_kv_slots = 0;
  // workspace
  void* arena = nullptr;
  void* xin = nullptr;      // [n][HW][64]
  std::vector<void*> act;   // main-path activations, one per producing layer
  void *gn_out = nullptr, *c1 = nullptr, *skipbuf = nullptr;
  float* R = nullptr;       // transformer residual stream fp32
  void *a = nullptr, *qkv = nullptr, *o = nullptr, *q2 = nullptr, *ff = nullptr, *rt = nullptr;
  void* kv = nullptr;       // [slots][n * ctx_len][2P_max]
  size_t kv_slot_elems = 0;    // context keys per cross-attention: [n * ctx_len][P]
  void* vt_self = nullptr;     // self-attention V^T [n][heads][Dp][round_up(HW, 64)]
  void* vt_ctx = nullptr;      // context V^T per cross-attention [n][heads][Dp][round_up(ctx_len, 64)]
  size_t vt_ctx_slot_elems = 0;
  void* ctx_t = nullptr;
  float* eps = nullptr;     // UNet output NHWC fp32
  float *gn_partial = nullptr, *gn_stats = nullptr;
  float *feat = nullptr, *hid = nullptr, *temb = nullptr, *tproj = nullptr;
  double* abar = nullptr;
  int cus = 256;                 // compute units of the device (GEMM planning)
  void* zero = nullptr;          // 256 zero bytes: implicit-conv padding reads
  float* split_ws = nullptr;     // split-K partial slabs (largest need of one step's GEMMs)
  size_t split_floats = 0;
  // shapes per layer output (for the executor)
  std::vector<int> act_h, act_w, act_c;
};

namespace {

struct Packer {
  Model* m;
  const float* blob;  // device fp32 blob
  std::map<std::string, const TensorSpec*> idx;
  char* packed_cur = nullptr;
  size_t packed_bytes = 0;
  float* params_cur = nullptr;
  size_t params_floats = 0;
  bool dry = true;  // first pass only sizes
  hipStream_t s = nullptr;

  const TensorSpec& t(const std::string& n) {
    auto it = idx.find(n);
    DN_CHECK(it != idx.end(), "internal: missing tensor " + n);
    return *it->second;
  }
  void* alloc_packed(size_t elems) {
    const size_t bytes = (elems * m->esz + 255) / 256 * 256;
    void* p = dry ? nullptr : packed_cur + packed_bytes;
    packed_bytes += bytes;
    return p;
  }
  float* alloc_params(size_t n) {
    const size_t f = (n + 63) / 64 * 64;
    float* p = dry ? nullptr : params_cur + params_floats;
    params_floats += f;
    return p;
  }
  float* copy_param(const std::string& n) {
    const TensorSpec& ts = t(n);
    float* d = alloc_params(ts.numel);
    if (!dry) DN_HIP(hipMemcpyAsync(d, blob + ts.offset, ts.numel * 4, hipMemcpyDeviceToDevice, s));
    return d;
  }
  void pack_mat(void* dst, int rows, int cols, int ld, const TensorSpec& src, int row_mode, int col_mode, int src_rows,
                int src_cols, int D = 0, int Dp = 0, int Cin = 0, int Cinp = 0) {
    if (dry) return;
    PackParams p;
    p.dst = dst;
    p.rows = rows;
    p.cols = cols;
    p.ld_dst = ld;
    p.src = blob + src.offset;
    p.row_mode = row_mode;
    p.col_mode = col_mode;
    p.src_rows = src_rows;
    p.src_cols = src_cols;
    p.D = D;
    p.Dp = Dp;
    p.Cin = Cin;
    p.Cinp = Cinp;
    p.frag = m->bf && gemm_frag_layout(rows, cols) && ld == cols;
    if (m->bf)
      pack<bf16>(p, s);
    else
      pack<float>(p, s);
  }
  ConvW conv(const std::string& n, int cin, int cout) {
    ConvW c;
    c.cin = cin;
    c.cinp = (cin + kCinPad - 1) / kCinPad * kCinPad;
    c.cout = cout;
    c.w = alloc_packed((size_t)cout * 9 * c.cinp);
    pack_mat(c.w, cout, 9 * c.cinp, 9 * c.cinp, t(n + ".w"), 0, 2, cout, 9 * cin, 0, 0, cin, c.cinp);
    c.b = copy_param(n + ".b");
    return c;
  }
  LinW lin(const std::string& n, int rows, int cols, bool bias) {
    LinW l;
    l.n = rows;
    l.k = cols;
    l.w = alloc_packed((size_t)rows * cols);
    pack_mat(l.w, rows, cols, cols, t(n + ".w"), 0, 0, rows, cols);
    if (bias) l.b = copy_param(n + ".b");
    return l;
  }
  Norm norm(const std::string& n) { return Norm{copy_param(n + ".g"), copy_param(n + ".b")}; }
  // fp8 (E4M3) matrix: codes in the fp8 fragment order and one scale per row (no bias);
  // row_mode 1 interleaves the GEGLU value / gate rows as pack_mat does
  LinW lin_fp8(const std::string& n, int rows, int cols, int row_mode) {
    LinW l;
    l.n = rows;
    l.k = cols;
    const size_t bytes = gemm_fp8_code_bytes(rows, cols);
    l.w = alloc_packed((bytes + m->esz - 1) / m->esz);
    l.scale = alloc_params((rows + 31) / 32 * 32);
    if (!dry) {
      PackParams p;
      p.dst = l.w;
      p.rows = rows;
      p.cols = cols;
      p.ld_dst = cols;
      p.src = blob + t(n + ".w").offset;
      p.row_mode = row_mode;
      p.col_mode = 0;
      p.src_rows = rows;
      p.src_cols = cols;
      pack_fp8(p, l.scale, s);
    }
    return l;
  }
};

void build(Model* m, Packer& pk, const dn_config& cfg, const std::vector<Walker::Ev>& ev) {
  m->res.clear();
  m->tx.clear();
  m->convs.clear();
  m->layers.clear();
  m->n_kv_slots = 0;
  const int c0 = cfg.model_channels;
  const int temb = 4 * c0;
  // time MLP (fp32)
  m->lin1_w = pk.copy_param("time.lin1.w");
  m->lin1_b = pk.copy_param("time.lin1.b");
  m->lin2_w = pk.copy_param("time.lin2.w");
  m->lin2_b = pk.copy_param("time.lin2.b");
  // temb projections of every ResBlock, concatenated [total][temb]
  int total = 0;
  for (const auto& e : ev)
    if (e.kind == Walker::RES) total += e.cout;
  m->temb_total = total;
  m->tproj_w = pk.alloc_params((size_t)total * temb);
  m->tproj_b = pk.alloc_params(total);
  int toff = 0;
  for (const auto& e : ev) {
    Layer L{e.kind};
    switch (e.kind) {
      case Walker::CONV_IN:
        m->conv_in = pk.conv("conv_in", cfg.latent_c, c0);
        break;
      case Walker::RES: {
        ResL r;
        r.cin = e.cin;
        r.cout = e.cout;
        r.gn1 = pk.norm(e.prefix + ".gn1");
        r.conv1 = pk.conv(e.prefix + ".conv1", e.cin, e.cout);
        r.gn2 = pk.norm(e.prefix + ".gn2");
        r.conv2 = pk.conv(e.prefix + ".conv2", e.cout, e.cout);
        r.has_skip = e.cin != e.cout;
        if (r.has_skip) {
          r.skip = pk.lin(e.prefix + ".skip", e.cout, e.cin, true);
        }
        r.temb_off = toff;
        if (!pk.dry) {
          const TensorSpec& tw = pk.t(e.prefix + ".temb.w");
          const TensorSpec& tb = pk.t(e.prefix + ".temb.b");
          DN_HIP(hipMemcpyAsync(m->tproj_w + (size_t)toff * temb, pk.blob + tw.offset, tw.numel * 4,
                                hipMemcpyDeviceToDevice, pk.s));
          DN_HIP(hipMemcpyAsync(m->tproj_b + toff, pk.blob + tb.offset, tb.numel * 4, hipMemcpyDeviceToDevice, pk.s));
        }
        toff += e.cout;
        L.res = static_cast<int>(m->res.size());
        m->res.push_back(r);
        break;
      }
      case Walker::TX: {
        TxL x;
        x.c = e.c;
        x.heads = e.heads;
        x.D = e.head_dim;
        x.Dp = e.head_dim <= 32 ? 32 : 64;
        const int C = e.c, P = x.heads * x.Dp, F = cfg.ff_mult;
        x.gn = pk.norm(e.prefix + ".gn");
        x.proj_in = pk.lin(e.prefix + ".proj_in", C, C, true);
        for (int k = 0; k < e.depth; ++k) {
          const std::string b = e.prefix + ".blk" + std::to_string(k);
          TxBlock tb;
          tb.ln1 = pk.norm(b + ".ln1");
          tb.qkv.n = 3 * P;
          tb.qkv.k = C;
          tb.qkv.w = pk.alloc_packed((size_t)3 * P * C);
          const char* qkvn[3] = {".attn1.q", ".attn1.k", ".attn1.v"};
          for (int j = 0; j < 3; ++j)
            pk.pack_mat(pk.dry ? nullptr : static_cast<char*>(tb.qkv.w) + (size_t)j * P * C * m->esz, P, C, C,
                        pk.t(b + qkvn[j] + std::string(".w")), 2, 0, C, C, x.D, x.Dp);
          tb.o1.n = C;
          tb.o1.k = P;
          tb.o1.w = pk.alloc_packed((size_t)C * P);
          pk.pack_mat(tb.o1.w, C, P, P, pk.t(b + ".attn1.o.w"), 0, 1, C, C, x.D, x.Dp);
          tb.o1.b = pk.copy_param(b + ".attn1.o.b");
          tb.ln2 = pk.norm(b + ".ln2");
          tb.q2.n = P;
          tb.q2.k = C;
          tb.q2.w = pk.alloc_packed((size_t)P * C);
          pk.pack_mat(tb.q2.w, P, C, C, pk.t(b + ".attn2.q.w"), 2, 0, C, C, x.D, x.Dp);
          tb.kv2.n = 2 * P;
          tb.kv2.k = cfg.ctx_dim;
          tb.kv2.w = pk.alloc_packed((size_t)2 * P * cfg.ctx_dim);
          pk.pack_mat(tb.kv2.w, P, cfg.ctx_dim, cfg.ctx_dim, pk.t(b + ".attn2.k.w"), 2, 0, C, cfg.ctx_dim, x.D, x.Dp);
          pk.pack_mat(pk.dry ? nullptr : static_cast<char*>(tb.kv2.w) + (size_t)P * cfg.ctx_dim * m->esz, P,
                      cfg.ctx_dim, cfg.ctx_dim, pk.t(b + ".attn2.v.w"), 2, 0, C, cfg.ctx_dim, x.D, x.Dp);
          tb.o2.n = C;
          tb.o2.k = P;
          tb.o2.w = pk.alloc_packed((size_t)C * P);
          pk.pack_mat(tb.o2.w, C, P, P, pk.t(b + ".attn2.o.w"), 0, 1, C, C, x.D, x.Dp);
          tb.o2.b = pk.copy_param(b + ".attn2.o.b");
          tb.ln3 = pk.norm(b + ".ln3");
          tb.ff1.n = 2 * F * C;
          tb.ff1.k = C;
          if (m->fp8ff) {
            tb.ff1 = pk.lin_fp8(b + ".ff1", 2 * F * C, C, 1);
          } else {
            tb.ff1.w = pk.alloc_packed((size_t)2 * F * C * C);
            pk.pack_mat(tb.ff1.w, 2 * F * C, C, C, pk.t(b + ".ff1.w"), 1, 0, 2 * F * C, C);
          }
          tb.ff1.b = pk.alloc_params(2 * F * C);
          if (!pk.dry) pack_bias(tb.ff1.b, 2 * F * C, pk.blob + pk.t(b + ".ff1.b").offset, 2 * F * C, 1, 0, 0, pk.s);
          if (m->fp8ff) {
            tb.ff2 = pk.lin_fp8(b + ".ff2", C, F * C, 0);
            tb.ff2.b = pk.copy_param(b + ".ff2.b");
          } else {
            tb.ff2 = pk.lin(b + ".ff2", C, F * C, true);
          }
          tb.kv_slot = m->n_kv_slots++;
          x.blocks.push_back(tb);
        }
        x.proj_out = pk.lin(e.prefix + ".proj_out", C, C, true);
        L.tx = static_cast<int>(m->tx.size());
        m->tx.push_back(x);
        break;
      }
      case Walker::DOWN:
      case Walker::UP:
        L.conv = static_cast<int>(m->convs.size());
        m->convs.push_back(pk.conv(e.prefix, e.c, e.c));
        break;
      case Walker::OUT:
        m->out_gn = pk.norm("out.gn");
        m->conv_out = pk.conv("conv_out", e.cin, cfg.latent_c);
        break;
      case Walker::POP_CONCAT:
        L.skip_c = e.c;
        break;
      default:
        break;
    }
    m->layers.push_back(L);
  }
}

}  // namespace

// ============================================================================ workspace

namespace {

struct Sizer {
  size_t gn_out = 0, c1 = 0, skip = 0, R = 0, a = 0, qkv = 0, o = 0, q2 = 0, ff = 0, kvslot = 0, gn_partial = 0,
         gn_stats = 0, vt_self = 0, vt_ctx = 0;
  std::vector<size_t> acts;  // elements per main-path activation
};

// Walks the layers with spatial shapes to size every buffer.
void size_workspace(Model* m, Sizer& z) {
  const dn_config& c = m->cfg;
  const int n = m->n;
  int H = c.latent_h, W = c.latent_w, ch = c.model_channels;
  std::vector<int> skipc;
  auto gn = [&](int HW, int C) {
    z.gn_out = std::max(z.gn_out, (size_t)n * HW * C);
    z.gn_partial = std::max(z.gn_partial, groupnorm_workspace_floats(n, HW, C, m->cfg.gn_groups));
    z.gn_stats = std::max(z.gn_stats, (size_t)2 * n * C);
  };
  m->act_h.clear();
  m->act_w.clear();
  m->act_c.clear();
  auto produce = [&](int h, int w, int cc) {
    z.acts.push_back((size_t)n * h * w * cc);
    m->act_h.push_back(h);
    m->act_w.push_back(w);
    m->act_c.push_back(cc);
  };
  int pending_skip = 0;
  for (auto& L : m->layers) {
    const int HW = H * W;
    switch (L.kind) {
      case Walker::CONV_IN:
        produce(H, W, ch);
        break;
      case Walker::POP_CONCAT:
        pending_skip = L.skip_c;
        break;
      case Walker::RES: {
        const ResL& r = m->res[L.res];
        gn(HW, r.cin);
        gn(HW, r.cout);
        z.c1 = std::max(z.c1, (size_t)n * HW * r.cout);
        if (r.has_skip) z.skip = std::max(z.skip, (size_t)n * HW * r.cout);
        ch = r.cout;
        pending_skip = 0;
        produce(H, W, ch);
        break;
      }
      case Walker::TX: {
        const TxL& x = m->tx[L.tx];
        const int P = x.heads * x.Dp;
        gn(HW, x.c);
        z.R = std::max(z.R, (size_t)n * HW * x.c);
        z.a = std::max(z.a, (size_t)n * HW * x.c);
        z.qkv = std::max(z.qkv, (size_t)n * HW * 2 * P);
        z.vt_self = std::max(z.vt_self, (size_t)n * P * ((HW + 63) / 64 * 64));
        z.vt_ctx = std::max(z.vt_ctx, (size_t)n * P * ((c.ctx_len + 63) / 64 * 64));
        z.o = std::max(z.o, (size_t)n * HW * P);
        z.q2 = std::max(z.q2, (size_t)n * HW * P);
        z.ff = std::max(z.ff, (size_t)n * HW * c.ff_mult * x.c);
        z.kvslot = std::max(z.kvslot, (size_t)n * c.ctx_len * P);
        produce(H, W, ch);
        break;
      }
      case Walker::DOWN:
        H /= 2;
        W /= 2;
        produce(H, W, ch);
        break;
      case Walker::UP:
        H *= 2;
        W *= 2;
        produce(H, W, ch);
        break;
      case Walker::OUT:
        gn(HW, ch);
        break;
      default:
        break;
    }
  }
  (void)pending_skip;
}

}  // namespace

// ============================================================================ create / destroy

namespace {
size_t step_split_need(Model* m);  // executor section
}  // namespace


Model* model_create(const dn_config& cfg, const float* weights, size_t n_floats, bool on_device) {
  const std::vector<TensorSpec> table = weight_table(cfg);
  const int64_t total = table.empty() ? 0 : table.back().offset + table.back().numel;
  DN_CHECK(weights != nullptr, "dn_create: null weights");
  DN_CHECK((int64_t)n_floats == total, "dn_create: weight blob has " + std::to_string(n_floats) +
                                           " floats, configuration needs " + std::to_string(total));
  int dev = 0;
  DN_HIP(hipGetDevice(&dev));
  hipDeviceProp_t prop;
  DN_HIP(hipGetDeviceProperties(&prop, dev));
  if (std::string(prop.gcnArchName).find("gfx950") == std::string::npos)
    throw Error(DN_EUNSUPPORTED, std::string("dn_create: device is ") + prop.gcnArchName + ", library built for gfx950");

  std::unique_ptr<Model> m(new Model());
  m->cfg = cfg;
  m->n = 2 * cfg.batch;
  m->bf = cfg.dtype != DN_FP32;
  m->fp8ff = cfg.dtype == DN_FP8;
  m->esz = m->bf ? 2 : 4;
  m->temb_dim = 4 * cfg.model_channels;
  const auto ev = walk(cfg);

  hipStream_t s = nullptr;
  float* blob = nullptr;
  bool own_blob = false;
  try {
    if (on_device) {
      blob = const_cast<float*>(weights);
    } else {
      DN_HIP(hipMalloc(&blob, (size_t)total * 4));
      own_blob = true;
      DN_HIP(hipMemcpy(blob, weights, (size_t)total * 4, hipMemcpyHostToDevice));
    }
    Packer pk;
    pk.m = m.get();
    pk.blob = blob;
    for (const auto& t : table) pk.idx[t.name] = &t;
    pk.dry = true;
    build(m.get(), pk, cfg, ev);
    const size_t packed_bytes = pk.packed_bytes, params_floats = pk.params_floats;
    DN_HIP(hipMalloc(&m->packed, packed_bytes));
    DN_HIP(hipMalloc(&m->params, params_floats * 4));
    pk.packed_cur = static_cast<char*>(m->packed);
    pk.params_cur = m->params;
    pk.packed_bytes = 0;
    pk.params_floats = 0;
    pk.dry = false;
    pk.s = s;
    build(m.get(), pk, cfg, ev);
    DN_HIP(hipStreamSynchronize(s));
    if (own_blob) {
      DN_HIP(hipFree(blob));
      blob = nullptr;
    }

    // Workspace.
    Sizer z;
    size_workspace(m.get(), z);
    const int HW0 = cfg.latent_h * cfg.latent_w;
    const size_t e = m->esz;
    std::vector<std::pair<void**, size_t>> want;  // (slot, bytes)
    want.push_back({&m->xin, (size_t)m->n * HW0 * kCinPad * e});
    m->act.assign(z.acts.size(), nullptr);
    for (size_t i = 0; i < z.acts.size(); ++i) want.push_back({&m->act[i], z.acts[i] * e});
    want.push_back({&m->gn_out, z.gn_out * e});
    want.push_back({&m->c1, z.c1 * e});
    want.push_back({&m->skipbuf, std::max<size_t>(z.skip, 1) * e});
    want.push_back({reinterpret_cast<void**>(&m->R), std::max<size_t>(z.R, 1) * 4});
    want.push_back({&m->a, std::max<size_t>(z.a, 1) * e});
    want.push_back({&m->rt, std::max<size_t>(z.a, 1) * e});
    want.push_back({&m->qkv, std::max<size_t>(z.qkv, 1) * e});
    want.push_back({&m->o, std::max<size_t>(z.o, 1) * e});
    want.push_back({&m->q2, std::max<size_t>(z.q2, 1) * e});
    want.push_back({&m->ff, std::max<size_t>(z.ff, 1) * e});
    m->kv_slot_elems = z.kvslot;
    want.push_back({&m->kv, std::max<size_t>(z.kvslot * m->n_kv_slots, 1) * e});
    m->vt_ctx_slot_elems = z.vt_ctx;
    want.push_back({&m->vt_ctx, std::max<size_t>(z.vt_ctx * m->n_kv_slots, 1) * e});
    want.push_back({&m->vt_self, std::max<size_t>(z.vt_self, 1) * e});
    want.push_back({&m->ctx_t, (size_t)m->n * cfg.ctx_len * cfg.ctx_dim * e});
    want.push_back({reinterpret_cast<void**>(&m->eps), (size_t)m->n * HW0 * cfg.latent_c * 4});
    want.push_back({reinterpret_cast<void**>(&m->gn_partial), z.gn_partial * 4});
    want.push_back({reinterpret_cast<void**>(&m->gn_stats), z.gn_stats * 4});
    want.push_back({reinterpret_cast<void**>(&m->feat), (size_t)kMaxSteps * cfg.model_channels * 4});
    want.push_back({reinterpret_cast<void**>(&m->hid), (size_t)kMaxSteps * m->temb_dim * 4});
    want.push_back({reinterpret_cast<void**>(&m->temb), (size_t)kMaxSteps * m->temb_dim * 4});
    want.push_back({reinterpret_cast<void**>(&m->tproj), (size_t)kMaxSteps * m->temb_total * 4});
    want.push_back({reinterpret_cast<void**>(&m->abar), (size_t)cfg.n_train_steps * 8});
    want.push_back({&m->zero, 256});
    size_t bytes = 0;
    for (auto& w : want) bytes += (w.second + 255) / 256 * 256;
    DN_HIP(hipMalloc(&m->arena, bytes));
    size_t off = 0;
    for (auto& w : want) {
      *w.first = static_cast<char*>(m->arena) + off;
      off += (w.second + 255) / 256 * 256;
    }
    DN_HIP(hipMemset(m->xin, 0, (size_t)m->n * HW0 * kCinPad * e));
    DN_HIP(hipMemset(m->zero, 0, 256));
    // V^T rows are padded to whole 64-key tiles; the padding must hold finite values.
    DN_HIP(hipMemset(m->vt_ctx, 0, std::max<size_t>(z.vt_ctx * m->n_kv_slots, 1) * e));
    DN_HIP(hipMemset(m->vt_self, 0, std::max<size_t>(z.vt_self, 1) * e));
    m->cus = prop.multiProcessorCount;
    m->split_floats = step_split_need(m.get());
    if (m->split_floats) DN_HIP(hipMalloc(&m->split_ws, m->split_floats * 4));
    abar_table(m->abar, cfg.n_train_steps, cfg.beta_start, cfg.beta_end, cfg.beta_schedule, s);
    DN_HIP(hipStreamSynchronize(s));
  } catch (...) {
    if (own_blob && blob) (void)hipFree(blob);
    model_destroy(m.release());
    throw;
  }
  return m.release();
}

void model_destroy(Model* m) {
  if (!m) return;
  (void)hipDeviceSynchronize();
  if (m->packed) (void)hipFree(m->packed);
  if (m->params) (void)hipFree(m->params);
  if (m->arena) (void)hipFree(m->arena);
  if (m->split_ws) (void)hipFree(m->split_ws);
  delete m;
}

// ============================================================================ executor

namespace {

template <typename T> struct Exec {
  Model* m;
  hipStream_t s;
  int n;
  bool dry = false;  // walk the step without launching anything
  size_t split_need = 0;  // dry walk: largest split-K workspace (floats) of the step

  void run_gemm(GemmParams& p) {
    const GemmPlan g = p.wscale ? gemm_plan_fp8(p.M, p.N, p.K, p.geglu, m->cus, true, false)
                                : gemm_plan<T>(p.M, p.N, p.K, p.geglu, m->cus, p.vt == nullptr, false, p.taps == 9);
    if (dry) {
      split_need = std::max(split_need, gemm_workspace_floats(g, p.M, p.N));
      return;
    }
    p.zero16 = m->zero;
    p.part = m->split_ws;
    p.part_floats = m->split_floats;
    if (p.wscale)
      gemm_fp8(p, g, s);
    else
      gemm<T>(p, g, s);
  }

  void conv(const ConvW& w, const void* x, int in_h, int in_w, int up, int stride, void* out, int out_h, int out_w,
            const float* rowvec, const void* resid, bool out_f32, int n_store, int ldo) {
    GemmParams p;
    p.a0 = x;
    p.c0 = w.cinp;
    p.lda0 = w.cinp;
    p.taps = 9;
    p.in_h = in_h;
    p.in_w = in_w;
    p.up = up;
    p.out_h = out_h;
    p.out_w = out_w;
    p.stride = stride;
    p.b = w.w;
    p.ldb = 9 * w.cinp;
    p.M = n * out_h * out_w;
    p.N = w.cout;
    p.K = 9 * w.cinp;
    p.bias = w.b;
    p.rowvec = rowvec;
    p.rowvec_ld = 0;
    p.rows_per_sample = out_h * out_w;
    p.resid = resid;
    p.ldr = w.cout;
    p.resid_f32 = 0;
    p.out = out;
    p.ldo = ldo;
    p.out_f32 = out_f32;
    p.n_store = n_store;
    run_gemm(p);
  }

  // Columns >= col0 of a projection written as per-head V^T (see GemmParams::vt).
  struct VtOut {
    void* vt = nullptr;
    int col0 = 0, dp = 0, heads = 0, seq = 1, ld = 0;
  };

  void linear(const LinW& w, const void* x, int ldx, long long M, void* out, int ldo, bool out_f32,
              const void* resid = nullptr, int ldr = 0, bool resid_f32 = false, bool geglu = false,
              const void* x1 = nullptr, int c0 = 0, int c1 = 0, const VtOut& vt = VtOut()) {
    GemmParams p;
    p.a0 = x;
    p.a1 = x1;
    p.c0 = x1 ? c0 : w.k;
    p.c1 = x1 ? c1 : 0;
    p.lda0 = x1 ? c0 : ldx;
    p.lda1 = c1;
    p.taps = 1;
    p.b = w.w;
    p.ldb = w.k;
    p.M = static_cast<int>(M);
    p.N = w.n;
    p.K = w.k;
    p.bias = w.b;
    p.resid = resid;
    p.ldr = ldr;
    p.resid_f32 = resid_f32;
    p.out = out;
    p.ldo = ldo;
    p.out_f32 = out_f32;
    p.geglu = geglu;
    p.n_store = geglu ? w.n / 2 : w.n;
    p.vt = vt.vt;
    p.vt_col0 = vt.col0;
    p.vt_dp = vt.dp;
    p.vt_heads = vt.heads;
    p.vt_seq = vt.seq;
    p.vt_ld = vt.ld;
    p.wscale = w.scale;
    p.out_fp8 = w.scale && geglu;  // the fp8 feed-forward's hidden layer stays in E4M3
    run_gemm(p);
  }

  void groupnorm_(const void* x0, int c0, const void* x1, int c1, int HW, const Norm& nm, float eps, bool silu,
                  void* y) {
    GroupNormParams p;
    p.x0 = x0;
    p.x1 = x1;
    p.c0 = c0;
    p.c1 = c1;
    p.n = n;
    p.HW = HW;
    p.G = m->cfg.gn_groups;
    p.gamma = nm.g;
    p.beta = nm.b;
    p.eps = eps;
    p.silu = silu;
    p.y = y;
    p.partial = m->gn_partial;
    p.stats = m->gn_stats;
    if (!dry) groupnorm<T>(p, s);
  }

  void resblock(const ResL& r, const void* x0, int c0, const void* x1, int c1, int H, int W, const float* tproj_row,
                void* out) {
    const int HW = H * W;
    groupnorm_(x0, c0, x1, c1, HW, r.gn1, m->cfg.gn_eps, true, m->gn_out);
    conv(r.conv1, m->gn_out, H, W, 0, 1, m->c1, H, W, tproj_row + r.temb_off, nullptr, false, r.cout, r.cout);
    groupnorm_(m->c1, r.cout, nullptr, 0, HW, r.gn2, m->cfg.gn_eps, true, m->gn_out);
    const void* resid = x0;
    if (r.has_skip) {
      linear(r.skip, x0, c0, (long long)n * HW, m->skipbuf, r.cout, false, nullptr, 0, false, false, x1, c0, c1);
      resid = m->skipbuf;
    }
    conv(r.conv2, m->gn_out, H, W, 0, 1, out, H, W, nullptr, resid, false, r.cout, r.cout);
  }

  void attention_(const void* q, int ldq, long long q_bs, const void* k, int ldk, long long k_bs, const void* vt,
                  int vt_ld, int Sq, int Skv, const TxL& x) {
    AttnParams a;
    a.q = q;
    a.k = k;
    a.vt = vt;
    a.o = m->o;
    a.ldq = ldq;
    a.ldk = ldk;
    a.vt_ld = vt_ld;
    a.ldo = x.heads * x.Dp;
    a.q_bs = q_bs;
    a.k_bs = k_bs;
    a.o_bs = (long long)Sq * x.heads * x.Dp;
    a.B = n;
    a.heads = x.heads;
    a.Sq = Sq;
    a.Skv = Skv;
    a.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt((double)x.D));
    if (!dry) attention<T>(a, x.Dp, s);
  }

  // A residual-stream update R = (resid ? R : 0) + x W^T + b whose result is layer-normalised
  // next (a = LN(R)). When the plan splits K, the GEMM writes fp32 partial slabs only and
  // one LayerNorm pass sums them with the bias and R, writes R and normalises (no separate
  // reduction kernel); otherwise the GEMM epilogue updates R and a plain LayerNorm follows.
  struct Pending {
    const LinW* w = nullptr;
    int nsplit = 0;   // 0: R already final
    bool resid = true;
  };
  Pending residual_gemm(const LinW& w, const void* x, int ldx, long long M, bool resid) {
    const GemmPlan g = w.scale ? gemm_plan_fp8(static_cast<int>(M), w.n, w.k, 0, m->cus, true, true)
                               : gemm_plan<T>(static_cast<int>(M), w.n, w.k, 0, m->cus, true, true);
    if (!g.frag || g.split == 1) {
      linear(w, x, ldx, M, m->R, w.n, true, resid ? m->R : nullptr, w.n, true);
      return Pending{};
    }
    GemmParams p;
    p.a0 = x;
    p.c0 = w.k;
    p.lda0 = ldx;
    p.taps = 1;
    p.b = w.w;
    p.ldb = w.k;
    p.M = static_cast<int>(M);
    p.N = w.n;
    p.K = w.k;
    p.out = m->R;
    p.ldo = w.n;
    p.out_f32 = 1;
    p.n_store = w.n;
    p.raw_partial = 1;
    p.wscale = w.scale;
    if (dry) {
      split_need = std::max(split_need, gemm_workspace_floats(g, p.M, p.N, true));
    } else {
      p.zero16 = m->zero;
      p.part = m->split_ws;
      p.part_floats = m->split_floats;
      if (w.scale)
        gemm_fp8(p, g, s);
      else
        gemm<T>(p, g, s);
    }
    return Pending{&w, g.split, resid};
  }
  // fp8: the LayerNorm feeding the fp8 feed-forward writes E4M3 codes
  void ln_after(const Pending& pd, long long M, int C, const Norm& nm, bool fp8 = false) {
    if (dry) return;
    if (fp8) {
      if (pd.nsplit)
        layernorm_reduce<uint8_t>(m->R, P_<uint8_t>(m->a), M, C, nm.g, nm.b, m->cfg.ln_eps, m->split_ws, pd.nsplit,
                                  pd.w->b, pd.resid, s);
      else
        layernorm<uint8_t>(m->R, P_<uint8_t>(m->a), M, C, nm.g, nm.b, m->cfg.ln_eps, s);
      return;
    }
    if (pd.nsplit)
      layernorm_reduce<T>(m->R, P_<T>(m->a), M, C, nm.g, nm.b, m->cfg.ln_eps, m->split_ws, pd.nsplit, pd.w->b,
                          pd.resid, s);
    else
      layernorm<T>(m->R, P_<T>(m->a), M, C, nm.g, nm.b, m->cfg.ln_eps, s);
  }

  void transformer(const TxL& x, const void* in, int H, int W, void* out) {
    const int HW = H * W, C = x.c, P = x.heads * x.Dp;
    const long long M = (long long)n * HW;
    const size_t e = sizeof(T);
    groupnorm_(in, C, nullptr, 0, HW, x.gn, m->cfg.tx_gn_eps, false, m->gn_out);
    Pending pd = residual_gemm(x.proj_in, m->gn_out, C, M, false);
    for (size_t bi = 0; bi < x.blocks.size(); ++bi) {
      const TxBlock& b = x.blocks[bi];
      const bool last = bi + 1 == x.blocks.size();
      ln_after(pd, M, C, b.ln1);
      // Q and K land in qkv [M][2P]; V goes to vt_self transposed per head.
      const int ld_self = (HW + 63) / 64 * 64;
      VtOut vs;
      vs.vt = m->vt_self;
      vs.col0 = 2 * P;
      vs.dp = x.Dp;
      vs.heads = x.heads;
      vs.seq = HW;
      vs.ld = ld_self;
      linear(b.qkv, m->a, C, M, m->qkv, 2 * P, false, nullptr, 0, false, false, nullptr, 0, 0, vs);
      const char* qkv = static_cast<const char*>(m->qkv);
      attention_(qkv, 2 * P, (long long)HW * 2 * P, qkv + (size_t)P * e, 2 * P, (long long)HW * 2 * P, m->vt_self,
                 ld_self, HW, HW, x);
      pd = residual_gemm(b.o1, m->o, P, M, true);
      ln_after(pd, M, C, b.ln2);
      linear(b.q2, m->a, C, M, m->q2, P, false);
      const char* kv = static_cast<const char*>(m->kv) + (size_t)b.kv_slot * m->kv_slot_elems * e;
      const char* vtc = static_cast<const char*>(m->vt_ctx) + (size_t)b.kv_slot * m->vt_ctx_slot_elems * e;
      attention_(m->q2, P, (long long)HW * P, kv, P, (long long)m->cfg.ctx_len * P, vtc,
                 (m->cfg.ctx_len + 63) / 64 * 64, HW, m->cfg.ctx_len, x);
      pd = residual_gemm(b.o2, m->o, P, M, true);
      ln_after(pd, M, C, b.ln3, m->fp8ff);
      linear(b.ff1, m->a, C, M, m->ff, m->cfg.ff_mult * C, false, nullptr, 0, false, true);
      if (!last)
        pd = residual_gemm(b.ff2, m->ff, m->cfg.ff_mult * C, M, true);
      else
        linear(b.ff2, m->ff, m->cfg.ff_mult * C, M, m->rt, C, false, m->R, C, true);
    }
    linear(x.proj_out, m->rt, C, M, out, C, false, in, C, false);
  }

  template <typename U> static U* P_(void* p) { return static_cast<U*>(p); }

  // Per-call preparation (after time_features): time embedding MLP and every
  // ResBlock's projection of it for all steps, context conversion, and the
  // context keys / values of every cross-attention.
  void prepare(const float* ctx, int n_steps) {
    const dn_config& c = m->cfg;
    if (!dry) {
      skinny_linear(m->feat, n_steps, c.model_channels, m->lin1_w, m->lin1_b, m->temb_dim, m->hid, m->temb_dim, 0,
                    s);
      skinny_linear(m->hid, n_steps, m->temb_dim, m->lin2_w, m->lin2_b, m->temb_dim, m->temb, m->temb_dim, 1, s);
      skinny_linear(m->temb, n_steps, m->temb_dim, m->tproj_w, m->tproj_b, m->temb_total, m->tproj,
                    m->temb_total, 1, s);
      convert_from_f32<T>(ctx, P_<T>(m->ctx_t), (long long)n * c.ctx_len * c.ctx_dim, s);
    }
    for (const auto& x : m->tx)
      for (const auto& b : x.blocks) {
        void* dst = static_cast<char*>(m->kv) + (size_t)b.kv_slot * m->kv_slot_elems * sizeof(T);
        VtOut vc;
        vc.vt = static_cast<char*>(m->vt_ctx) + (size_t)b.kv_slot * m->vt_ctx_slot_elems * sizeof(T);
        vc.col0 = b.kv2.n / 2;
        vc.dp = x.Dp;
        vc.heads = x.heads;
        vc.seq = c.ctx_len;
        vc.ld = (c.ctx_len + 63) / 64 * 64;
        linear(b.kv2, m->ctx_t, c.ctx_dim, (long long)n * c.ctx_len, dst, b.kv2.n / 2, false, nullptr, 0, false,
               false, nullptr, 0, 0, vc);
      }
  }

  // One UNet evaluation on m->xin for the time embedding of local step `step`;
  // writes m->eps (NHWC fp32 [n][HW][latent_c]).
  void unet(int step) {
    const dn_config& c = m->cfg;
    const float* trow = m->tproj + (size_t)step * m->temb_total;
    int H = c.latent_h, W = c.latent_w;
    std::vector<const void*> skips;
    std::vector<int> skipc;
    const void* h = nullptr;
    int ch = 0;
    size_t ai = 0;
    int pending = 0;
    const void* pend_ptr = nullptr;
    for (const Layer& L : m->layers) {
      switch (L.kind) {
        case Walker::CONV_IN: {
          void* out = m->act[ai++];
          conv(m->conv_in, m->xin, H, W, 0, 1, out, H, W, nullptr, nullptr, false, m->conv_in.cout, m->conv_in.cout);
          h = out;
          ch = m->conv_in.cout;
          break;
        }
        case Walker::PUSH:
          skips.push_back(h);
          skipc.push_back(ch);
          break;
        case Walker::POP_CONCAT:
          pend_ptr = skips.back();
          pending = skipc.back();
          skips.pop_back();
          skipc.pop_back();
          break;
        case Walker::RES: {
          const ResL& r = m->res[L.res];
          void* out = m->act[ai++];
          resblock(r, h, ch, pending ? pend_ptr : nullptr, pending, H, W, trow, out);
          pending = 0;
          pend_ptr = nullptr;
          h = out;
          ch = r.cout;
          break;
        }
        case Walker::TX: {
          void* out = m->act[ai++];
          transformer(m->tx[L.tx], h, H, W, out);
          h = out;
          break;
        }
        case Walker::DOWN: {
          void* out = m->act[ai++];
          conv(m->convs[L.conv], h, H, W, 0, 2, out, H / 2, W / 2, nullptr, nullptr, false, ch, ch);
          H /= 2;
          W /= 2;
          h = out;
          break;
        }
        case Walker::UP: {
          void* out = m->act[ai++];
          conv(m->convs[L.conv], h, H, W, 1, 1, out, 2 * H, 2 * W, nullptr, nullptr, false, ch, ch);
          H *= 2;
          W *= 2;
          h = out;
          break;
        }
        case Walker::OUT:
          groupnorm_(h, ch, nullptr, 0, H * W, m->out_gn, c.gn_eps, true, m->gn_out);
          conv(m->conv_out, m->gn_out, H, W, 0, 1, m->eps, H, W, nullptr, nullptr, true, c.latent_c, c.latent_c);
          break;
        default:
          break;
      }
    }
  }
};

// Largest split-K workspace of one denoise step (a walk that plans every GEMM).
size_t step_split_need(Model* m) {
  if (m->bf) {
    Exec<bf16> ex{m, nullptr, m->n};
    ex.dry = true;
    ex.prepare(nullptr, 1);
    ex.unet(0);
    return ex.split_need;
  }
  Exec<float> ex{m, nullptr, m->n};
  ex.dry = true;
  ex.prepare(nullptr, 1);
  ex.unet(0);
  return ex.split_need;
}

// Timesteps reach the device as kernel arguments (chunks of kTsChunk).
void time_features(Model* m, const int32_t* ts, int n, hipStream_t s) {
  for (int i = 0; i < n; i += kTsChunk) {
    TsChunk c;
    c.count = std::min(kTsChunk, n - i);
    for (int j = 0; j < c.count; ++j) c.t[j] = ts[i + j];
    sinusoid(m->feat + (size_t)i * m->cfg.model_channels, c, m->cfg.model_channels, s);
  }
}

// Writes the latent, rounded to bf16, to every capture slot j whose iteration count
// cap_at[j] equals `done` (the cache stores a prompt's state after K iterations).
void capture_latent(const float* latent, long long numel, int done, const int32_t* cap_at, int n_cap, uint16_t* out,
                    hipStream_t s) {
  for (int j = 0; j < n_cap; ++j)
    if (cap_at[j] == done) convert_from_f32<bf16>(latent, reinterpret_cast<bf16*>(out) + j * numel, numel, s);
}

template <typename T>
void denoise_t(Model* m, float* latent, const float* ctx, const int32_t* ts, int start, int n_steps, float scale,
               const int32_t* cap_at, int n_cap, uint16_t* cap_out, hipStream_t s) {
  const dn_config& c = m->cfg;
  Exec<T> ex{m, s, m->n};
  time_features(m, ts + start, n_steps, s);
  ex.prepare(ctx, n_steps);
  const int HW = c.latent_h * c.latent_w;
  const long long numel = (long long)c.batch * c.latent_c * HW;
  capture_latent(latent, numel, start, cap_at, n_cap, cap_out, s);
  latent_to_input<T>(latent, static_cast<T*>(m->xin), c.batch, c.latent_c, HW, kCinPad, s);
  for (int i = 0; i < n_steps; ++i) {
    ex.unet(i);
    cfg_ddim<T>(m->eps, latent, static_cast<T*>(m->xin), m->abar, ts[start + i], ts[start + i + 1], scale, c.batch,
                c.latent_c, HW, kCinPad, s);
    capture_latent(latent, numel, start + i + 1, cap_at, n_cap, cap_out, s);
  }
}

template <typename T>
void unet_eps_t(Model* m, const float* x, int t, const float* ctx, float scale, float* raw, float* guided,
                hipStream_t s) {
  const dn_config& c = m->cfg;
  Exec<T> ex{m, s, m->n};
  time_features(m, &t, 1, s);
  ex.prepare(ctx, 1);
  const int HW = c.latent_h * c.latent_w;
  latent_to_input<T>(x, static_cast<T*>(m->xin), c.batch, c.latent_c, HW, kCinPad, s);
  ex.unet(0);
  export_eps(m->eps, raw, guided, scale, c.batch, c.latent_c, HW, s);
}

}  // namespace

void model_denoise(Model* m, float* latent, const float* ctx, const int32_t* ts, int n_ts, int start, int n,
                   float scale, hipStream_t s, const int32_t* cap_at, int n_cap, uint16_t* cap_out) {
  DN_CHECK(latent && ctx && ts, "dn_denoise: null pointer");
  DN_CHECK(n_cap >= 0, "dn_denoise_capture: n_capture must be >= 0");
  DN_CHECK(n_cap == 0 || (cap_at && cap_out), "dn_denoise_capture: null capture pointer");
  for (int j = 0; j < n_cap; ++j)
    DN_CHECK(cap_at[j] >= start && (int64_t)cap_at[j] <= (int64_t)start + n,
             "dn_denoise_capture: capture iteration outside [start_step, start_step + n_steps]");
  DN_CHECK(start >= 0 && n >= 0, "dn_denoise: start_step and n_steps must be >= 0");
  DN_CHECK((int64_t)start + n + 1 <= n_ts, "dn_denoise: timesteps shorter than start_step + n_steps + 1");
  DN_CHECK(n <= kMaxSteps, "dn_denoise: n_steps > 1000");
  for (int i = start; i <= start + n; ++i)
    DN_CHECK(ts[i] >= -1 && ts[i] < m->cfg.n_train_steps, "dn_denoise: timestep out of range");
  if (n == 0) {
    // nothing to run; a capture at start_step is still the input latent
    capture_latent(latent, (long long)m->cfg.batch * m->cfg.latent_c * m->cfg.latent_h * m->cfg.latent_w, start,
                   cap_at, n_cap, cap_out, s);
    return;
  }
  if (m->bf)
    denoise_t<bf16>(m, latent, ctx, ts, start, n, scale, cap_at, n_cap, cap_out, s);
  else
    denoise_t<float>(m, latent, ctx, ts, start, n, scale, cap_at, n_cap, cap_out, s);
}

void model_unet_eps(Model* m, const float* x, int t, const float* ctx, float scale, float* raw, float* guided,
                    hipStream_t s) {
  DN_CHECK(x && ctx && raw, "dn_unet_eps: null pointer");
  DN_CHECK(t >= -1 && t < m->cfg.n_train_steps, "dn_unet_eps: timestep out of range");
  if (m->bf)
    unet_eps_t<bf16>(m, x, t, ctx, scale, raw, guided, s);
  else
    unet_eps_t<float>(m, x, t, ctx, scale, raw, guided, s);
}

}  // namespace dn
