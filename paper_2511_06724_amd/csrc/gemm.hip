// MFMA GEMM with an implicit-convolution A loader (gfx950).
//
// One kernel template covers every dense contraction of the UNet: the 3x3
// convolutions (implicit GEMM over NHWC activations, with stride-2 downsample,
// nearest-x2 upsample addressing and two-source channel concatenation), the
// 1x1 skip convolutions and every linear layer of the transformer blocks
// (fused QKV, attention outputs, GEGLU feed-forward, projections).
//
// Tiling: 256 threads = 4 waves in a 2x2 grid; block tile BM x BN in
// {128x128, 64x128, 64x64, 256x128, 128x256}, wave tile (BM/2) x (BN/2) built from 32x32x16 MFMA blocks; K
// step BK = 128 bytes of each row (64 bf16 / 32 fp32), staged through
// double-buffered LDS (one barrier per K step; the next tile's global loads are
// issued a full K step ahead). The MFMA is issued as C^T = B A^T so that each
// lane holds four consecutive output columns of one row: the epilogue stores
// 8 (bf16) or 16 (fp32) contiguous bytes per lane and reads bias / residual as
// vectors. Rows of A and B beyond M / N are clamped on load and masked on store.
//
// Work distribution: tiles are numbered so that each XCD (consecutive
// workgroup ids go round-robin over the 8 XCDs) works through a contiguous band
// of output columns with all row tiles, keeping that band of B in its L2.
#include <algorithm>
#include <cmath>

#include "gemm_epilogue.h"

namespace dn {
namespace {

constexpr int kThreads = 256;
constexpr int kXcds = 8;

template <typename T, int BM, int BN, bool CONV>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmParams p, int mt, int nt) {
  using MM = Mma<T>;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BK = gemm_bk<T>();
  constexpr int VPR = BK / VEC;          // 16-byte vectors per tile row (8)
  constexpr int SA = BK + VEC;           // LDS row stride in elements (16-byte pad)
  constexpr int RPP = kThreads / VPR;    // tile rows covered by one pass of the block (32)
  constexpr int AV = BM / RPP;
  constexpr int BV = BN / RPP;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int STAGE = (BM + BN) * SA;

  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* lds = reinterpret_cast<T*>(smem_raw);

  // ---- tile assignment (XCD-aware: each XCD walks a contiguous band of columns)
  const int total = mt * nt;
  const int wg = blockIdx.x;
  const int xcd = wg % kXcds, idx = wg / kXcds;
  const int base = total / kXcds, rem = total % kXcds;
  const int logical = xcd * base + min(xcd, rem) + idx;
  const int n_tile = logical / mt;
  const int m_tile = logical - n_tile * mt;
  const int n0 = n_tile * BN;
  const int m0 = m_tile * BM;
  const int kt_begin = 0;
  const int kt_end = p.K / BK;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int vc = tid % VPR;
  const int rr = tid / VPR;

  // Per-thread A row descriptors.
  int a_row[AV];
  int a_sy[AV], a_oy[AV], a_ox[AV];
  const int opix = p.out_h * p.out_w;
#pragma unroll
  for (int i = 0; i < AV; ++i) {
    const int m = min(m0 + rr + i * RPP, p.M - 1);
    a_row[i] = m;
    if (CONV) {
      const int s = m / opix;
      const int rem2 = m - s * opix;
      const int oy = rem2 / p.out_w;
      const int ox = rem2 - oy * p.out_w;
      a_sy[i] = s * p.in_h;
      a_oy[i] = oy * p.stride - 1;
      a_ox[i] = ox * p.stride - 1;
    }
  }
  const T* b_ptr[BV];
#pragma unroll
  for (int i = 0; i < BV; ++i) {
    const int n = min(n0 + rr + i * RPP, p.N - 1);
    b_ptr[i] = static_cast<const T*>(p.b) + (long long)n * p.ldb + vc * VEC;
  }

  uint4 ra[AV], rb[BV];
  const int ct = p.c0 + p.c1;
  const int hl = p.in_h << p.up, wl = p.in_w << p.up;

  auto load_tile = [&](int k0) {
    int tap = 0, c = k0;
    if (CONV) {
      tap = k0 / ct;
      c = k0 - tap * ct;
    }
    const T* src;
    int ld;
    if (c < p.c0) {
      src = static_cast<const T*>(p.a0);
      ld = p.lda0;
    } else {
      src = static_cast<const T*>(p.a1);
      ld = p.lda1;
      c -= p.c0;
    }
    c += vc * VEC;
    if (CONV) {
      const int ky = tap / 3, kx = tap - 3 * (tap / 3);
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        const int iy = a_oy[i] + ky, ix = a_ox[i] + kx;
        if (iy >= 0 && iy < hl && ix >= 0 && ix < wl) {
          const long long pix = (long long)(a_sy[i] + (iy >> p.up)) * p.in_w + (ix >> p.up);
          ra[i] = ld16(src + pix * ld + c);
        } else {
          ra[i] = make_uint4(0u, 0u, 0u, 0u);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < AV; ++i) ra[i] = ld16(src + (long long)a_row[i] * ld + c);
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) rb[i] = ld16(b_ptr[i] + k0);
  };
  auto store_tile = [&](int buf) {
    T* As = lds + buf * STAGE;
    T* Bs = As + BM * SA;
#pragma unroll
    for (int i = 0; i < AV; ++i) st16(As + (rr + i * RPP) * SA + vc * VEC, ra[i]);
#pragma unroll
    for (int i = 0; i < BV; ++i) st16(Bs + (rr + i * RPP) * SA + vc * VEC, rb[i]);
  };

  // acc[i][j]: rows = output columns n0 + wn*WN + 32 j + acc_row(r),
  //            column = output row m0 + wm*WM + 32 i + (lane % 32).
  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int frag_off = (lane & 31) * SA + (lane >> 5) * MM::KPL;
  if (kt_begin < kt_end) {
    load_tile(kt_begin * BK);
    store_tile(0);
    if (kt_begin + 1 < kt_end) load_tile((kt_begin + 1) * BK);
    __syncthreads();
    for (int kt = kt_begin; kt < kt_end; ++kt) {
      const int cur = (kt - kt_begin) & 1;
      const T* As = lds + cur * STAGE + wm * WM * SA + frag_off;
      const T* Bs = lds + cur * STAGE + BM * SA + wn * WN * SA + frag_off;
#pragma unroll
      for (int ks = 0; ks < BK / MM::KS; ++ks) {
        typename MM::frag a[FM], b[FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) a[i] = MM::load(As + i * 32 * SA + ks * MM::KS);
#pragma unroll
        for (int j = 0; j < FN; ++j) b[j] = MM::load(Bs + j * 32 * SA + ks * MM::KS);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) acc[i][j] = MM::mma(b[j], a[i], acc[i][j]);
      }
      if (kt + 1 < kt_end) {
        store_tile(cur ^ 1);
        if (kt + 2 < kt_end) load_tile((kt + 2) * BK);
      }
      __syncthreads();
    }
  }

  const int col = lane & 31;
  const int h4 = 4 * (lane >> 5);

  // ---- epilogue
  if (!p.geglu) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int m = m0 + wm * WM + i * 32 + col;
      if (m >= p.M) continue;
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = n0 + wn * WN + j * 32 + 8 * g + h4;
          float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
          epilogue_group<T>(p, m, n, v);
        }
    }
  } else {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int m = m0 + wm * WM + i * 32 + col;
      if (m >= p.M) continue;
#pragma unroll
      for (int j = 0; j < FN / 2; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int nv = n0 + wn * WN + 2 * j * 32 + 8 * g + h4;   // value column (gate = nv + 32)
          const int o = (n0 + wn * WN) / 2 + j * 32 + 8 * g + h4;  // output column
          if (o >= p.n_store) continue;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float a = acc[i][2 * j][4 * g + e] + (p.bias ? p.bias[nv + e] : 0.f);
            const float gg = acc[i][2 * j + 1][4 * g + e] + (p.bias ? p.bias[nv + 32 + e] : 0.f);
            v[e] = a * gelu_erf(gg);
          }
          store4<T>(p, m, o, v, p.n_store);
        }
    }
  }
}

template <typename T, int BM, int BN, bool CONV>
void launch(const GemmParams& p, hipStream_t s) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SA = gemm_bk<T>() + VEC;
  const size_t lds = size_t(2) * (BM + BN) * SA * sizeof(T);
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<T, BM, BN, CONV>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  const int mt = ceil_div(p.M, BM), nt = ceil_div(p.N, BN);
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, CONV>), dim3(mt * nt), dim3(kThreads), lds, s, p, mt, nt);
  DN_HIP(hipGetLastError());
}

template <typename T, bool CONV> void dispatch(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  if (g.bm == 256 && g.bn == 128)
    launch<T, 256, 128, CONV>(p, s);
  else if (g.bm == 128 && g.bn == 256)
    launch<T, 128, 256, CONV>(p, s);
  else if (g.bm == 64 && g.bn == 128)
    launch<T, 64, 128, CONV>(p, s);
  else if (g.bm == 64 && g.bn == 64)
    launch<T, 64, 64, CONV>(p, s);
  else
    launch<T, 128, 128, CONV>(p, s);
}

}  // namespace

// Tile choice of the register-staged kernel (fp32, the check mode, and bf16 shapes the
// fragment layout does not take: N % 32 != 0 or K % 64 != 0, e.g. conv_in and the
// output head): 64 x 64 tiles when there are fewer 128 x 128 tiles than CUs (GEGLU
// needs 64-column value/gate pairs per wave, i.e. a block width of at least 128), else
// 128 x 128 tiles with two resident workgroups per CU.
// Fragment-B kernel (bf16 weights in fragment order). Three tile variants share a CU
// between several workgroups: 128 x 256 (two per CU), 128 x 128 (two) and 64 x 128
// (four); five-wave 64 x 160 and 128 x 160 tiles run one workgroup per CU (the M = 2048,
// N = 1280 projections are exactly one 64 x 160 tile per CU, where 64 x 128 tiles put
// two workgroups on a quarter of the CUs; 128 x 160 tiles cover the 8192-row N = 640
// layers in one round and the N = 320 convolutions without padding columns). The plan
// minimises a cost model fitted to measured SD-XL GEMM times on MI355X
// (bf16, weights streamed from HBM; one fit for the linear layers, one for the implicit
// convolutions): a run takes ceil(units / slots) rounds, a round
// costs the MFMA work of the units resident on a CU at a per-CU rate R plus a fixed
// prologue cost O; the epilogue adds E per million outputs, and a K split adds the fp32
// slabs written and read by the reduction (when the consumer, a LayerNorm, sums the
// slabs itself: its extra slab reads, at the cost per slab measured for that kernel
// together with the GEMM). GEGLU needs 64-column value/gate pairs per wave (128 x 256).
GemmPlan frag_plan(int M, int N, int K, int geglu, int cus, bool allow_split, bool fused_reduce, bool conv) {
  struct Var {
    int bm, bn, wg;
    double rate, fixed, epi;  // FLOP per us per CU, us per round, us per 1e6 outputs
  };
  // separate fits for the linear layers and the implicit convolutions (whose A gather
  // and tap masks change the per-stage cost)
  static const Var lin_vars[] = {{128, 256, 2, 2.4e6, 5.0, 1.0},
                                 {128, 128, 2, 2.0e6, 8.0, 0.0},
                                 {64, 128, 4, 1.6e6, 3.0, 0.0},
                                 {64, 160, 1, 3.1e6, 9.4, 0.0},
                                 {128, 160, 1, 4.14e6, 16.7, 0.0}};
  static const Var conv_vars[] = {{128, 256, 2, 2.4e6, 5.0, 3.0},
                                  {128, 128, 2, 1.6e6, 1.0, 0.0},
                                  {64, 128, 4, 1.6e6, 1.0, 0.0},
                                  {128, 160, 1, 3.39e6, 10.7, 0.0}};
  const Var* vars = conv ? conv_vars : lin_vars;
  const int nvars = conv ? 4 : 5;  // the five-wave 64 x 160 tile takes linear layers only
  // convolutions: a partly filled round costs more than its average load per CU (the
  // CUs that hold one more unit finish last)
  const double fill_penalty = conv ? 0.25 : 0.0;
  GemmPlan best{128, 256, 0};
  best.stages = 3;
  best.frag = 1;
  double best_t = 1e300;
  const int nk = K / 64;
  for (int vi = 0; vi < nvars; ++vi) {
    const Var& v = vars[vi];
    if (geglu && v.bn != 256) continue;
    // the five-wave 64 x 160 tile wins where the fixed cost dominates (measured up to
    // K = 2560); deeper contractions (FF-out, K = 5120) run faster as split 128 x 256 tiles
    if (v.bm == 64 && v.bn == 160 && K > 2560) continue;
    const long long tiles = (long long)ceil_div(M, v.bm) * ceil_div(N, v.bn);
    for (int sp = 1; sp <= kMaxSplit; ++sp) {
      // the five-wave tiles (one workgroup per CU) were measured unsplit only
      if (sp > 1 && (geglu || !allow_split || nk / sp < 4 || v.wg == 1)) break;
      const long long units = tiles * sp;
      const long long slots = (long long)cus * v.wg;
      const long long rounds = (units + slots - 1) / slots;
      const double load = (double)std::min(units, slots) / cus;
      const double per_cu = std::max(1.0, load) + fill_penalty * (std::ceil(load) - load);
      double t = rounds * (per_cu * 2.0 * v.bm * v.bn * ((double)K / sp) / v.rate + v.fixed) + v.epi * M * N / 1e6;
      if (sp > 1) t += fused_reduce ? 0.3 * (sp - 1.0) * M * N * 4.0 / 1e6 : 0.1 * (sp + 1.0) * M * N * 4.0 / 1e6 + 2.0;
      if (t < best_t) {
        best_t = t;
        best.bm = v.bm;
        best.bn = v.bn;
        best.split = sp;
      }
    }
  }
  // 128 x 160 tiles run on four waves, two workgroups per CU (the five-wave tile leaves
  // one SIMD with two waves' work and one workgroup per CU) for every convolution
  // (measured: 32768-row convolutions 17 % faster, the 8192-row upsampling convolution
  // from 1280 channels 373 -> 268 us, the other 8192-row ones equal or up to 6 % faster)
  // and for linear layers with more tiles than CUs; with one tile per CU the linear
  // layers run as fast or faster on five waves
  if (best.bm == 128 && best.bn == 160 &&
      (conv || (long long)ceil_div(M, 128) * ceil_div(N, 160) * best.split > cus))
    best.stages = 5;
  // 128 x 256 linear tiles (two workgroups per CU) whose count leaves a last round at most
  // half full: those last whole column bands run as 64-row tiles over every CU
  if (!conv && best.bm == 128 && best.bn == 256 && best.split == 1) {
    const long long mt = ceil_div(M, 128), nt = ceil_div(N, 256), slots = 2LL * cus;
    const long long tiles = mt * nt, rem = tiles % slots;
    if (rem > 0 && 2 * rem <= slots && rem % mt == 0) {
      const long long bands = rem / mt, tail = (long long)ceil_div(M, 64) * bands;
      if ((tiles - rem) % 8 == 0 && tail % 8 == 0 && bands < nt) best.tail_bands = static_cast<int>(bands);
    }
  }
  return best;
}

template <typename T>
GemmPlan gemm_plan(int M, int N, int K, int geglu, int cus, bool allow_split, bool fused_reduce, bool conv) {
  if (sizeof(T) == 2 && gemm_frag_layout(N, K)) return frag_plan(M, N, K, geglu, cus, allow_split, fused_reduce, conv);
  const long long t128 = (long long)ceil_div(M, 128) * ceil_div(N, 128);
  if (!geglu && t128 < cus) return GemmPlan{64, 64, 0};
  return GemmPlan{128, 128, 0};
}

template <typename T> void gemm(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  constexpr int BK = gemm_bk<T>();
  DN_CHECK(p.M >= 1 && p.N >= 1 && p.K >= BK, "gemm: empty or too small problem");
  DN_CHECK(p.K % BK == 0, "gemm: K must be a multiple of the K tile");
  DN_CHECK(p.taps == 1 || p.taps == 9, "gemm: taps must be 1 or 9");
  DN_CHECK(p.K == p.taps * (p.c0 + p.c1), "gemm: K != taps * channels");
  DN_CHECK(p.c1 == 0 || p.c0 % BK == 0, "gemm: concatenation split must be a multiple of the K tile");
  DN_CHECK(p.taps == 1 || (p.c0 + p.c1) % BK == 0, "gemm: conv channels must be a multiple of the K tile");
  DN_CHECK(p.a0 && p.b && p.out && (p.c1 == 0 || p.a1), "gemm: null operand");
  DN_CHECK(!p.geglu || (p.N % 64 == 0), "gemm: GEGLU needs N % 64 == 0");
  DN_CHECK(!p.geglu || (g.bn / 2) % 64 == 0,
           "gemm: GEGLU needs 64-column value/gate pairs per wave");
  DN_CHECK(p.ldb % (16 / (int)sizeof(T)) == 0 && p.lda0 % (16 / (int)sizeof(T)) == 0 &&
               (p.c1 == 0 || p.lda1 % (16 / (int)sizeof(T)) == 0),
           "gemm: leading dimensions must be multiples of 16 bytes");
  if (g.frag) {
    DN_CHECK(sizeof(T) == 2, "gemm: the fragment-B kernel is bf16 only");
    gemm_bf16_frag(p, g, s);
    return;
  }
  if (p.taps == 9)
    dispatch<T, true>(p, g, s);
  else
    dispatch<T, false>(p, g, s);
}

template GemmPlan gemm_plan<float>(int, int, int, int, int, bool, bool, bool);
template GemmPlan gemm_plan<bf16>(int, int, int, int, int, bool, bool, bool);
template void gemm<float>(const GemmParams&, const GemmPlan&, hipStream_t);
template void gemm<bf16>(const GemmParams&, const GemmPlan&, hipStream_t);

}  // namespace dn
