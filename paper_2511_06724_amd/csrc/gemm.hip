// MFMA GEMM with an implicit-convolution A loader (gfx950).
//
// One kernel template covers every dense contraction of the UNet: the 3x3
// convolutions (implicit GEMM over NHWC activations, with stride-2 downsample,
// nearest-x2 upsample addressing and two-source channel concatenation), the
// 1x1 skip convolutions and every linear layer of the transformer blocks
// (fused QKV, attention outputs, GEGLU feed-forward, projections).
//
// Tiling: 256 threads = 4 waves in a 2x2 grid; block tile BM x 128, wave tile
// (BM/2) x 64 built from 32x32 MFMA blocks; K step BK = 128 bytes of each row
// (64 bf16 / 32 fp32), staged through double-buffered LDS with one barrier per
// K step. Rows of A and B beyond M / N are clamped on load and masked on store.
#include "kernels.h"

namespace dn {
namespace {

constexpr int kThreads = 256;
constexpr int kBN = 128;

template <typename T> __device__ __forceinline__ void store_out(void* out, long long idx, float v, int f32) {
  if (f32)
    static_cast<float*>(out)[idx] = v;
  else
    static_cast<T*>(out)[idx] = from_f32<T>(v);
}

template <typename T> __device__ __forceinline__ float load_resid(const void* r, long long idx, int f32) {
  return f32 ? static_cast<const float*>(r)[idx] : to_f32(static_cast<const T*>(r)[idx]);
}

__device__ __forceinline__ float gelu_erf(float g) { return 0.5f * g * (1.0f + erff(g * 0.70710678118654752f)); }

template <typename T, int BM, bool CONV>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmParams p) {
  using MM = Mma<T>;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BK = gemm_bk<T>();
  constexpr int BN = kBN;
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

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int n0 = blockIdx.x * BN;
  const int m0 = blockIdx.y * BM;
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
      const int rem = m - s * opix;
      const int oy = rem / p.out_w;
      const int ox = rem - oy * p.out_w;
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

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = p.K / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  const int frag_off = (lane & 31) * SA + (lane >> 5) * MM::KPL;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tile((kt + 1) * BK);
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
        for (int j = 0; j < FN; ++j) acc[i][j] = MM::mma(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < nk) store_tile(cur ^ 1);
    __syncthreads();
  }

  // Epilogue.
  const int col = lane & 31;
  if (!p.geglu) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * WN + j * 32 + col;
      if (n >= p.n_store) continue;
      const float bn = p.bias ? p.bias[n] : 0.f;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + wm * WM + i * 32 + acc_row(r, lane);
          if (m >= p.M) continue;
          float v = acc[i][j][r] + bn;
          if (p.rowvec) v += p.rowvec[(long long)(m / p.rows_per_sample) * p.rowvec_ld + n];
          if (p.resid) v += load_resid<T>(p.resid, (long long)m * p.ldr + n, p.resid_f32);
          store_out<T>(p.out, (long long)m * p.ldo + n, v, p.out_f32);
        }
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < FN / 2; ++j) {
      const int nv = n0 + wn * WN + 2 * j * 32 + col;
      const int o = (n0 + wn * WN) / 2 + j * 32 + col;
      if (o >= p.n_store) continue;
      const float bv = p.bias ? p.bias[nv] : 0.f;
      const float bg = p.bias ? p.bias[nv + 32] : 0.f;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + wm * WM + i * 32 + acc_row(r, lane);
          if (m >= p.M) continue;
          const float v = (acc[i][2 * j][r] + bv) * gelu_erf(acc[i][2 * j + 1][r] + bg);
          store_out<T>(p.out, (long long)m * p.ldo + o, v, p.out_f32);
        }
      }
    }
  }
}

template <typename T, int BM, bool CONV> void launch(const GemmParams& p, hipStream_t s) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SA = gemm_bk<T>() + VEC;
  const size_t lds = size_t(2) * (BM + kBN) * SA * sizeof(T);
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<T, BM, CONV>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  dim3 grid(ceil_div(p.N, kBN), ceil_div(p.M, BM));
  hipLaunchKernelGGL((gemm_kernel<T, BM, CONV>), grid, dim3(kThreads), lds, s, p);
  DN_HIP(hipGetLastError());
}

}  // namespace

template <typename T> void gemm(const GemmParams& p, hipStream_t s) {
  constexpr int BK = gemm_bk<T>();
  DN_CHECK(p.M >= 1 && p.N >= 1 && p.K >= BK, "gemm: empty or too small problem");
  DN_CHECK(p.K % BK == 0, "gemm: K must be a multiple of the K tile");
  DN_CHECK(p.taps == 1 || p.taps == 9, "gemm: taps must be 1 or 9");
  DN_CHECK(p.K == p.taps * (p.c0 + p.c1), "gemm: K != taps * channels");
  DN_CHECK(p.c1 == 0 || p.c0 % BK == 0, "gemm: concatenation split must be a multiple of the K tile");
  DN_CHECK(p.taps == 1 || (p.c0 + p.c1) % BK == 0, "gemm: conv channels must be a multiple of the K tile");
  DN_CHECK(p.a0 && p.b && p.out && (p.c1 == 0 || p.a1), "gemm: null operand");
  DN_CHECK(!p.geglu || (p.N % 64 == 0), "gemm: GEGLU needs N % 64 == 0");
  DN_CHECK(p.ldb % (16 / (int)sizeof(T)) == 0 && p.lda0 % (16 / (int)sizeof(T)) == 0 &&
               (p.c1 == 0 || p.lda1 % (16 / (int)sizeof(T)) == 0),
           "gemm: leading dimensions must be multiples of 16 bytes");
  const long long t256 = (long long)ceil_div(p.M, 256) * ceil_div(p.N, kBN);
  const bool big = p.M >= 256 && t256 >= 512;
  if (p.taps == 9) {
    if (big)
      launch<T, 256, true>(p, s);
    else
      launch<T, 128, true>(p, s);
  } else {
    if (big)
      launch<T, 256, false>(p, s);
    else
      launch<T, 128, false>(p, s);
  }
}

template void gemm<float>(const GemmParams&, hipStream_t);
template void gemm<bf16>(const GemmParams&, hipStream_t);

}  // namespace dn
