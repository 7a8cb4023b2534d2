// bf16 MFMA GEMM / implicit-GEMM conv with direct-to-LDS loads (gfx950).
//
// Same contraction and epilogue as gemm.hip (see kernels.h), organised for
// the dense bf16 hot path:
//  - operands go global -> LDS with global_load_lds_dwordx4 (no VGPR staging,
//    no LDS store instructions); 4 LDS stages of BK = 32 keep three K steps of
//    loads in flight behind the one being multiplied;
//  - LDS rows are 64 bytes (4 chunks of 16 bytes) without padding; the chunk
//    order of row r is XOR-swizzled with f(r) = ((r >> 1) & 3) ^ ((r >> 3) & 1),
//    so the 16-byte fragment reads of 8 (or 16) consecutive rows hit distinct
//    banks. A DMA instruction writes 1 KB = 16 rows contiguously, lane L
//    filling chunk L & 3 of row L >> 2 from logical chunk (L & 3) ^ f(L >> 2);
//  - implicit-conv rows that fall in the zero padding read a 16-byte zero
//    block instead, so the LDS tile needs no second pass;
//  - MFMA 32x32x16 issued as C^T = B A^T (four consecutive output columns per
//    lane in the epilogue), XCD-aware tile order as in gemm.hip.
#include "gemm_epilogue.h"

namespace dn {
namespace {

constexpr int kXcds = 8;
constexpr int kBK = 32;        // bf16 elements per LDS row
constexpr int kRowBytes = 64;
constexpr int kStages = 4;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void gbl_void;

// s_waitcnt immediate: vmcnt <= vm (bits 3:0 and 15:14), lgkmcnt <= 0 (bits 11:8),
// expcnt unconstrained (bits 6:4 = 7).
constexpr int wait_vm_lgkm0(int vm) { return (vm & 0xF) | (((vm >> 4) & 3) << 14) | (7 << 4); }

__device__ __forceinline__ int swz(int row) { return ((row >> 1) & 3) ^ ((row >> 3) & 1); }


template <int BM, int BN, int WGM, int WGN, bool CONV>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_dma_kernel(GemmParams p, int mt, int nt) {
  constexpr int NW = WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int STAGE = (BM + BN) * kRowBytes;   // bytes per LDS stage
  constexpr int INSTR = (BM + BN) / 16;           // DMA instructions per stage
  constexpr int PER_WAVE = INSTR / NW;
  static_assert(INSTR % NW == 0, "DMA instructions must divide over the waves");
  static_assert(BM % 16 == 0 && BN % 16 == 0, "tile rows must be multiples of 16");

  extern __shared__ __align__(16) unsigned char smem[];

  // ---- tile assignment (XCD-aware: each XCD walks a contiguous band of columns)
  const int total = mt * nt;
  const int wg = blockIdx.x;
  const int xcd = wg % kXcds, idx = wg / kXcds;
  const int base = total / kXcds, rem = total % kXcds;
  const int logical = xcd * base + min(xcd, rem) + idx;
  const int n_tile = logical / mt;
  const int m_tile = logical - n_tile * mt;
  const int n0 = n_tile * BN, m0 = m_tile * BM;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WGN, wn = wave - (wave / WGN) * WGN;

  // ---- per-lane DMA sources: instruction j of this wave covers tile rows
  // [16 q, 16 q + 16), q = wave * PER_WAVE + j, over A's rows then B's rows.
  const int lrow = lane >> 2;
  const int lchunk = (lane & 3) ^ swz(lrow);  // logical 16-byte chunk this lane fetches
  const bf16* src_ptr[PER_WAVE];
  int src_is_a[PER_WAVE];
  int a_m[PER_WAVE];
  int c_sy[PER_WAVE], c_oy[PER_WAVE], c_ox[PER_WAVE];
  const int opix = p.out_h * p.out_w;
#pragma unroll
  for (int j = 0; j < PER_WAVE; ++j) {
    const int q = wave * PER_WAVE + j;
    const int row = 16 * q + lrow;
    if (row < BM) {
      src_is_a[j] = 1;
      const int m = min(m0 + row, p.M - 1);
      a_m[j] = m;
      if (CONV) {
        const int s = m / opix;
        const int r2 = m - s * opix;
        const int oy = r2 / p.out_w;
        c_sy[j] = s * p.in_h;
        c_oy[j] = oy * p.stride - 1;
        c_ox[j] = (r2 - oy * p.out_w) * p.stride - 1;
        src_ptr[j] = nullptr;
      } else {
        src_ptr[j] = static_cast<const bf16*>(p.a0) + (long long)m * p.lda0 + lchunk * 8;
      }
    } else {
      src_is_a[j] = 0;
      a_m[j] = 0;
      const int n = min(n0 + row - BM, p.N - 1);
      src_ptr[j] = static_cast<const bf16*>(p.b) + (long long)n * p.ldb + lchunk * 8;
    }
  }
  const int ct = p.c0 + p.c1;
  const int hl = p.in_h << p.up, wl = p.in_w << p.up;

  auto issue = [&](int kt, int slot) {
    const int k0 = kt * kBK;
    unsigned char* stage = smem + slot * STAGE;
    // A-side source for this K step (single source for linear rows handled via src_ptr)
    int tap = 0, c = k0;
    if (CONV) {
      tap = k0 / ct;
      c = k0 - tap * ct;
    }
    const bf16* a_src;
    int a_ld, a_c;
    if (c < p.c0) {
      a_src = static_cast<const bf16*>(p.a0);
      a_ld = p.lda0;
      a_c = c;
    } else {
      a_src = static_cast<const bf16*>(p.a1);
      a_ld = p.lda1;
      a_c = c - p.c0;
    }
    const int ky = tap / 3, kx = tap - 3 * (tap / 3);
#pragma unroll
    for (int j = 0; j < PER_WAVE; ++j) {
      const int q = wave * PER_WAVE + j;
      const void* g;
      if (src_is_a[j]) {
        if (CONV) {
          const int iy = c_oy[j] + ky, ix = c_ox[j] + kx;
          if (iy >= 0 && iy < hl && ix >= 0 && ix < wl) {
            const long long pix = (long long)(c_sy[j] + (iy >> p.up)) * p.in_w + (ix >> p.up);
            g = a_src + pix * a_ld + a_c + lchunk * 8;
          } else {
            g = p.zero16;
          }
        } else if (p.c1) {
          g = a_src + (long long)a_m[j] * a_ld + a_c + lchunk * 8;
        } else {
          g = src_ptr[j] + k0;
        }
      } else {
        g = src_ptr[j] + k0;
      }
      __builtin_amdgcn_global_load_lds((gbl_void*)g, (lds_void*)(stage + q * 1024), 16, 0, 0);
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Fragment offsets within a stage (bytes): row (lane % 32) of the block, logical
  // chunk 2 s + (lane / 32) for MFMA step s, swizzled by the row.
  const int frow = lane & 31;
  const int fs = swz(frow);
  const int h = lane >> 5;
  const int off_s0 = frow * kRowBytes + ((0 + h) ^ fs) * 16;
  const int off_s1 = frow * kRowBytes + ((2 + h) ^ fs) * 16;
  const int a_base = (wm * WM) * kRowBytes;
  const int b_base = (BM + wn * WN) * kRowBytes;

  const int nk = p.K / kBK;
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s)
    if (s < nk) issue(s, s);

  for (int kt = 0; kt < nk; ++kt) {
    // Tile kt has landed once at most the loads of the (up to kStages - 2) later tiles
    // are pending; lgkmcnt(0) retires this wave's fragment reads of the slot about
    // to be refilled. Then one barrier makes every wave's DMA visible.
    const int later = min(nk - 1 - kt, kStages - 2);
    if (later >= 2)
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(2 * PER_WAVE));
    else if (later == 1)
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(PER_WAVE));
    else
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
    __builtin_amdgcn_s_barrier();
    if (kt + kStages - 1 < nk) issue(kt + kStages - 1, (kt + kStages - 1) % kStages);

    const unsigned char* stage = smem + (kt % kStages) * STAGE;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int off = s ? off_s1 : off_s0;
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(stage + a_base + i * 32 * kRowBytes + off);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(stage + b_base + j * 32 * kRowBytes + off);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
    }
  }

  // ---- epilogue (lane = output row, 4 consecutive output columns per register group)
  const int col = lane & 31;
  const int h4 = 4 * (lane >> 5);
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
          epilogue_group<bf16>(p, m, n, v);
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
          const int nv = n0 + wn * WN + 2 * j * 32 + 8 * g + h4;
          const int o = (n0 + wn * WN) / 2 + j * 32 + 8 * g + h4;
          if (o >= p.n_store) continue;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float a = acc[i][2 * j][4 * g + e] + (p.bias ? p.bias[nv + e] : 0.f);
            const float gg = acc[i][2 * j + 1][4 * g + e] + (p.bias ? p.bias[nv + 32 + e] : 0.f);
            v[e] = a * gelu_erf(gg);
          }
          store4<bf16>(p, m, o, v, p.n_store);
        }
    }
  }
}

template <int BM, int BN, int WGM, int WGN, bool CONV> void launch_dma(const GemmParams& p, hipStream_t s) {
  const size_t lds = size_t(kStages) * (BM + BN) * kRowBytes;
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_dma_kernel<BM, BN, WGM, WGN, CONV>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  const int mt = ceil_div(p.M, BM), nt = ceil_div(p.N, BN);
  hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, WGN, CONV>), dim3(mt * nt), dim3(64 * WGM * WGN), lds, s, p, mt,
                     nt);
  DN_HIP(hipGetLastError());
}

template <bool CONV> void dispatch_dma(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  if (g.bm == 256 && g.bn == 256)
    launch_dma<256, 256, 2, 4, CONV>(p, s);
  else if (g.bm == 256 && g.bn == 128)
    launch_dma<256, 128, 2, 2, CONV>(p, s);
  else if (g.bm == 128 && g.bn == 256)
    launch_dma<128, 256, 2, 2, CONV>(p, s);
  else
    launch_dma<128, 128, 2, 2, CONV>(p, s);
}

}  // namespace

void gemm_bf16_dma(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  DN_CHECK(p.K % kBK == 0, "gemm: K must be a multiple of 32");
  DN_CHECK(p.taps == 1 || (p.c0 + p.c1) % kBK == 0, "gemm: conv channels must be a multiple of 32");
  DN_CHECK(p.c1 == 0 || p.c0 % kBK == 0, "gemm: concatenation split must be a multiple of 32");
  DN_CHECK(p.taps == 9 || p.c1 == 0 || p.lda0 > 0, "gemm: bad leading dimension");
  DN_CHECK(p.taps == 1 || p.zero16, "gemm: implicit conv needs the zero block");
  if (p.taps == 9)
    dispatch_dma<true>(p, g, s);
  else
    dispatch_dma<false>(p, g, s);
}

}  // namespace dn
