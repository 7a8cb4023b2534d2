// bf16 MFMA GEMM / implicit-GEMM conv with direct-to-LDS loads (gfx950).
//
// Same contraction and epilogue as gemm.hip (see kernels.h), organised for
// the dense bf16 hot path:
//  - operands go global -> LDS with global_load_lds_dwordx4 (no VGPR staging,
//    no LDS store instructions) into S LDS stages of BK = 64 (128-byte rows);
//    the loads of stage kt + S are issued as soon as every wave has finished
//    reading stage kt, so S - 1 later stages are in flight behind the one
//    being multiplied;
//  - each stage is consumed in four k-steps of 16; the MFMA fragments of
//    k-step s + 1 are read from LDS while the MFMAs of k-step s run (two
//    register sets), and the fragments of the next stage's first k-step are
//    read right after the stage barrier, before the last MFMAs of the current
//    stage, so the matrix cores need not wait for an LDS read latency;
//  - LDS rows hold 8 chunks of 16 bytes without padding; chunk c of row r is
//    stored at position c ^ f(r), f(r) = (r & 7) ^ ((r >> 3) & 1), so that the
//    fragment reads of 8 consecutive rows and of 16 consecutive rows (8 or 16
//    lanes served per LDS cycle) hit distinct banks. A DMA instruction writes
//    1 KB = 8 rows contiguously, lane L filling position L & 7 of row L >> 3
//    from logical chunk (L & 7) ^ f(row);
//  - implicit-conv rows that fall in the zero padding read a 16-byte zero
//    block instead, so the LDS tile needs no second pass;
//  - MFMA 32x32x16 issued as C^T = B A^T (four consecutive output columns per
//    lane in the epilogue), XCD-aware tile order as in gemm.hip.
#include <type_traits>

#include "gemm_epilogue.h"

namespace dn {
namespace {

constexpr int kXcds = 8;
constexpr int kBK = 64;         // bf16 elements per LDS row
constexpr int kRowBytes = 128;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void gbl_void;

// s_waitcnt immediate: vmcnt <= vm (bits 3:0 and 15:14), lgkmcnt <= 0 (bits 11:8),
// expcnt unconstrained (bits 6:4 = 7).
constexpr int wait_vm_lgkm0(int vm) { return (vm & 0xF) | (((vm >> 4) & 3) << 14) | (7 << 4); }

// Scheduling-group pattern of one k-step: MFMA i is followed by one LDS fragment read
// (while reads remain) and by its share of VM loads (NV spread over the NM MFMAs).
template <int I, int NM, int NR, int NV> struct KStepSched {
  __device__ static __forceinline__ void apply() {
    if constexpr (I < NM) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      if constexpr (I < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      constexpr int v = NV * (I + 1) / NM - NV * I / NM;
      if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);  // VM load
      KStepSched<I + 1, NM, NR, NV>::apply();
    } else {
      if constexpr (NR > NM) __builtin_amdgcn_sched_group_barrier(0x100, NR - NM, 0);
    }
  }
};

// MODE: 0 linear layer (one A source), 1 linear layer over two concatenated A sources,
// 2 implicit 3x3 convolution (one source).
template <int BM, int BN, int WGM, int WGN, int S, int MODE>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_dma_kernel(GemmParams p, int mt, int nt) {
  constexpr int NW = WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int STAGE = (BM + BN) * kRowBytes;   // bytes per LDS stage
  constexpr int INSTR = (BM + BN) / 8;            // DMA instructions per stage (8 rows each)
  constexpr int PW = INSTR / NW;                  // ... per wave
  static_assert(INSTR % NW == 0, "DMA instructions must divide over the waves");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert(S >= 2 && S <= 4, "2 to 4 stages");
  static_assert(PW * (S - 1) < 64, "vmcnt range");

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
  // [8 q, 8 q + 8), q = wave * PW + j, over A's rows then B's rows; the lane fetches
  // logical chunk (lane & 7) ^ f(row), f(row) = (lane >> 3) ^ (q & 1). Each row keeps
  // a 32-bit element offset at k = 0 (B rows and linear A rows: row * ld + chunk; conv
  // A rows: the input pixel of tap (0, 0), possibly outside the image, times lda +
  // chunk), so a stage adds one uniform offset per instruction. Conv rows also keep a
  // tap mask (bit 3 ky + kx: tap inside the input; bits 9 / 10: output row / column
  // parity, which picks the source pixel of the taps of a nearest-x2 upsampled input).
  const int lrow = lane >> 3;
  const int lc_even = ((lane & 7) ^ lrow) * 8, lc_odd = ((lane & 7) ^ lrow ^ 1) * 8;
  constexpr int QA = BM / 8;  // instructions q < QA load A rows
  int off0[PW];
  int off1[PW];  // MODE 1: offset into the second source; MODE 2: tap mask
  const int hl = p.in_h << p.up, wl = p.in_w << p.up;
#pragma unroll
  for (int j = 0; j < PW; ++j) {
    const int q = wave * PW + j;
    const int lc = (q & 1) ? lc_odd : lc_even;
    off1[j] = 0;
    if (q < QA) {
      const int m = min(m0 + 8 * q + lrow, p.M - 1);
      if (MODE == 2) {
        const int opix = p.out_h * p.out_w;
        const int smp = m / opix;
        const int r2 = m - smp * opix;
        const int oy = r2 / p.out_w, ox = r2 - (r2 / p.out_w) * p.out_w;
        const int iy0 = oy * p.stride - 1, ix0 = ox * p.stride - 1;  // tap (0, 0), upsampled coordinates
        int msk = 0;
#pragma unroll
        for (int t = 0; t < 9; ++t) {
          const int iy = iy0 + t / 3, ix = ix0 + t % 3;
          msk |= (iy >= 0 && iy < hl && ix >= 0 && ix < wl) ? (1 << t) : 0;
        }
        msk |= (oy & 1) << 9 | (ox & 1) << 10;
        const int pix = (smp * p.in_h + (iy0 >> p.up)) * p.in_w + (ix0 >> p.up);
        off0[j] = pix * p.lda0 + lc;
        off1[j] = msk;
      } else {
        off0[j] = m * p.lda0 + lc;
        if (MODE == 1) off1[j] = m * p.lda1 + lc;
      }
    } else {
      const int n = min(n0 + 8 * q + lrow - BM, p.N - 1);
      off0[j] = n * p.ldb + lc;
    }
  }
  const int ct = p.c0 + p.c1;
  const bf16* const gA0 = static_cast<const bf16*>(p.a0);
  const bf16* const gA1 = static_cast<const bf16*>(p.a1);
  const bf16* const gB = static_cast<const bf16*>(p.b);

  // DMA of stage kt into LDS slot `slot`: PW global_load_lds per wave, no branches
  // (uniform choices are selects). Stages past the last one (kt >= nk) read the 16-byte
  // zero block instead, so that every hand-over issues the same number of loads.
  const int nk = p.K / kBK;
  auto issue = [&](int kt_in, int slot) {
    const bool real = kt_in < nk;
    const int kt = real ? kt_in : nk - 1;
    const int k0 = kt * kBK;
    unsigned char* stage = smem + slot * STAGE;
    // uniform per stage: A source, its element offset, tap
    int tap = 0, c = k0;
    if (MODE == 2) {
      tap = k0 / ct;
      c = k0 - tap * ct;
    }
    const int ky = tap / 3, kx = tap - 3 * (tap / 3);
    const bool second = MODE == 1 && c >= p.c0;
    const bf16* a_src = second ? gA1 : gA0;
    const int a_c = second ? c - p.c0 : c;
    // conv, input at original resolution: tap (ky, kx) adds (ky * in_w + kx) pixels
    const int tap_off = (MODE == 2 && !p.up) ? (ky * p.in_w + kx) * p.lda0 : 0;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int q = wave * PW + j;
      const bf16* g;
      if (q < QA) {
        if (MODE == 2) {
          int off = off0[j] + a_c + tap_off;
          if (p.up) {
            // nearest-x2 input: the source row advances by one for ky = 2, and for ky = 1
            // when the output row is even (likewise for columns)
            const int dy = ky == 2 || (ky == 1 && !(off1[j] & (1 << 9)));
            const int dx = kx == 2 || (kx == 1 && !(off1[j] & (1 << 10)));
            off += (dy ? p.in_w * p.lda0 : 0) + (dx ? p.lda0 : 0);
          }
          const bool inb = (off1[j] >> tap) & 1;
          g = inb ? a_src + off : static_cast<const bf16*>(p.zero16);
        } else {
          g = a_src + ((MODE == 1 && second) ? off1[j] : off0[j]) + a_c;
        }
      } else {
        g = gB + (off0[j] + k0);
      }
      if (!real) g = static_cast<const bf16*>(p.zero16);
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

  // Fragment offsets within a stage (bytes): row (lane % 32) of a 32-row block,
  // logical chunk 2 s + (lane / 32) for k-step s, at its swizzled position.
  const int frow = lane & 31;
  const int fs = (lane & 7) ^ ((lane >> 3) & 1);
  const int h = lane >> 5;
  const int a_base = (wm * WM + frow) * kRowBytes;
  const int b_base = (BM + wn * WN + frow) * kRowBytes;

  bf16x8 fa[2][FM], fb[2][FN];
  auto read_frags = [&](const unsigned char* stage, int s, bf16x8* a, bf16x8* b) {
    const int off = ((2 * s + h) ^ fs) * 16;
#pragma unroll
    for (int i = 0; i < FM; ++i)
      a[i] = *reinterpret_cast<const bf16x8*>(stage + a_base + i * 32 * kRowBytes + off);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      b[j] = *reinterpret_cast<const bf16x8*>(stage + b_base + j * 32 * kRowBytes + off);
  };
  auto mfmas = [&](const bf16x8* a, const bf16x8* b) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
  };

  // One LDS stage: four k-steps, the fragments of k-step s + 1 read while the MFMAs of
  // k-step s issue (one LDS read after each MFMA, pinned with scheduling groups). Unless
  // `last`, the stage ends with the hand-over to stage kt + 1: stage kt + 1 has landed
  // once at most the stages after it are pending, and this wave's reads of stage kt are
  // complete (lgkmcnt 0); after the barrier every wave is done with slot kt % S, which
  // takes stage kt + S, and the first fragments of stage kt + 1 are read while the last
  // MFMAs of stage kt issue.
  constexpr int NR = FM + FN, NM = FM * FN;
  // k-step: fragment reads for the next k-step and MFMAs of this one, one read after
  // each MFMA; with `dma`, the loads of a later stage are spread over the MFMAs too.
  auto step = [&](const unsigned char* next_stage, int next_s, const bf16x8* a, const bf16x8* b, bf16x8* na,
                  bf16x8* nb, auto dma, int dma_kt, int dma_slot) {
    if constexpr (decltype(dma)::value) issue(dma_kt, dma_slot);
    read_frags(next_stage, next_s, na, nb);
    mfmas(a, b);
    KStepSched<0, NM, NR, decltype(dma)::value ? PW : 0>::apply();
    __builtin_amdgcn_sched_barrier(0);
  };
  auto run_stage = [&](int kt, int rd, int nx, bool last) {
    const unsigned char* stage = smem + rd * STAGE;
    step(stage, 1, fa[0], fb[0], fa[1], fb[1], std::false_type{}, 0, 0);
    step(stage, 2, fa[1], fb[1], fa[0], fb[0], std::false_type{}, 0, 0);
    step(stage, 3, fa[0], fb[0], fa[1], fb[1], std::false_type{}, 0, 0);
    if (!last) {
      // stage kt + 1 has landed once at most the S - 2 stages issued after it are pending
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0((S - 2) * PW));
      __builtin_amdgcn_s_barrier();
      // after the barrier every wave is done with slot rd: stage kt + S goes there
      step(smem + nx * STAGE, 0, fa[1], fb[1], fa[0], fb[0], std::true_type{}, kt + S, rd);
    } else {
      mfmas(fa[1], fb[1]);
    }
  };

#pragma unroll
  for (int s = 0; s < S; ++s) issue(s, s);
  __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0((S - 1) * PW));
  __builtin_amdgcn_s_barrier();
  read_frags(smem, 0, fa[0], fb[0]);
  int rd = 0;
  for (int kt = 0; kt < nk - 1; ++kt) {
    const int nx = rd + 1 == S ? 0 : rd + 1;
    run_stage(kt, rd, nx, false);
    rd = nx;
  }
  run_stage(nk - 1, rd, rd, true);
  __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));  // the zero-block loads of the tail stages

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

template <int BM, int BN, int WGM, int WGN, int S, int MODE> void launch_dma(const GemmParams& p, hipStream_t s) {
  const size_t lds = size_t(S) * (BM + BN) * kRowBytes;
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_dma_kernel<BM, BN, WGM, WGN, S, MODE>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  const int mt = ceil_div(p.M, BM), nt = ceil_div(p.N, BN);
  hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WGM, WGN, S, MODE>), dim3(mt * nt), dim3(64 * WGM * WGN), lds, s,
                     p, mt, nt);
  DN_HIP(hipGetLastError());
}

#define DN_DMA_CASE(BM_, BN_, WGM_, WGN_, S_)                                           \
  if (g.bm == BM_ && g.bn == BN_ && g.wgm == WGM_ && g.wgn == WGN_ && g.stages == S_) { \
    launch_dma<BM_, BN_, WGM_, WGN_, S_, MODE>(p, s);                                   \
    return;                                                                             \
  }

template <int MODE> void dispatch_dma(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  DN_DMA_CASE(256, 256, 2, 4, 2)
  DN_DMA_CASE(256, 320, 4, 2, 2)
  DN_DMA_CASE(128, 320, 2, 2, 2)
  DN_DMA_CASE(128, 320, 2, 2, 3)
  DN_DMA_CASE(256, 160, 4, 1, 2)
  DN_DMA_CASE(256, 160, 4, 1, 3)
  DN_DMA_CASE(256, 128, 4, 2, 2)
  DN_DMA_CASE(256, 128, 4, 2, 3)
  DN_DMA_CASE(128, 256, 2, 4, 2)
  DN_DMA_CASE(128, 256, 2, 4, 3)
  DN_DMA_CASE(128, 128, 2, 2, 2)
  DN_DMA_CASE(128, 128, 2, 2, 3)
  DN_DMA_CASE(128, 128, 2, 2, 4)
  DN_DMA_CASE(128, 64, 2, 2, 3)
  DN_DMA_CASE(64, 128, 2, 2, 3)
  DN_DMA_CASE(64, 64, 2, 2, 2)
  DN_DMA_CASE(64, 64, 2, 2, 3)
  DN_DMA_CASE(64, 64, 2, 2, 4)
  throw Error(-1, "gemm: no direct-to-LDS kernel for this tile plan");
}
#undef DN_DMA_CASE

}  // namespace

void gemm_bf16_dma(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  DN_CHECK(p.K % kBK == 0, "gemm: K must be a multiple of 64");
  DN_CHECK(p.taps == 1 || (p.c0 + p.c1) % kBK == 0, "gemm: conv channels must be a multiple of 64");
  DN_CHECK(p.c1 == 0 || p.c0 % kBK == 0, "gemm: concatenation split must be a multiple of 64");
  DN_CHECK(p.taps == 9 || p.c1 == 0 || p.lda0 > 0, "gemm: bad leading dimension");
  DN_CHECK(p.taps == 1 || p.zero16, "gemm: implicit conv needs the zero block");
  DN_CHECK(p.taps == 1 || p.c1 == 0, "gemm: the direct-to-LDS conv takes one input source");
  if (p.taps == 9)
    dispatch_dma<2>(p, g, s);
  else if (p.c1)
    dispatch_dma<1>(p, g, s);
  else
    dispatch_dma<0>(p, g, s);
}

}  // namespace dn
