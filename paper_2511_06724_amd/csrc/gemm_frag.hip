// bf16 GEMM / implicit-GEMM conv with fragment-ordered weights (gfx950).
//
// Same contraction and epilogue as gemm.hip (see kernels.h), organised for the
// dense bf16 hot path:
//  - B, the packed weight matrix, is stored in MFMA fragment order (to_frag, below):
//    for each block of 32 output columns and each k-step of 16, the 64 lanes' 16-byte
//    operands lie in 1 KB of contiguous memory. Each wave loads its own B fragments
//    with one coalesced 16-byte load per lane straight into registers, one to three LDS
//    stages ahead, so B costs no LDS bandwidth (as far ahead as the A stages where the
//    registers allow: the compiler, which does not see the A loads, waits for a B
//    register by counting B loads only, so each such wait also retires the oldest A
//    loads issued after that B load);
//  - A (the activations, or the implicit-convolution gather) goes global -> LDS with
//    global_load_lds_dwordx4 into S stages of BK = 64 (128-byte rows, chunk c of row r
//    at position c ^ f(r), f(r) = (r & 7) ^ ((r >> 3) & 1)), shared by the waves (four
//    issue the loads);
//  - block tile BM x NW * 32 FN: the NW (4 or 5) waves split the columns, each computes
//    BM x 32 FN with 32x32x16 MFMAs issued as C^T = B A^T (four consecutive output
//    columns per lane). The 160-column tiles take four waves (X5): wave w owns column
//    block w and computes column block 4 over k-step w of every stage, so the four SIMDs
//    carry equal work; the four partial sums of block 4 meet in LDS in wave order;
//  - every k-step interleaves one MFMA, one LDS fragment read for the next k-step and
//    its share of B loads (scheduling groups); the stage hand-over (wait + barrier)
//    sits before the last k-step, whose MFMAs cover the first reads of the next stage;
//  - split-K: the units (tile, split) cover contiguous K ranges and write fp32 partial
//    tiles; a second kernel sums the slabs in split order (deterministic) and applies
//    the epilogue;
//  - epilogue through LDS: each wave writes its accumulators to LDS and reads them back
//    row-contiguous, so bias / residual loads and output stores are whole row segments
//    of 64-256 bytes instead of 16-byte pieces of 32 different rows. The per-head V^T
//    columns keep the register layout, where consecutive lanes are consecutive tokens.
//  - tiles go to XCDs in contiguous ranges (workgroup ids are dealt round-robin over the
//    8 XCDs), ordered by column band, split, then row tile, so that the units sharing a
//    band of B run on one XCD and share its L2;
//  - a 128 x 256 grid whose last round would be at most half full runs its last column
//    bands as 64-row tiles in the same launch (a wrapper decodes full and tail units), so
//    that the fraction of a round spreads over every CU.
#include <algorithm>
#include <type_traits>

#include "gemm_epilogue.h"

namespace dn {
namespace {

constexpr int kXcds = 8;
constexpr int kBK = 64;
constexpr int kRowBytes = 128;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void gbl_void;

// s_waitcnt immediate: vmcnt <= vm (bits 3:0 and 15:14), lgkmcnt <= 0 (bits 11:8),
// expcnt unconstrained (bits 6:4 = 7).
constexpr int wait_vm_lgkm0(int vm) { return (vm & 0xF) | (((vm >> 4) & 3) << 14) | (7 << 4); }

// 16 bytes per lane global -> LDS (lane i writes lds + 16 i). Issued from inline
// assembly: the compiler's wait insertion treats a global_load_lds it knows about as
// making the vector-memory counter out of order and then drains every load
// (vmcnt(0)) before the next use of any loaded register, which would serialise the
// B-register prefetch with every A stage. The LDS data this writes is guarded by the
// kernel's own waits and barriers (hand-overs, and a full drain before the epilogue);
// it writes no VGPRs. M0 holds the LDS address; nothing else in these kernels keeps a
// value in M0.
__device__ __forceinline__ void dma16(const void* g, lds_void* lds) {
  const unsigned a = static_cast<unsigned>(reinterpret_cast<__UINTPTR_TYPE__>(lds));
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(a) : "memory", "m0");
}

// Scheduling-group pattern of one k-step: NM MFMAs, each followed by one LDS read
// (while the NR reads last) and by its share of the NV B loads.
template <int I, int NM, int NR, int NV> struct KSched {
  __device__ static __forceinline__ void apply() {
    if constexpr (I < NM) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      if constexpr (I < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
      constexpr int v = NV * (I + 1) / NM - NV * I / NM;
      if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);  // VM load
      KSched<I + 1, NM, NR, NV>::apply();
    }
  }
};

// Epilogue inputs and outputs of 8 consecutive columns [n, n + 8) of row m (n % 8 == 0).
// The 16-byte forms need the whole group inside n_store, a leading dimension that keeps
// every row's group 16-byte aligned and a 16-byte aligned base; otherwise element-wise,
// with zeros (loads) or nothing (stores) past n_store.
__device__ __forceinline__ bool aligned16(const void* q) {
  return (reinterpret_cast<__UINTPTR_TYPE__>(q) & 15) == 0;
}
__device__ __forceinline__ bool resid_vec8(const GemmParams& p) {
  return aligned16(p.resid) && (p.ldr & (p.resid_f32 ? 3 : 7)) == 0;
}
__device__ __forceinline__ bool out_vec8(const GemmParams& p) {
  return aligned16(p.out) && (p.ldo & (p.out_f32 ? 3 : 7)) == 0;
}
__device__ __forceinline__ void load_rowvec8(const GemmParams& p, int m, int n, float v[8]) {
  const float* r = p.rowvec + (long long)(m / p.rows_per_sample) * p.rowvec_ld + n;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = n + e < p.n_store ? r[e] : 0.f;
}
__device__ __forceinline__ void load_resid8(const GemmParams& p, int m, int n, bool vec, float v[8]) {
  const long long ro = (long long)m * p.ldr + n;
  if (vec) {
    if (p.resid_f32) {
      const f32x4* r = reinterpret_cast<const f32x4*>(static_cast<const float*>(p.resid) + ro);
      const f32x4 a = r[0], b = r[1];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = a[e];
        v[e + 4] = b[e];
      }
    } else {
      const bf16x8 r = *reinterpret_cast<const bf16x8*>(static_cast<const bf16*>(p.resid) + ro);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = static_cast<float>(r[e]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      v[e] = n + e >= p.n_store ? 0.f
             : p.resid_f32      ? static_cast<const float*>(p.resid)[ro + e]
                                : static_cast<float>(static_cast<const bf16*>(p.resid)[ro + e]);
  }
}
__device__ __forceinline__ void store8(const GemmParams& p, int m, int n, const float v[8], bool vec) {
  const long long o = (long long)m * p.ldo + n;
  if (vec) {
    if (p.out_f32) {
      f32x4* d = reinterpret_cast<f32x4*>(static_cast<float*>(p.out) + o);
      d[0] = f32x4{v[0], v[1], v[2], v[3]};
      d[1] = f32x4{v[4], v[5], v[6], v[7]};
    } else {
      bf16x8 w;
#pragma unroll
      for (int e = 0; e < 8; ++e) w[e] = static_cast<bf16>(v[e]);
      *reinterpret_cast<bf16x8*>(static_cast<bf16*>(p.out) + o) = w;
    }
  } else {
    store4<bf16>(p, m, n, v, p.n_store);
    store4<bf16>(p, m, n + 4, v + 4, p.n_store);
  }
}

template <int BM, int FN, int S, int NW, bool X5 = false> constexpr size_t frag_lds_bytes() {
  constexpr size_t stages = size_t(S) * BM * kRowBytes;
  constexpr size_t epi = size_t(NW) * 32 * (32 * FN + 4) * 4;
  constexpr size_t part5 = X5 ? size_t(4) * (BM / 32) * 16 * 64 * 4 : 0;  // block-4 partial sums
  constexpr size_t m1 = stages > epi ? stages : epi;
  return m1 > part5 ? m1 : part5;
}

// MODE: 0 linear layer (one A source), 1 linear layer over two concatenated A sources,
// 2 implicit 3x3 convolution (one source). SPLIT: write fp32 partial tiles.
// D: B register buffers (B is loaded D stages ahead). WPE: waves per SIMD the register
// allocation must allow (2: two workgroups share a CU, so one's prologue, barriers and
// epilogue overlap the other's MFMAs). PRE: read a whole LDS stage of A fragments one
// stage ahead into registers (small tiles, whose few MFMAs per k-step cannot cover an
// LDS read latency), instead of one k-step ahead. NW: waves per workgroup, each owning
// 32 FN columns; with five (a 160-column tile) the first four issue the A DMA. X5: the
// 160-column tile on four waves (see the file comment).
// One unit: the BM x BN tile at (m0, n0) over the K stages [kt0, kt1) (split-K part
// `split` when SPLIT).
template <int BM, int FN, int S, int D, int WPE, int MODE, bool SPLIT, int PRE, int NW, bool X5>
__device__ __forceinline__ void frag_tile(const GemmParams& p, const int m0, const int n0, const int split,
                                          const int kt0, const int kt1) {
  constexpr int FM = BM / 32;
  constexpr int WN = 32 * FN;
  constexpr int BN = X5 ? 160 : NW * WN;
  static_assert(!X5 || (NW == 4 && FN == 1 && !PRE), "X5: four waves of one column block each");
  constexpr int NB = 4 * FN + (X5 ? 1 : 0);  // B loads per wave and stage
  constexpr int STAGE = BM * kRowBytes;
  constexpr int PW = BM / 32;  // DMA instructions (8 rows of 128 B) per DMA wave per stage
  static_assert(NW == 4 || NW == 5, "four or five waves");
  constexpr int NM = FM * FN;
  static_assert(D >= 1 && D <= 3 && (!PRE || D <= 2), "one to three B buffers (two with read-ahead)");
  static_assert(S >= 2 && S <= 6, "2 to 6 LDS stages");
  static_assert(BM % 32 == 0 && BM <= 256, "BM");

  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  // ---- A rows: instruction j of this wave loads tile rows [8 q, 8 q + 8), q = wave * PW + j;
  // the lane fetches logical chunk (lane & 7) ^ f(row) of row 8 q + (lane >> 3). Each row
  // keeps a 32-bit element offset at k = 0 (linear: row * lda; conv: the input pixel of tap
  // (0, 0), possibly outside the image, times lda) and, for conv, a tap mask (bit 3 ky + kx:
  // tap inside the input; bits 9 / 10: output row / column parity, which picks the source
  // pixel of the taps of a nearest-x2 upsampled input); MODE 1 keeps the second source's
  // offset instead.
  const int lrow = lane >> 3;
  const int lc_even = ((lane & 7) ^ lrow) * 8, lc_odd = ((lane & 7) ^ lrow ^ 1) * 8;
  int off0[PW];
  int off1[PW];
  const int hl = p.in_h << p.up, wl = p.in_w << p.up;
#pragma unroll
  for (int j = 0; j < PW; ++j) {
    const int q = wave * PW + j;
    const int lc = (q & 1) ? lc_odd : lc_even;
    const int m = min(m0 + 8 * q + lrow, p.M - 1);
    off1[j] = 0;
    if (MODE == 2) {
      const int opix = p.out_h * p.out_w;
      const int smp = m / opix;
      const int r2 = m - smp * opix;
      const int oy = r2 / p.out_w, ox = r2 - (r2 / p.out_w) * p.out_w;
      const int iy0 = oy * p.stride - 1, ix0 = ox * p.stride - 1;
      int mk = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int iy = iy0 + t / 3, ix = ix0 + t % 3;
        mk |= (iy >= 0 && iy < hl && ix >= 0 && ix < wl) ? (1 << t) : 0;
      }
      mk |= (oy & 1) << 9 | (ox & 1) << 10;
      const int pix = (smp * p.in_h + (iy0 >> p.up)) * p.in_w + (ix0 >> p.up);
      off0[j] = pix * p.lda0 + lc;
      off1[j] = mk;
    } else {
      off0[j] = m * p.lda0 + lc;
      if (MODE == 1) off1[j] = m * p.lda1 + lc;
    }
  }
  const int ct = p.c0 + p.c1;
  const bf16* const gA0 = static_cast<const bf16*>(p.a0);
  const bf16* const gA1 = static_cast<const bf16*>(p.a1);

  // DMA of A stage kt into LDS slot `slot`: PW global_load_lds per DMA wave, no branches
  // (a fifth wave issues none).
  // Stages past this unit's range read the 16-byte zero block instead, so every
  // hand-over issues the same number of loads.
  auto issue_a = [&](int kt_in, int slot) {
    const bool real = kt_in < kt1;
    const int kt = real ? kt_in : kt1 - 1;
    const int k0 = kt * kBK;
    unsigned char* stage = smem + slot * STAGE;
    int tap = 0, c = k0;
    if (MODE == 2) {
      tap = k0 / ct;
      c = k0 - tap * ct;
    }
    const int ky = tap / 3, kx = tap - 3 * (tap / 3);
    const bool second = MODE == 1 && c >= p.c0;
    const bf16* a_src = second ? gA1 : gA0;
    const int a_c = second ? c - p.c0 : c;
    const int tap_off = (MODE == 2 && !p.up) ? (ky * p.in_w + kx) * p.lda0 : 0;
    if (NW > 4 && wave >= 4) return;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int q = wave * PW + j;
      const bf16* g;
      if (MODE == 2) {
        int off = off0[j] + a_c + tap_off;
        if (p.up) {
          const int dy = ky == 2 || (ky == 1 && !(off1[j] & (1 << 9)));
          const int dx = kx == 2 || (kx == 1 && !(off1[j] & (1 << 10)));
          off += (dy ? p.in_w * p.lda0 : 0) + (dx ? p.lda0 : 0);
        }
        const bool inb = (off1[j] >> tap) & 1;
        g = inb ? a_src + off : static_cast<const bf16*>(p.zero16);
      } else {
        g = a_src + ((MODE == 1 && second) ? off1[j] : off0[j]) + a_c;
      }
      if (!real) g = static_cast<const bf16*>(p.zero16);
      dma16(g, (lds_void*)(stage + q * 1024));
    }
  };

  // ---- B fragments of this wave: column blocks nb = (n0 + wave * WN) / 32 + j, clamped
  // to the packed rows (columns past N are computed and dropped by the epilogue).
  const int kbs = p.K / 16;
  const int nb_last = (p.N + 31) / 32 - 1;
  const bf16* bptr[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int nb = min((n0 + wave * WN) / 32 + j, nb_last);
    bptr[j] = static_cast<const bf16*>(p.b) + (long long)nb * kbs * 512 + lane * 8;
  }
  typedef bf16x8 BReg[4][FN];
  auto load_b_step = [&](int kt_in, int s, BReg& dst) {
    const int kt = kt_in < kt1 ? kt_in : kt1 - 1;
#pragma unroll
    for (int j = 0; j < FN; ++j) dst[s][j] = *reinterpret_cast<const bf16x8*>(bptr[j] + (kt * 4 + s) * 512);
  };
  // X5: the fragment of column block 4 for k-step `wave` of a stage
  const bf16* const bptr5 =
      static_cast<const bf16*>(p.b) + (long long)min(n0 / 32 + 4, nb_last) * kbs * 512 + lane * 8 + wave * 512;
  auto load_b5 = [&](int kt_in, bf16x8& dst) {
    const int kt = kt_in < kt1 ? kt_in : kt1 - 1;
    dst = *reinterpret_cast<const bf16x8*>(bptr5 + kt * 4 * 512);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  f32x16 acc5[X5 ? FM : 1];
#pragma unroll
  for (int i = 0; i < (X5 ? FM : 1); ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc5[i][r] = 0.f;

  // Epilogue input of the plain path (the residual or the per-sample row vector, when
  // exactly one is present) for small wave tiles of the linear modes without stage
  // read-ahead (where the registers are free): loaded into FM x ENP x 2 16-byte registers
  // per lane, in the layout of the row-contiguous epilogue (8 consecutive columns per
  // lane). The loads are issued right after the prologue's A and B loads, so the first
  // wait (in-order vector-memory counter) does not include them and the main loop's
  // latency hides them.
  constexpr int ELPR = WN / 8;     // lanes per row in the row-contiguous epilogue
  constexpr int ERPI = 64 / ELPR;  // rows per pass
  constexpr int ENP = 32 / ERPI;   // passes per 32-row block
  constexpr bool kPreIn = !SPLIT && !PRE && MODE != 2 && FM * ENP * 8 <= 32 && WPE <= 2;
  const int enw0 = n0 + wave * WN;
  const bool pre_in = kPreIn && !p.geglu && !(p.vt && enw0 + WN > p.vt_col0) &&
                      ((p.resid != nullptr) != (p.rowvec != nullptr));
  f32x4 pin[kPreIn ? FM : 1][kPreIn ? ENP : 1][2];
  auto load_pre_in = [&]() {
    if constexpr (kPreIn) {
      if (pre_in) {
        const int n = enw0 + (lane % ELPR) * 8;
        const bool rvec = n + 8 <= p.n_store && p.resid && resid_vec8(p);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int t = 0; t < ENP; ++t) {
            const int m = m0 + i * 32 + t * ERPI + lane / ELPR;
            float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            if (m < p.M && n < p.n_store) {
              if (p.rowvec)
                load_rowvec8(p, m, n, v);
              else
                load_resid8(p, m, n, rvec, v);
            }
            pin[i][t][0] = f32x4{v[0], v[1], v[2], v[3]};
            pin[i][t][1] = f32x4{v[4], v[5], v[6], v[7]};
          }
      }
    }
  };

  // A fragment of k-step s: row (lane % 32) of each 32-row block, logical chunk
  // 2 s + (lane / 32) at its swizzled position.
  const int frow = lane & 31;
  const int fs = (lane & 7) ^ ((lane >> 3) & 1);
  const int hh = lane >> 5;
  bf16x8 fa[2][FM];
  auto read_a = [&](int slot, int s, bf16x8* a) {
    const unsigned char* st = smem + slot * STAGE + frow * kRowBytes + (((2 * s + hh) ^ fs) * 16);
#pragma unroll
    for (int i = 0; i < FM; ++i) a[i] = *reinterpret_cast<const bf16x8*>(st + i * 32 * kRowBytes);
  };
  auto mfmas = [&](const bf16x8* a, const bf16x8* b) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
  };
  bf16x8 a5[X5 ? FM : 1];
  auto mfmas5 = [&](const bf16x8& b) {
#pragma unroll
    for (int i = 0; i < FM; ++i) acc5[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a5[i], acc5[i], 0, 0, 0);
  };

  BReg bq[D];
  if constexpr (PRE) {
    // Stage kt: hand-over first (this wave's DMA of stage kt + 1 landed: at most VM_PRE
    // later VM loads pending; after the barrier every wave's has, and every wave is done
    // with the slot of stage kt - 1, whose fragments it read a stage earlier and used),
    // then the DMA of stage kt + S - 1 into that slot, the reads of all of stage kt + 1's
    // fragments into the other register set, and stage kt's MFMAs from registers with the
    // B loads of stage kt + D as B registers free up.
    // VM loads after the DMA of stage kt + 1 (issued at the start of stage kt + 2 - S):
    // 4 FN B loads of that stage, then S - 3 stages of PW DMA + 4 FN B loads. When that DMA
    // came from the prologue (kt = kt0 + r, r <= S - 2; stage kt0 issues no DMA) the count
    // is (S - 3) PW + 4 D FN + 4 r FN, enough once D + r >= S - 2; r = 0 is the prologue wait.
    static_assert(S == 3 || (S == 4 && D >= 1), "stage read-ahead: 3 or 4 LDS stages");
    constexpr int VM_PRE = 4 * FN + (S - 3) * (PW + 4 * FN);
    static_assert(VM_PRE < 64 && (S - 2) * PW + D * 4 * FN < 64, "vmcnt range");
    typedef bf16x8 AStage[4][FM];
    AStage sa[2];
    auto read_stage = [&](int slot, AStage& dst) {
#pragma unroll
      for (int s = 0; s < 4; ++s) read_a(slot, s, dst[s]);
    };
#pragma unroll
    for (int s = 0; s < S; ++s) issue_a(kt0 + s, s);
#pragma unroll
    for (int d = 0; d < D; ++d)
#pragma unroll
      for (int s = 0; s < 4; ++s) load_b_step(kt0 + d, s, bq[d]);
    __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0((S - 2) * PW + D * 4 * FN));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    read_stage(0, sa[0]);
    auto pstage = [&](int kt, AStage& cur, AStage& nxt, BReg& bb) {
      const int r = kt - kt0;
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(VM_PRE));
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      if (r >= 1) issue_a(kt + S - 1, (r - 1) % S);
      read_stage((r + 1) % S, nxt);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        mfmas(cur[s], bb[s]);
        load_b_step(kt + D, s, bb);
      }
      KSched<0, 4 * NM, 4 * FM, 4 * FN>::apply();
      __builtin_amdgcn_sched_barrier(0);
    };
    // Pairs of stages, then the odd one: no stage of the loop body is conditional, so the
    // compiler's wait for a B register counts both stages' loads issued after it.
    int kt = kt0;
    for (; kt + 1 < kt1; kt += 2) {
      pstage(kt, sa[0], sa[1], bq[0]);
      pstage(kt + 1, sa[1], sa[0], bq[D - 1]);
    }
    if (kt < kt1) pstage(kt, sa[0], sa[1], bq[0]);
  } else {
    BReg bq[D];
    bf16x8 b5q[X5 ? D : 1];
    // One k-step: [the DMA of a later A stage first, when `dma`], the next k-step's A
    // fragments from LDS, this k-step's MFMAs and the B loads of stage kt + D for this
    // k-step, interleaved one MFMA / one LDS read / a share of the VM loads. X5 (part):
    // k-step 0 also reads the A fragments of k-step `wave` of the stage, k-step 1 runs
    // the column-block-4 MFMAs on them, k-step 2 loads the block-4 fragment of stage
    // kt + D (after its use).
    auto kstep = [&](auto dma, auto part, int dma_kt, int dma_slot, int rd_slot, int rd_s, bf16x8* a_use,
                     bf16x8* a_next, bf16x8* b_use, int bkt, int s, BReg& bb, bf16x8& b5) {
      constexpr int X = X5 ? decltype(part)::value : 0;
      if constexpr (decltype(dma)::value) issue_a(dma_kt, dma_slot);
      read_a(rd_slot, rd_s, a_next);
      if constexpr (X == 1) read_a(rd_slot, wave, a5);
      mfmas(a_use, b_use);
      if constexpr (X == 2) mfmas5(b5);
      load_b_step(bkt, s, bb);
      if constexpr (X == 3) load_b5(bkt, b5);
      KSched<0, NM + (X == 2 ? FM : 0), FM, FN + (X == 3 ? 1 : 0)>::apply();
      __builtin_amdgcn_sched_barrier(0);
    };
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    using P2 = std::integral_constant<int, 2>;
    using P3 = std::integral_constant<int, 3>;

    // prologue: A stages kt0 .. kt0 + S - 1 (every slot), B stages kt0 .. kt0 + D - 1; the
    // wait covers A stages kt0 .. kt0 + Q (see the hand-over below)
    constexpr int Q = (S - 1 - D) > 1 ? (S - 1 - D) : 1;
  #pragma unroll
    for (int s = 0; s < S; ++s) issue_a(kt0 + s, s);
  #pragma unroll
    for (int d = 0; d < D; ++d) {
  #pragma unroll
      for (int s = 0; s < 4; ++s) load_b_step(kt0 + d, s, bq[d]);
      if constexpr (X5) load_b5(kt0 + d, b5q[d]);
    }
    // the epilogue inputs come after every prologue load: the waits below count only
    // loads issued after their target, so more of them (these) keep the waits exact or
    // conservative
    load_pre_in();
    __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0((S - 1 - Q) * PW + D * NB));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    read_a(0, 0, fa[0]);

    // Stage kt (slot (kt - kt0) % S, B buffer bb): k-steps 0..2; the hand-over: this wave's
    // DMA of stage kt + 1 has landed once at most VM_END later VM loads are pending, and
    // after the barrier every wave's has, and every wave is done reading slot kt; then
    // k-step 3 issues stage kt + S into that slot and reads stage kt + 1's first fragments.
    // VM loads issued after the DMA of stage kt + 1 (made in k-step 3 of stage kt + 1 - S):
    // B(3) of that stage, S - 2 whole stages (NB B loads + PW DMA each), the B loads of
    // k-steps 0..2 of stage kt (NB - FN). When stage kt + 1 (kt = kt0 + r) came from the
    // prologue, the loads after its DMA are (S - 2 - r) PW + D NB + r (NB + PW) + NB - FN,
    // at least VM_END once D + r >= S - 1; the prologue itself waited for stages up to
    // kt0 + Q, Q = max(1, S - 1 - D).
    constexpr int VM_END = NB + (S - 2) * (NB + PW);
    static_assert(VM_END < 64 && (S - 1 - Q) * PW + D * NB < 64, "vmcnt range");
    auto stage = [&](int kt, BReg& bb, bf16x8& b5) {
      const int rel = kt - kt0;
      const int slot = rel % S;
      const int nslot = (rel + 1) % S;
      kstep(std::false_type{}, P1{}, 0, 0, slot, 1, fa[0], fa[1], bb[0], kt + D, 0, bb, b5);
      kstep(std::false_type{}, P2{}, 0, 0, slot, 2, fa[1], fa[0], bb[1], kt + D, 1, bb, b5);
      kstep(std::false_type{}, P3{}, 0, 0, slot, 3, fa[0], fa[1], bb[2], kt + D, 2, bb, b5);
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(VM_END));
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      kstep(std::true_type{}, P0{}, kt + S, slot, nslot, 0, fa[1], fa[0], bb[3], kt + D, 3, bb, b5);
    };

    if constexpr (D == 3) {
      // Triples of stages, then the rest (as for pairs below)
      int kt = kt0;
      for (; kt + 2 < kt1; kt += 3) {
        stage(kt, bq[0], b5q[0]);
        stage(kt + 1, bq[1], b5q[X5 ? 1 : 0]);
        stage(kt + 2, bq[2], b5q[X5 ? 2 : 0]);
      }
      if (kt < kt1) stage(kt, bq[0], b5q[0]);
      if (kt + 1 < kt1) stage(kt + 1, bq[1], b5q[X5 ? 1 : 0]);
    } else if constexpr (D == 2) {
      // Pairs of stages, then the odd one: no stage of the loop body is conditional, so
      // the compiler's wait for a B register counts both stages' loads issued after it.
      int kt = kt0;
      for (; kt + 1 < kt1; kt += 2) {
        stage(kt, bq[0], b5q[0]);
        stage(kt + 1, bq[1], b5q[X5 ? 1 : 0]);
      }
      if (kt < kt1) stage(kt, bq[0], b5q[0]);
    } else {
      for (int kt = kt0; kt < kt1; ++kt) stage(kt, bq[0], b5q[0]);
    }
  }
  // The loads past the range (zero block, clamped B) must land before LDS is reused.
  __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
  __syncthreads();

  // ---- epilogue
  const int col = lane & 31;
  const int h4 = 4 * (lane >> 5);
  const int nw0 = n0 + wave * WN;
  // X5: the partial sums of column block 4 go to LDS in the register layout; wave w < FM
  // then sums row block w of it over the four waves in wave order.
  f32x16 acc5t;
  if constexpr (X5) {
    float* part5 = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) part5[((wave * FM + i) * 16 + r) * 64 + lane] = acc5[i][r];
    __syncthreads();
    if (wave < FM) {
#pragma unroll
      for (int r = 0; r < 16; ++r) acc5t[r] = part5[((0 * FM + wave) * 16 + r) * 64 + lane];
#pragma unroll
      for (int w = 1; w < 4; ++w)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc5t[r] += part5[((w * FM + wave) * 16 + r) * 64 + lane];
    }
    __syncthreads();
  }
  if (!X5 && !SPLIT && p.vt && nw0 + WN > p.vt_col0) {
    // columns of the per-head V^T output (or a wave straddling it): register layout,
    // lanes 0..31 = 32 consecutive tokens of one column
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int m = m0 + i * 32 + col;
      if (m >= p.M) continue;
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = nw0 + j * 32 + 8 * g + h4;
          float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
          epilogue_group<bf16>(p, m, n, v);
        }
    }
    return;
  }
  // Row-contiguous phase: 32 rows x WN fp32 per wave in LDS (row pitch WN + 4 floats:
  // the 16-byte writes of rows r .. r + 7 fall on distinct banks).
  constexpr int EPL = WN + 4;
  float* ep = reinterpret_cast<float*>(smem) + wave * (32 * EPL);
  float* slab = SPLIT ? p.part + (long long)split * p.M * p.n_store : nullptr;
  // One 32-row block of this wave's columns [nw0, nw0 + WN): blk[j] the accumulators of
  // column block j, rows mb .. mb + 31; i < 0: no preloaded epilogue input (the extra
  // column-block-4 block of X5), else its row block.
  auto epi_block = [&](const f32x16* blk, const int mb, const int nw0, const int i) {
    const bool pre_in_b = pre_in && i >= 0;
    const int ip = i >= 0 ? i : 0;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(ep + col * EPL + j * 32 + 8 * g + h4) =
            f32x4{blk[j][4 * g], blk[j][4 * g + 1], blk[j][4 * g + 2], blk[j][4 * g + 3]};
    if (SPLIT) {
      constexpr int LPR = WN / 4;   // lanes per row
      constexpr int RPI = 64 / LPR; // rows per pass
#pragma unroll
      for (int t = 0; t < 32 / RPI; ++t) {
        const int rr = t * RPI + lane / LPR;
        const int c4 = (lane % LPR) * 4;
        const f32x4 v4 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + c4);
        const int m = mb + rr, n = nw0 + c4;
        if (m >= p.M || n >= p.n_store) continue;
        *reinterpret_cast<f32x4*>(slab + (long long)m * p.n_store + n) = v4;
      }
    } else if (!p.geglu) {
      // A lane takes 8 consecutive columns of a row (16-byte bf16 stores: 4 lanes cover
      // a row's 64-byte segment), the same in every pass; the row vector and residual of
      // every pass of this 32-row block are loaded before the block is read back from
      // LDS, so the block waits on one memory latency instead of one per pass. Same
      // arithmetic as epilogue_group: ((acc + bias) + row vector) + residual.
      constexpr int LPR = WN / 8;
      constexpr int RPI = 64 / LPR;
      constexpr int NP = 32 / RPI;
      const int c8 = (lane % LPR) * 8;
      const int n = nw0 + c8;
      const bool ncol = n < p.n_store;
      const bool full = n + 8 <= p.n_store;
      const bool rvec = full && p.resid && resid_vec8(p);
      float rv[NP][8], rs[NP][8];
#pragma unroll
      for (int t = 0; t < NP; ++t) {
        const int m = mb + t * RPI + lane / LPR;
#pragma unroll
        for (int e = 0; e < 8; ++e) rv[t][e] = rs[t][e] = 0.f;
        if (m >= p.M || !ncol || pre_in_b) continue;
        if (p.rowvec) load_rowvec8(p, m, n, rv[t]);
        if (p.resid) load_resid8(p, m, n, rvec, rs[t]);
      }
      float bias8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) bias8[e] = p.bias && n + e < p.n_store ? p.bias[n + e] : 0.f;
      const bool ovec = full && out_vec8(p);
#pragma unroll
      for (int t = 0; t < NP; ++t) {
        const int rr = t * RPI + lane / LPR;
        const f32x4 a0 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + c8);
        const f32x4 a1 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + c8 + 4);
        const int m = mb + rr;
        if (m >= p.M || !ncol) continue;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float x = e < 4 ? a0[e] : a1[e - 4];
          if (p.bias) x += bias8[e];
          if constexpr (kPreIn) {
            if (pre_in_b) x += pin[ip][t][e / 4][e % 4];
          }
          if (!pre_in_b) {
            if (p.rowvec) x += rv[t][e];
            if (p.resid) x += rs[t][e];
          }
          v[e] = x;
        }
        store8(p, m, n, v, ovec);
      }
    } else {
      // GEGLU: within each 64-column pair block, columns [0, 32) are values and
      // [32, 64) the matching gates; output column = (pair block) * 32 + c. A lane takes
      // 8 consecutive outputs of a row, so each store is 16 bytes (4 lanes cover a row's
      // 64-byte segment); its value and gate columns are the same in every pass, so
      // their biases load once.
      // (tiles with 32 columns per wave never take GEGLU: the host rejects them)
      if constexpr (WN % 64 == 0) {
        constexpr int LPR = WN / 16;
        constexpr int RPI = 64 / LPR;
        const int cq = (lane % LPR) * 8;            // 0 .. WN/2 - 8
        const int pb = cq / 32, c8 = cq % 32;       // pair block, column in it
        const int lc = pb * 64 + c8;                // value column within the wave
        const int nv = nw0 + lc;
        const int o = nw0 / 2 + cq;
        float ba[8], bg[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) ba[e] = bg[e] = 0.f;
        if (p.bias && o < p.n_store) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            ba[e] = p.bias[nv + e];
            bg[e] = p.bias[nv + 32 + e];
          }
        }
        const bool vec8 = !p.out_f32 && o + 8 <= p.n_store && out_vec8(p);
#pragma unroll
        for (int t = 0; t < 32 / RPI; ++t) {
          const int rr = t * RPI + lane / LPR;
          const f32x4 a0 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc);
          const f32x4 a1 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc + 4);
          const f32x4 g0 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc + 32);
          const f32x4 g1 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc + 36);
          const int m = mb + rr;
          if (m >= p.M || o >= p.n_store) continue;
          float v[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = (a0[e] + ba[e]) * gelu_erf(g0[e] + bg[e]);
            v[e + 4] = (a1[e] + ba[e + 4]) * gelu_erf(g1[e] + bg[e + 4]);
          }
          if (vec8) {
            bf16x8 w;
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = static_cast<bf16>(v[e]);
            *reinterpret_cast<bf16x8*>(static_cast<bf16*>(p.out) + (long long)m * p.ldo + o) = w;
          } else {
            store4<bf16>(p, m, o, v, p.n_store);
            store4<bf16>(p, m, o + 4, v + 4, p.n_store);
          }
        }
      }
    }
  };
#pragma unroll
  for (int i = 0; i < FM; ++i) epi_block(acc[i], m0 + i * 32, nw0, i);
  if constexpr (X5) {
    if (wave < FM) epi_block(&acc5t, m0 + wave * 32, n0 + 128, -1);
  }
}

// The kernel: unit assignment (see the file comment), then the unit's tile. TBM > 0 with
// tail_bands > 0 (no split): the first tail_full units are BM-row tiles of the column
// bands before the last tail_bands, the rest TBM-row tiles of those last bands; each
// XCD takes its share of both kinds, full tiles first (tail_full and the tail count
// are multiples of the XCD count). A grid of BM-row tiles that fills a whole number of
// rounds plus a fraction of one leaves that fraction to half the CUs; TBM-row tiles
// spread it over all of them.
template <int BM, int FN, int S, int D, int WPE, int MODE, bool SPLIT, int PRE, int NW = 4, bool X5 = false,
          int TBM = 0>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(WPE, WPE))) void gemm_frag_kernel(
    GemmParams p, int mt, int nt, int nsplit, int tail_full, int tail_bands) {
  constexpr int BN = X5 ? 160 : NW * 32 * FN;
  const int wg = blockIdx.x;
  const int xcd = wg % kXcds, idx = wg / kXcds;
  const int nk = p.K / kBK;
  if constexpr (TBM > 0) {
    static_assert(!SPLIT, "tail tiles take no split");
    if (tail_bands > 0) {
      const int fx = tail_full / kXcds;
      const int tm = (p.M + TBM - 1) / TBM;
      const int tx = tm * tail_bands / kXcds;
      if (idx < fx) {
        const int f = xcd * fx + idx;
        frag_tile<BM, FN, S, D, WPE, MODE, SPLIT, PRE, NW, X5>(p, (f % mt) * BM, (f / mt) * BN, 0, 0, nk);
      } else {
        const int t = xcd * tx + (idx - fx);
        frag_tile<TBM, FN, S, 1, WPE, MODE, SPLIT, PRE, NW, X5>(p, (t % tm) * TBM,
                                                                (nt - tail_bands + t / tm) * BN, 0, 0, nk);
      }
      return;
    }
  }
  const int units = mt * nt * nsplit;
  const int base = units / kXcds, rem = units % kXcds;
  const int logical = xcd * base + min(xcd, rem) + idx;
  const int m_tile = logical % mt;
  const int ns = logical / mt;
  const int split = ns % nsplit;
  const int n_tile = ns / nsplit;
  const int kt0 = (int)((long long)split * nk / nsplit);
  const int kt1 = (int)((long long)(split + 1) * nk / nsplit);
  frag_tile<BM, FN, S, D, WPE, MODE, SPLIT, PRE, NW, X5>(p, m_tile * BM, n_tile * BN, split, kt0, kt1);
}

// Sum of the split-K partial slabs [NS][M][n_store] in split order, then the epilogue;
// one thread per 4 consecutive columns of a row, all slab loads issued before the sum.
template <int NS> __global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmParams p) {
  const int q = p.n_store / 4;
  const long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (i >= (long long)p.M * q) return;
  const int m = (int)(i / q);
  const int n = (int)(i - (long long)m * q) * 4;
  const long long slab = (long long)p.M * p.n_store;
  const float* src = p.part + (long long)m * p.n_store + n;
  f32x4 t[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) t[k] = *reinterpret_cast<const f32x4*>(src + k * slab);
  f32x4 s = t[0];
#pragma unroll
  for (int k = 1; k < NS; ++k) {
    s[0] += t[k][0];
    s[1] += t[k][1];
    s[2] += t[k][2];
    s[3] += t[k][3];
  }
  float v[4] = {s[0], s[1], s[2], s[3]};
  epilogue_group<bf16>(p, m, n, v);
}

void splitk_reduce(const GemmParams& p, int nsplit, hipStream_t s) {
  const long long nq = (long long)p.M * (p.n_store / 4);
  const dim3 grid(static_cast<unsigned>((nq + 255) / 256));
  switch (nsplit) {
    case 2: hipLaunchKernelGGL(splitk_reduce_kernel<2>, grid, dim3(256), 0, s, p); break;
    case 3: hipLaunchKernelGGL(splitk_reduce_kernel<3>, grid, dim3(256), 0, s, p); break;
    case 4: hipLaunchKernelGGL(splitk_reduce_kernel<4>, grid, dim3(256), 0, s, p); break;
    case 5: hipLaunchKernelGGL(splitk_reduce_kernel<5>, grid, dim3(256), 0, s, p); break;
    case 6: hipLaunchKernelGGL(splitk_reduce_kernel<6>, grid, dim3(256), 0, s, p); break;
    case 7: hipLaunchKernelGGL(splitk_reduce_kernel<7>, grid, dim3(256), 0, s, p); break;
    case 8: hipLaunchKernelGGL(splitk_reduce_kernel<8>, grid, dim3(256), 0, s, p); break;
    default: throw Error(-1, "gemm: split-K reduction takes 2 to 8 slabs");
  }
  DN_HIP(hipGetLastError());
}

template <int BM, int FN, int S, int D, int WPE, int MODE, bool SPLIT, int PRE, int NW, bool X5, int TBM = 0>
void launch_frag(const GemmParams& p, int nsplit, hipStream_t s, int tail_bands = 0) {
  constexpr size_t lds_full = frag_lds_bytes<BM, FN, S, NW, X5>();
  constexpr size_t lds_tail = TBM > 0 ? frag_lds_bytes<(TBM > 0 ? TBM : BM), FN, S, NW, X5>() : 0;
  constexpr size_t lds = lds_full > lds_tail ? lds_full : lds_tail;
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(
        reinterpret_cast<const void*>(&gemm_frag_kernel<BM, FN, S, D, WPE, MODE, SPLIT, PRE, NW, X5, TBM>),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  const int mt = ceil_div(p.M, BM), nt = ceil_div(p.N, X5 ? 160 : 32 * FN * NW);
  int grid = mt * nt * nsplit, tail_full = 0;
  if (TBM > 0 && tail_bands > 0) {
    tail_full = mt * (nt - tail_bands);
    const int tail = ceil_div(p.M, TBM > 0 ? TBM : BM) * tail_bands;
    DN_CHECK(nsplit == 1 && tail_bands < nt && tail_full % kXcds == 0 && tail % kXcds == 0,
             "gemm: tail tiles need no split and tile counts divisible by the XCD count");
    grid = tail_full + tail;
  }
  hipLaunchKernelGGL((gemm_frag_kernel<BM, FN, S, D, WPE, MODE, SPLIT, PRE, NW, X5, TBM>), dim3(grid), dim3(64 * NW),
                     lds, s, p, mt, nt, nsplit, tail_full, TBM > 0 ? tail_bands : 0);
  DN_HIP(hipGetLastError());
}

template <int BM, int FN, int S, int D, int WPE, int MODE, int PRE = 0, int NW = 4, bool X5 = false>
void run_frag(const GemmParams& p, int nsplit, hipStream_t s) {
  if (p.raw_partial) {
    launch_frag<BM, FN, S, D, WPE, MODE, true, PRE, NW, X5>(p, nsplit, s);
  } else if (nsplit > 1) {
    launch_frag<BM, FN, S, D, WPE, MODE, true, PRE, NW, X5>(p, nsplit, s);
    splitk_reduce(p, nsplit, s);
  } else {
    launch_frag<BM, FN, S, D, WPE, MODE, false, PRE, NW, X5>(p, 1, s);
  }
}

// Tile plans (three LDS stages): 128 x 256 (FN = 2) with two B buffers (one for the
// convolution), two workgroups per CU; 128 x 128 (FN = 1) and 64 x 128 with two B buffers,
// two / four workgroups per CU; 64 x 160 and 128 x 160 on five waves with three B buffers,
// one workgroup per CU, or (stages = 5) on four waves (X5) with three / two B buffers, two
// workgroups per CU. stages = 2 selects the 128 x 256 variant with two B buffers and one
// workgroup per CU.
template <int MODE> void dispatch_frag(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  if (g.bm == 128 && g.bn == 256 && g.stages == 3) {
    // B two stages ahead where the registers allow it (the implicit convolution's
    // address registers do not leave room)
    if constexpr (MODE == 2) {
      return run_frag<128, 2, 3, 1, 2, MODE>(p, g.split, s);
    } else {
      // the last column bands of a grid with a partial last round as 64-row tiles
      if (g.tail_bands > 0 && g.split == 1 && !p.raw_partial) {
        launch_frag<128, 2, 3, 2, 2, MODE, false, 0, 4, false, 64>(p, 1, s, g.tail_bands);
        return;
      }
      return run_frag<128, 2, 3, 2, 2, MODE>(p, g.split, s);
    }
  }
  if (g.bm == 128 && g.bn == 256 && g.stages == 2) return run_frag<128, 2, 3, 2, 1, MODE>(p, g.split, s);
  if (g.bm == 128 && g.bn == 128 && g.stages == 3) return run_frag<128, 1, 3, 2, 2, MODE>(p, g.split, s);
  if (g.bm == 64 && g.bn == 128 && g.stages == 3) return run_frag<64, 1, 3, 2, 4, MODE>(p, g.split, s);
  if (g.bm == 64 && g.bn == 128 && g.stages == 13) return run_frag<64, 1, 3, 2, 3, MODE, 1>(p, g.split, s);
  if (g.bm == 64 && g.bn == 128 && g.stages == 14) return run_frag<64, 1, 4, 2, 3, MODE, 1>(p, g.split, s);
  if (g.bm == 128 && g.bn == 128 && g.stages == 13) return run_frag<128, 1, 3, 2, 2, MODE, 1>(p, g.split, s);
  if (g.bm == 64 && g.bn == 256 && g.stages == 13) return run_frag<64, 2, 3, 2, 2, MODE, 1>(p, g.split, s);
  if (g.bm == 32 && g.bn == 128 && g.stages == 13) return run_frag<32, 1, 3, 2, 4, MODE, 1>(p, g.split, s);
  if constexpr (MODE != 2) {
    if (g.bm == 64 && g.bn == 160 && (g.stages == 3 || p.vt)) return run_frag<64, 1, 3, 3, 2, MODE, 0, 5>(p, g.split, s);
  }
  if (!p.vt) {
    if (g.bm == 64 && g.bn == 160 && g.stages == 5) return run_frag<64, 1, 3, 3, 2, MODE, 0, 4, true>(p, g.split, s);
    if (g.bm == 32 && g.bn == 160 && g.stages == 5) return run_frag<32, 1, 3, 3, 2, MODE, 0, 4, true>(p, g.split, s);
  }
  if (g.bm == 128 && g.bn == 160 && (g.stages == 3 || p.vt)) return run_frag<128, 1, 3, 3, 2, MODE, 0, 5>(p, g.split, s);
  if (g.bm == 128 && g.bn == 160 && g.stages == 5) return run_frag<128, 1, 3, 2, 2, MODE, 0, 4, true>(p, g.split, s);
  throw Error(-1, "gemm: no fragment-B kernel for this tile plan");
}

// ---------------------------------------------------------------- fp8 (E4M3) kernel
//
// The same organisation as gemm_frag_kernel for E4M3 operands on the 32x32x64 fp8
// matrix-core step (v_mfma_scale_f32_32x32x64_f8f6f4 with unit block scales): an LDS
// stage still holds 128-byte rows, now 128 k-values, i.e. two matrix-core steps; lane l
// supplies row (l % 32) and the 32 consecutive k-values 32 (l / 32) .. + 32 of a step
// (two 16-byte LDS reads; any k order common to both operands gives the same sum).
// B is packed by pack_fp8: per 32 output rows and 64-deep step, the lanes' 32-byte
// operands in 2 KB. The epilogue multiplies each column by its row scale of B.
typedef int v8i __attribute__((ext_vector_type(8)));

__device__ __forceinline__ v8i v8i_of(const uint4& a, const uint4& b) {
  v8i r;
  r[0] = (int)a.x, r[1] = (int)a.y, r[2] = (int)a.z, r[3] = (int)a.w;
  r[4] = (int)b.x, r[5] = (int)b.y, r[6] = (int)b.z, r[7] = (int)b.w;
  return r;
}

// Eight outputs [n, n + 8) of row m as E4M3 codes (8 bytes), or element-wise past n_store.
__device__ __forceinline__ void store8_fp8(const GemmParams& p, int m, int n, const float v[8]) {
  uint8_t* o = static_cast<uint8_t*>(p.out) + (long long)m * p.ldo + n;
  if (n + 8 <= p.n_store && ((reinterpret_cast<__UINTPTR_TYPE__>(o) & 7) == 0)) {
    uint2 w;
    w.x = fp8x4(v[0], v[1], v[2], v[3]);
    w.y = fp8x4(v[4], v[5], v[6], v[7]);
    *reinterpret_cast<uint2*>(o) = w;
  } else {
    for (int e = 0; e < 8; ++e)
      if (n + e < p.n_store) o[e] = static_cast<uint8_t>(fp8x4(v[e], 0.f, 0.f, 0.f) & 0xff);
  }
}

template <int BM, int FN, int S, int WPE, bool SPLIT>
__device__ __forceinline__ void fp8_tile(const GemmParams& p, const int m0, const int n0, const int split,
                                         const int kt0, const int kt1) {
  constexpr int NW = 4;
  constexpr int FM = BM / 32;
  constexpr int WN = 32 * FN;
  constexpr int BN = NW * WN;
  constexpr int STAGE = BM * kRowBytes;
  constexpr int PW = BM / 32;  // DMA instructions (8 rows of 128 B) per wave per stage
  constexpr int NM = FM * FN;
  static_assert(S >= 3 && S <= 4, "three or four LDS stages");

  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  // A rows: DMA instruction j of this wave fills tile rows [8 q, 8 q + 8), q = wave PW + j
  const int lrow = lane >> 3;
  const int lc_even = ((lane & 7) ^ lrow) * 16, lc_odd = ((lane & 7) ^ lrow ^ 1) * 16;
  int off0[PW];
#pragma unroll
  for (int j = 0; j < PW; ++j) {
    const int q = wave * PW + j;
    const int m = min(m0 + 8 * q + lrow, p.M - 1);
    off0[j] = m * p.lda0 + ((q & 1) ? lc_odd : lc_even);
  }
  const uint8_t* const gA = static_cast<const uint8_t*>(p.a0);
  auto issue_a = [&](int kt_in, int slot) {
    const bool real = kt_in < kt1;
    unsigned char* stage = smem + slot * STAGE;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int q = wave * PW + j;
      const uint8_t* g = real ? gA + off0[j] + kt_in * 128 : static_cast<const uint8_t*>(p.zero16);
      dma16(g, (lds_void*)(stage + q * 1024));
    }
  };

  // B operands of this wave: column blocks nb = (n0 + wave WN) / 32 + j (clamped)
  const int ksteps = p.K / 64;
  const int nb_last = (p.N + 31) / 32 - 1;
  const uint8_t* bptr[FN];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int nb = min((n0 + wave * WN) / 32 + j, nb_last);
    bptr[j] = static_cast<const uint8_t*>(p.b) + (long long)nb * ksteps * 2048 + lane * 32;
  }
  typedef uint4 BStep[FN][2];  // one 64-deep step: FN column blocks, 32 bytes per lane
  auto load_b = [&](int step_in, BStep& dst) {
    const int st = step_in < 2 * kt1 ? step_in : 2 * kt1 - 1;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const uint8_t* src = bptr[j] + (long long)st * 2048;
      dst[j][0] = *reinterpret_cast<const uint4*>(src);
      dst[j][1] = *reinterpret_cast<const uint4*>(src + 16);
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int frow = lane & 31;
  const int fs = (lane & 7) ^ ((lane >> 3) & 1);
  const int hh = lane >> 5;
  auto read_a = [&](int slot, int s2, v8i* a) {
    const unsigned char* st = smem + slot * STAGE + frow * kRowBytes;
    const int c0 = 4 * s2 + 2 * hh;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const uint4 lo = *reinterpret_cast<const uint4*>(st + i * 32 * kRowBytes + ((c0 ^ fs) * 16));
      const uint4 hi = *reinterpret_cast<const uint4*>(st + i * 32 * kRowBytes + (((c0 + 1) ^ fs) * 16));
      a[i] = v8i_of(lo, hi);
    }
  };
  auto mfmas = [&](const v8i* a, const BStep& b) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(v8i_of(b[j][0], b[j][1]), a[i], acc[i][j], 0, 0,
                                                                    0, 127, 0, 127);
  };

  // B is loaded two 64-deep steps ahead into two register sets. Stage kt (r = kt - kt0):
  // wait until this wave's DMA of stage kt landed, barrier; step 2 kt, then B of step
  // 2 kt + 2 into its set; step 2 kt + 1, then B of step 2 kt + 3; last, the DMA of stage
  // kt + 2 into the slot of stage kt - 1. The compiler waits for a B set counting only the
  // B loads issued after it, so each of its waits also retires the oldest DMA issued
  // after that B load: with this order that is at most the DMA of stage kt + 1, in the
  // second half of stage kt, just before it is needed (with FN = 1 the first wait of a
  // stage retires half of it). Loads issued after the DMA of stage kt: PW + 4 FN
  // (r = 0: the prologue's second DMA and B sets; steady state: stage kt - 1's B loads
  // and DMA), 8 FN + PW (r = 1: the prologue's B sets and stage kt0's loads).
  static_assert(S == 3, "three LDS stages");
  constexpr int WS = PW + 4 * FN;
  constexpr int W1 = 8 * FN + PW;
  static_assert(W1 < 64, "vmcnt range");
  issue_a(kt0, 0);
  issue_a(kt0 + 1, 1);
  BStep b0, b1;
  load_b(2 * kt0, b0);
  load_b(2 * kt0 + 1, b1);
  for (int kt = kt0; kt < kt1; ++kt) {
    const int r = kt - kt0;
    if (r == 1)
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(W1));
    else
      __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(WS));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    const int slot = r % 3;
    v8i a[FM];
    read_a(slot, 0, a);
    mfmas(a, b0);
    KSched<0, NM, 0, 0>::apply();
    __builtin_amdgcn_sched_barrier(0);
    load_b(2 * kt + 2, b0);
    read_a(slot, 1, a);
    mfmas(a, b1);
    KSched<0, NM, 0, 0>::apply();
    __builtin_amdgcn_sched_barrier(0);
    load_b(2 * kt + 3, b1);
    issue_a(kt + 2, (r + 2) % 3);
  }
  __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
  __syncthreads();

  // ---- epilogue (row-contiguous through LDS, as gemm_frag_kernel), columns scaled
  const int col = lane & 31;
  const int h4 = 4 * (lane >> 5);
  const int nw0 = n0 + wave * WN;
  constexpr int EPL = WN + 4;
  float* ep = reinterpret_cast<float*>(smem) + wave * (32 * EPL);
  float* slab = SPLIT ? p.part + (long long)split * p.M * p.n_store : nullptr;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(ep + col * EPL + j * 32 + 8 * g + h4) =
            f32x4{acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
    const int mb = m0 + i * 32;
    if (SPLIT) {
      constexpr int LPR = WN / 4;
      constexpr int RPI = 64 / LPR;
      const int c4 = (lane % LPR) * 4;
      const int n = nw0 + c4;
      float sc[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) sc[e] = n + e < p.n_store ? p.wscale[n + e] : 0.f;
#pragma unroll
      for (int t = 0; t < 32 / RPI; ++t) {
        const int rr = t * RPI + lane / LPR;
        f32x4 v4 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + c4);
        const int m = mb + rr;
        if (m >= p.M || n >= p.n_store) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] *= sc[e];
        *reinterpret_cast<f32x4*>(slab + (long long)m * p.n_store + n) = v4;
      }
    } else if (!p.geglu) {
      constexpr int LPR = WN / 8;
      constexpr int RPI = 64 / LPR;
      constexpr int NP = 32 / RPI;
      const int c8 = (lane % LPR) * 8;
      const int n = nw0 + c8;
      const bool ncol = n < p.n_store;
      const bool full = n + 8 <= p.n_store;
      const bool rvec = full && p.resid && resid_vec8(p);
      float sc[8], bias8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sc[e] = n + e < p.n_store ? p.wscale[n + e] : 0.f;
        bias8[e] = p.bias && n + e < p.n_store ? p.bias[n + e] : 0.f;
      }
      const bool ovec = full && out_vec8(p);
#pragma unroll
      for (int t = 0; t < NP; ++t) {
        const int rr = t * RPI + lane / LPR;
        const int m = mb + rr;
        if (m >= p.M || !ncol) continue;
        float rs[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (p.resid) load_resid8(p, m, n, rvec, rs);
        const f32x4 a0 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + c8);
        const f32x4 a1 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + c8 + 4);
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (e < 4 ? a0[e] : a1[e - 4]) * sc[e] + bias8[e] + rs[e];
        if (p.out_fp8)
          store8_fp8(p, m, n, v);
        else
          store8(p, m, n, v, ovec);
      }
    } else {
      // GEGLU over 64-column (value, gate) pair blocks, as gemm_frag_kernel
      if constexpr (WN % 64 == 0) {
        constexpr int LPR = WN / 16;
        constexpr int RPI = 64 / LPR;
        const int cq = (lane % LPR) * 8;
        const int pb = cq / 32, c8 = cq % 32;
        const int lc = pb * 64 + c8;
        const int nv = nw0 + lc;
        const int o = nw0 / 2 + cq;
        float ba[8], bg[8], sa[8], sg[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool in = o < p.n_store;
          ba[e] = in && p.bias ? p.bias[nv + e] : 0.f;
          bg[e] = in && p.bias ? p.bias[nv + 32 + e] : 0.f;
          sa[e] = in ? p.wscale[nv + e] : 0.f;
          sg[e] = in ? p.wscale[nv + 32 + e] : 0.f;
        }
        const bool vec8 = !p.out_f32 && o + 8 <= p.n_store && out_vec8(p);
#pragma unroll
        for (int t = 0; t < 32 / RPI; ++t) {
          const int rr = t * RPI + lane / LPR;
          const f32x4 a0 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc);
          const f32x4 a1 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc + 4);
          const f32x4 g0 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc + 32);
          const f32x4 g1 = *reinterpret_cast<const f32x4*>(ep + rr * EPL + lc + 36);
          const int m = mb + rr;
          if (m >= p.M || o >= p.n_store) continue;
          float v[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = (a0[e] * sa[e] + ba[e]) * gelu_erf(g0[e] * sg[e] + bg[e]);
            v[e + 4] = (a1[e] * sa[e + 4] + ba[e + 4]) * gelu_erf(g1[e] * sg[e + 4] + bg[e + 4]);
          }
          if (p.out_fp8) {
            store8_fp8(p, m, o, v);
          } else if (vec8) {
            bf16x8 w;
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = static_cast<bf16>(v[e]);
            *reinterpret_cast<bf16x8*>(static_cast<bf16*>(p.out) + (long long)m * p.ldo + o) = w;
          } else {
            store4<bf16>(p, m, o, v, p.n_store);
            store4<bf16>(p, m, o + 4, v + 4, p.n_store);
          }
        }
      }
    }
  }
}

// The fp8 kernel: unit assignment as gemm_frag_kernel (XCD-contiguous; with TBM > 0 and
// tail_bands > 0 the last column bands as TBM-row tiles, full tiles first on every XCD).
template <int BM, int FN, int S, int WPE, bool SPLIT, int TBM = 0>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE, WPE))) void gemm_fp8_kernel(
    GemmParams p, int mt, int nt, int nsplit, int tail_full, int tail_bands) {
  constexpr int BN = 4 * 32 * FN;
  const int wg = blockIdx.x;
  const int xcd = wg % kXcds, idx = wg / kXcds;
  const int nk = p.K / 128;
  if constexpr (TBM > 0) {
    static_assert(!SPLIT, "tail tiles take no split");
    if (tail_bands > 0) {
      const int fx = tail_full / kXcds;
      const int tm = (p.M + TBM - 1) / TBM;
      const int tx = tm * tail_bands / kXcds;
      if (idx < fx) {
        const int f = xcd * fx + idx;
        fp8_tile<BM, FN, S, WPE, SPLIT>(p, (f % mt) * BM, (f / mt) * BN, 0, 0, nk);
      } else {
        const int t = xcd * tx + (idx - fx);
        fp8_tile<TBM, FN, S, WPE, SPLIT>(p, (t % tm) * TBM, (nt - tail_bands + t / tm) * BN, 0, 0, nk);
      }
      return;
    }
  }
  const int units = mt * nt * nsplit;
  const int base = units / kXcds, rem = units % kXcds;
  const int logical = xcd * base + min(xcd, rem) + idx;
  const int m_tile = logical % mt;
  const int ns = logical / mt;
  const int split = ns % nsplit;
  const int n_tile = ns / nsplit;
  const int kt0 = (int)((long long)split * nk / nsplit);
  const int kt1 = (int)((long long)(split + 1) * nk / nsplit);
  fp8_tile<BM, FN, S, WPE, SPLIT>(p, m_tile * BM, n_tile * BN, split, kt0, kt1);
}

template <int BM, int FN, int S, int WPE, bool SPLIT, int TBM = 0>
void launch_fp8(const GemmParams& p, int nsplit, hipStream_t s, int tail_bands = 0) {
  constexpr size_t lds_full = frag_lds_bytes<BM, FN, S, 4>();
  constexpr size_t lds_tail = TBM > 0 ? frag_lds_bytes<(TBM > 0 ? TBM : BM), FN, S, 4>() : 0;
  constexpr size_t lds = lds_full > lds_tail ? lds_full : lds_tail;
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_fp8_kernel<BM, FN, S, WPE, SPLIT, TBM>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  const int mt = ceil_div(p.M, BM), nt = ceil_div(p.N, 32 * FN * 4);
  int grid = mt * nt * nsplit, tail_full = 0;
  if (TBM > 0 && tail_bands > 0) {
    tail_full = mt * (nt - tail_bands);
    const int tail = ceil_div(p.M, TBM > 0 ? TBM : BM) * tail_bands;
    DN_CHECK(nsplit == 1 && tail_bands < nt && tail_full % kXcds == 0 && tail % kXcds == 0,
             "gemm_fp8: tail tiles need no split and tile counts divisible by the XCD count");
    grid = tail_full + tail;
  }
  hipLaunchKernelGGL((gemm_fp8_kernel<BM, FN, S, WPE, SPLIT, TBM>), dim3(grid), dim3(256), lds, s, p, mt, nt, nsplit,
                     tail_full, TBM > 0 ? tail_bands : 0);
  DN_HIP(hipGetLastError());
}

template <int BM, int FN, int S, int WPE> void run_fp8(const GemmParams& p, int nsplit, hipStream_t s) {
  if (p.raw_partial) {
    launch_fp8<BM, FN, S, WPE, true>(p, nsplit, s);
  } else if (nsplit > 1) {
    launch_fp8<BM, FN, S, WPE, true>(p, nsplit, s);
    // the slabs hold scaled sums; the reduction applies bias / residual (unit scales)
    GemmParams q = p;
    splitk_reduce(q, nsplit, s);
  } else {
    launch_fp8<BM, FN, S, WPE, false>(p, 1, s);
  }
}

// Fragment order of a packed [N][K] weight matrix (N rounded up to 32, K % 16 == 0):
// element (n, k) lives at ((n / 32) * (K / 16) + k / 16) * 512 + lane * 8 + k % 8 with
// lane = n % 32 + 32 * ((k % 16) / 8).
__global__ void to_frag_kernel(const bf16* src, int N, int K, int lds, bf16* dst, int Npad) {
  const long long nv = (long long)Npad * K / 8;
  const int kbs = K / 16;
  for (long long v = blockIdx.x * (long long)blockDim.x + threadIdx.x; v < nv; v += (long long)gridDim.x * blockDim.x) {
    const int lane = (int)(v % 64);
    const long long t = v / 64;
    const int kb = (int)(t % kbs);
    const int nb = (int)(t / kbs);
    const int n = nb * 32 + (lane & 31);
    const int k = kb * 16 + (lane >> 5) * 8;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (n < N) val = *reinterpret_cast<const uint4*>(src + (long long)n * lds + k);
    *reinterpret_cast<uint4*>(dst + v * 8) = val;
  }
}

}  // namespace

bool gemm_frag_layout(int N, int K) { return N >= 32 && N % 32 == 0 && K >= kBK && K % kBK == 0; }

size_t gemm_frag_elems(int N, int K) { return (size_t)((N + 31) / 32 * 32) * K; }

void to_frag(const bf16* src, int N, int K, int ld_src, bf16* dst, hipStream_t s) {
  DN_CHECK(K % 16 == 0 && ld_src % 8 == 0 && ld_src >= K, "to_frag: K and the source pitch must suit 16-byte rows");
  const int Npad = (N + 31) / 32 * 32;
  const long long nv = (long long)Npad * K / 8;
  const int blocks = static_cast<int>(std::min<long long>((nv + 255) / 256, 16384));
  hipLaunchKernelGGL(to_frag_kernel, dim3(std::max(blocks, 1)), dim3(256), 0, s, src, N, K, ld_src, dst, Npad);
  DN_HIP(hipGetLastError());
}

bool gemm_fp8_layout(int N, int K) { return N >= 32 && N % 32 == 0 && K >= 128 && K % 128 == 0; }

size_t gemm_fp8_code_bytes(int N, int K) { return (size_t)((N + 31) / 32 * 32) * K; }

GemmPlan gemm_plan_fp8(int M, int N, int K, int geglu, int cus, bool allow_split, bool fused_reduce) {
  // the bf16 planner's choice among its 128 x 256 and 128 x 128 tiles (and its split)
  GemmPlan g = frag_plan(M, N, K, geglu, cus, allow_split, fused_reduce, false);
  if (!(g.bm == 128 && (g.bn == 256 || g.bn == 128))) {
    g.bm = 128;
    g.bn = (geglu || N >= 1024) ? 256 : 128;
    g.split = 1;
    g.tail_bands = 0;
  }
  while (g.split > 1 && K / 128 < 2 * g.split) --g.split;
  g.frag = 1;
  g.stages = 3;
  // the bf16 planner's tail bands hold for the same 128 x 256 grid (two workgroups per CU)
  if (!(g.bn == 256 && g.split == 1)) g.tail_bands = 0;
  return g;
}

void gemm_fp8(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  DN_CHECK(gemm_fp8_layout(p.N, p.K), "gemm_fp8: N % 32 == 0 and K % 128 == 0 needed");
  DN_CHECK(p.taps == 1 && p.c1 == 0 && p.c0 == p.K, "gemm_fp8: one linear A source");
  DN_CHECK(p.a0 && p.b && p.out && p.wscale && p.zero16, "gemm_fp8: null operand");
  DN_CHECK(p.lda0 % 16 == 0, "gemm_fp8: A rows must be 16-byte aligned");
  DN_CHECK(!p.vt, "gemm_fp8: no V^T output");
  DN_CHECK(g.split >= 1 && g.split <= kMaxSplit && p.K / 128 >= g.split, "gemm_fp8: bad split");
  DN_CHECK(!p.geglu || g.bn == 256, "gemm_fp8: GEGLU needs 64-column value/gate pairs per wave");
  if (g.split > 1 || p.raw_partial) {
    DN_CHECK(!p.geglu && !p.out_fp8, "gemm_fp8: split-K takes neither GEGLU nor fp8 output");
    DN_CHECK(p.n_store % 4 == 0 && p.n_store == p.N, "gemm_fp8: split-K needs n_store == N, a multiple of 4");
    DN_CHECK(p.part && p.part_floats >= (size_t)g.split * p.M * p.n_store, "gemm_fp8: split-K workspace too small");
  }
  if (g.bn == 256 && g.split == 1 && g.tail_bands > 0 && !p.raw_partial)
    launch_fp8<128, 2, 3, 2, false, 64>(p, 1, s, g.tail_bands);
  else if (g.bn == 256)
    run_fp8<128, 2, 3, 2>(p, g.split, s);
  else
    run_fp8<128, 1, 3, 2>(p, g.split, s);
}

void gemm_bf16_frag(const GemmParams& p, const GemmPlan& g, hipStream_t s) {
  DN_CHECK(gemm_frag_layout(p.N, p.K), "gemm: fragment-B kernel needs N % 32 == 0 and K % 64 == 0");
  DN_CHECK(p.taps == 1 || (p.c0 + p.c1) % kBK == 0, "gemm: conv channels must be a multiple of 64");
  DN_CHECK(p.c1 == 0 || p.c0 % kBK == 0, "gemm: concatenation split must be a multiple of 64");
  DN_CHECK(p.taps == 1 || p.zero16, "gemm: implicit conv needs the zero block");
  DN_CHECK(p.taps == 1 || p.c1 == 0, "gemm: the fragment-B conv takes one input source");
  DN_CHECK(g.split >= 1 && g.split <= kMaxSplit && p.K / kBK >= g.split, "gemm: bad split");
  DN_CHECK(!p.geglu || (g.bn / 4) % 64 == 0, "gemm: GEGLU needs 64-column value/gate pairs per wave");
  if (g.split > 1 || p.raw_partial) {
    DN_CHECK(!p.geglu && !p.vt, "gemm: split-K takes neither GEGLU nor the V^T output");
    DN_CHECK(p.n_store % 4 == 0 && p.n_store == p.N, "gemm: split-K needs n_store == N, a multiple of 4");
    DN_CHECK(p.part && p.part_floats >= (size_t)g.split * p.M * p.n_store, "gemm: split-K workspace too small");
  }
  if (p.taps == 9)
    dispatch_frag<2>(p, g, s);
  else if (p.c1)
    dispatch_frag<1>(p, g, s);
  else
    dispatch_frag<0>(p, g, s);
}

}  // namespace dn
