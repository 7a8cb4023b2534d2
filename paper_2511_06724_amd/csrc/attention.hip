// Flash-style multi-head attention for the UNet transformer blocks (gfx950).
//
// O = softmax(Q K^T * scale) V per (sample, head), never materialising the
// score matrix. A workgroup holds 32 queries per wave; key tiles of 64 rows of K
// and the matching 64 columns of V^T (V stored transposed per head by the
// projection GEMM, so both tiles are row-contiguous) are double-buffered in LDS:
// the next tile's global loads are in flight while the current one is used.
//
// Each wave computes S^T = K Q^T with 32x32 MFMA so that a lane owns one query
// column: the softmax row statistics are a per-lane reduction plus one exchange
// with the partner lane (lane ^ 32), and the probabilities already sit in the
// B-operand layout of O^T = V^T P^T; the V^T operand is read with the key
// permutation of the accumulator layout (two 8-byte reads per fragment).
//
// Lazy rescaling: the reference maximum m of a row is only moved (and O, l
// rescaled by exp2(m_old - m_new)) when a tile's maximum exceeds it by more than
// 2^8 in the exponent; otherwise probabilities up to 2^8 are accumulated against
// the old reference. softmax(x) = exp(x - m) / sum exp(x - m) holds for any m, so
// this changes rounding only, and saves the O rescale on most tiles.
#include <algorithm>

#include "kernels.h"

namespace dn {
namespace {

constexpr int kKT = 64;          // keys per LDS tile
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;
// s_waitcnt immediate: vmcnt <= vm, lgkmcnt <= 0, expcnt unconstrained.
constexpr int attn_wait_vm_lgkm0(int vm) { return (vm & 0xF) | (((vm >> 4) & 3) << 14) | (7 << 4); }
constexpr float kLazy = 8.0f;    // log2 headroom before the reference max moves

// 2^x with the hardware exponential (v_exp_f32): arguments here are <= kLazy, and
// results below 2^-126 (flushed to zero) are far below bf16 / fp32 resolution of the
// row sums they join.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <typename T> struct PvFrag;
template <> struct PvFrag<bf16> {
  // P registers [8c, 8c + 8) of a 32-key block, lane half h, hold keys
  // 16c + 4h + {0..3} and 16c + 8 + 4h + {0..3}.
  __device__ static __forceinline__ bf16x8 v(const bf16* vt_row, int kb, int c, int h) {
    const bf16* base = vt_row + kb * 32 + 16 * c + 4 * h;
    const bf16x4 lo = *reinterpret_cast<const bf16x4*>(base);
    const bf16x4 hi = *reinterpret_cast<const bf16x4*>(base + 8);
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
  }
  __device__ static __forceinline__ bf16x8 p(const f32x16& s, int c) {
    bf16x8 r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = static_cast<bf16>(s[8 * c + e]);
    return r;
  }
};
template <> struct PvFrag<float> {
  // Register c of a 32-key block belongs to key 8 (c / 4) + 4h + (c % 4).
  __device__ static __forceinline__ float v(const float* vt_row, int kb, int c, int h) {
    return vt_row[kb * 32 + 8 * (c >> 2) + 4 * h + (c & 3)];
  }
  __device__ static __forceinline__ float p(const f32x16& s, int c) { return s[c]; }
};

template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) void attn_kernel(AttnParams p) {
  using MM = Mma<T>;
  constexpr int NT = 64 * NW;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SK = D + VEC;                      // K tile row stride (elements)
  constexpr int SV = kKT + VEC;                    // V^T tile row stride (keys)
  constexpr int NS = D / MM::KS;                   // MFMA steps over the head dim
  constexpr int DB = D / 32;                       // 32-row blocks of O^T
  constexpr int PCH = 16 / MM::KPL;                // MFMAs per 32-key block (P side)
  constexpr int KV_VEC = kKT * D / VEC;            // 16-byte vectors per K tile (= per V^T tile)
  constexpr int PER_T = (2 * KV_VEC + NT - 1) / NT;
  constexpr int STAGE = kKT * SK + D * SV;

  extern __shared__ __align__(16) unsigned char attn_smem[];
  T* lds = reinterpret_cast<T*>(attn_smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  const int b = blockIdx.z, h = blockIdx.y;
  const int q0 = blockIdx.x * (32 * NW) + wave * 32;

  const T* qp = static_cast<const T*>(p.q) + b * p.q_bs + h * D;
  const T* kp = static_cast<const T*>(p.k) + b * p.k_bs + h * D;
  const T* vtp = static_cast<const T*>(p.vt) + ((long long)b * p.heads + h) * D * p.vt_ld;

  const int qrow = min(q0 + (lane & 31), p.Sq - 1);
  typename MM::frag qf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) qf[s] = MM::load(qp + (long long)qrow * p.ldq + s * MM::KS + half * MM::KPL);

  f32x16 o[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.f;
  float m_ref = -INFINITY, l_run = 0.f;

  uint4 reg[PER_T];
  auto load = [&](int t) {
    const int k0 = t * kKT;
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int v = tid + i * NT;
      if (v < KV_VEC) {  // K row (key) kr, vector kc
        const int kr = v / (D / VEC), kc = v - (v / (D / VEC)) * (D / VEC);
        const long long key = min(k0 + kr, p.Skv - 1);
        reg[i] = ld16(kp + key * p.ldk + kc * VEC);
      } else if (v < 2 * KV_VEC) {  // V^T row d, keys [k0 + kc*VEC, +VEC)
        const int w = v - KV_VEC;
        const int d = w / (kKT / VEC), kc = w - (w / (kKT / VEC)) * (kKT / VEC);
        reg[i] = ld16(vtp + (long long)d * p.vt_ld + k0 + kc * VEC);
      }
    }
  };
  auto store = [&](int buf) {
    T* Ks = lds + buf * STAGE;
    T* Vt = Ks + kKT * SK;
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int v = tid + i * NT;
      if (v < KV_VEC) {
        const int kr = v / (D / VEC), kc = v - (v / (D / VEC)) * (D / VEC);
        st16(Ks + kr * SK + kc * VEC, reg[i]);
      } else if (v < 2 * KV_VEC) {
        const int w = v - KV_VEC;
        const int d = w / (kKT / VEC), kc = w - (w / (kKT / VEC)) * (kKT / VEC);
        st16(Vt + d * SV + kc * VEC, reg[i]);
      }
    }
  };

  const int ntiles = (p.Skv + kKT - 1) / kKT;
  load(0);
  store(0);
  if (ntiles > 1) load(1);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int k0 = t * kKT;
    const T* Ks = lds + (t & 1) * STAGE;
    const T* Vt = Ks + kKT * SK;

    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        sacc[kb] = MM::mma(MM::load(&Ks[(kb * 32 + (lane & 31)) * SK + s * MM::KS + half * MM::KPL]), qf[s],
                           sacc[kb]);

    if (k0 + kKT > p.Skv) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (k0 + kb * 32 + acc_row(r, lane) >= p.Skv) sacc[kb][r] = -INFINITY;
    }

    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * p.scale_log2;
    if (__any(mx > m_ref + kLazy)) {
      const float m_new = fmaxf(m_ref, mx);
      const float alpha = fast_exp2(m_ref - m_new);
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[d][r] *= alpha;
      m_ref = m_new;
    }
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = fast_exp2(sacc[kb][r] * p.scale_log2 - m_ref);
        sacc[kb][r] = e;
        rs += e;
      }
    l_run += rs + __shfl_xor(rs, 32, 64);

#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        const typename MM::frag pf = PvFrag<T>::p(sacc[kb], c);
#pragma unroll
        for (int d = 0; d < DB; ++d)
          o[d] = MM::mma(PvFrag<T>::v(&Vt[(d * 32 + (lane & 31)) * SV], kb, c, half), pf, o[d]);
      }

    if (t + 1 < ntiles) {
      store((t + 1) & 1);
      if (t + 2 < ntiles) load(t + 2);
    }
    __syncthreads();
  }

  const int qi = q0 + (lane & 31);
  if (qi < p.Sq) {
    const float inv = 1.f / l_run;
    T* op = static_cast<T*>(p.o) + b * p.o_bs + (long long)qi * p.ldo + h * D;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = o[d][4 * g + e] * inv;
        T* dst = op + d * 32 + 8 * g + 4 * half;
#pragma unroll
        for (int e = 0; e < 4; ++e) dst[e] = from_f32<T>(v[e]);
      }
  }
}

// ---------------------------------------------------------------------------
// bf16, head dim 64: direct-to-LDS variant for long key ranges.
//
// Same math as attn_kernel, organised like the direct-to-LDS GEMM:
//  - a workgroup covers NQ x 32 queries of one (sample, head); workgroup ids are
//    mapped so that consecutive ids of one XCD walk the query tiles of the same
//    heads, which keeps those heads' K / V^T in that XCD's L2;
//  - NQ query groups of 32 x NK key groups of waves: wave (wq, wk) takes queries
//    [q0 + 32 wq, +32) and, of every NK consecutive key tiles (a tile group), tile
//    wk; the NK partial softmax states (reference max, row sum, unnormalised O) of a
//    query group are merged through LDS at the end (twice the waves of a one-pass
//    kernel for the same queries);
//  - key tiles of 64 (K rows of 128 bytes and the 64 V^T rows of 64 keys, 16 KB)
//    go global -> LDS with global_load_lds_dwordx4 into a ring of kRing tile
//    groups: a hand-over retires one group and refills its slots with the group
//    kRing ahead; past the last group the last one is loaded again (the same count
//    of loads per hand-over; nothing reads it);
//  - 128-byte LDS rows without padding, chunk c of row r at c ^ f(r),
//    f(r) = (r & 7) ^ ((r >> 3) & 1) (conflict-free 16-byte fragment reads);
//  - every K fragment of a tile is read before the S MFMAs, every V^T fragment
//    before the PV MFMAs; row max and sum use independent partial reductions.
constexpr int kRing = 2;  // ring depth in tile groups

template <int NQ, int NK>
__global__ __launch_bounds__(64 * NQ * NK) void attn_dma_kernel(AttnParams p, int qtiles) {
  constexpr int NW = NQ * NK;
  constexpr int D = 64;
  constexpr int ROWB = 128;                  // bytes per LDS row (64 bf16)
  constexpr int TILE = 2 * kKT * ROWB;       // K tile then V^T tile (16 KB)
  constexpr int TI = 2 * kKT / 8;            // DMA instructions per tile (8 rows each)
  constexpr int PW = NK * TI / NW;           // per wave per hand-over
  static_assert((NK * TI) % NW == 0, "DMA instructions must divide over the waves");

  extern __shared__ __align__(16) unsigned char smem[];

  // ---- (query tile, head, sample) of this workgroup, XCD-contiguous
  const int total = qtiles * p.heads * p.B;
  const int wg = blockIdx.x;
  const int xcd = wg % 8, idx = wg / 8;
  const int base = total / 8, rem = total % 8;
  const int logical = xcd * base + min(xcd, rem) + idx;
  const int qt = logical % qtiles;
  const int bh = logical / qtiles;
  const int h = bh % p.heads, b = bh / p.heads;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wq = wave % NQ, wk = wave / NQ;
  const int half = lane >> 5;
  const int q0 = qt * (32 * NQ) + wq * 32;

  const bf16* qp = static_cast<const bf16*>(p.q) + b * p.q_bs + h * D;
  const bf16* kp = static_cast<const bf16*>(p.k) + b * p.k_bs + h * D;
  const bf16* vtp = static_cast<const bf16*>(p.vt) + ((long long)b * p.heads + h) * D * p.vt_ld;

  bf16x8 qf[4];
  {
    const int qrow = min(q0 + (lane & 31), p.Sq - 1);
#pragma unroll
    for (int s = 0; s < 4; ++s)
      qf[s] = *reinterpret_cast<const bf16x8*>(qp + (long long)qrow * p.ldq + s * 16 + half * 8);
  }

  // ---- DMA: instruction j of this wave fills rows [8 r, 8 r + 8) of tile (i / TI) of the
  // group, r = i % TI, i = wave * PW + j (rows 0..63: keys of K, 64..127: V^T head dims);
  // the lane fetches logical chunk (lane & 7) ^ f(row). Groups past the last one load
  // the last group again (same count of loads per hand-over; nothing reads them).
  const int lrow = lane >> 3;
  const int ntiles = (p.Skv + kKT - 1) / kKT;
  const int ngroups = (ntiles + NK - 1) / NK;
  auto issue = [&](int grp_in, int gslot) {
    const int grp = min(grp_in, ngroups - 1);
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int i = wave * PW + j;
      const int tt = i / TI, r = i % TI;
      const int t = min(grp * NK + tt, ntiles - 1);
      const int k0 = t * kKT;
      const int row = 8 * r + lrow;
      const int lc = ((lane & 7) ^ lrow ^ (r & 1)) * 8;
      const bf16* g;
      if (r < kKT / 8) {
        const int key = min(k0 + row, p.Skv - 1);
        g = kp + (long long)key * p.ldk + lc;
      } else {
        g = vtp + (long long)(row - kKT) * p.vt_ld + k0 + lc;
      }
      __builtin_amdgcn_global_load_lds((gbl_void_t*)g,
                                       (lds_void_t*)(smem + (gslot * NK + tt) * TILE + r * 1024), 16, 0, 0);
    }
  };

  const int frow = lane & 31;
  const int fs = (lane & 7) ^ ((lane >> 3) & 1);

  f32x16 o[2];
#pragma unroll
  for (int d = 0; d < 2; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.f;
  float m_ref = -INFINITY, l_run = 0.f;

#pragma unroll
  for (int g = 0; g < kRing; ++g) issue(g, g);
  __builtin_amdgcn_s_waitcnt(attn_wait_vm_lgkm0((kRing - 1) * PW));
  __builtin_amdgcn_s_barrier();

  int gslot = 0;
  for (int grp = 0; grp < ngroups; ++grp) {
    const int t = grp * NK + wk;
    if (t < ntiles) {
      const int k0 = t * kKT;
      const unsigned char* Ks = smem + (gslot * NK + wk) * TILE;
      const unsigned char* Vs = Ks + kKT * ROWB;

      // S^T = K Q^T for 64 keys (two 32-key blocks): every K fragment first
      bf16x8 kf[2][4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          kf[kb][s] = *reinterpret_cast<const bf16x8*>(Ks + (kb * 32 + frow) * ROWB + ((2 * s + half) ^ fs) * 16);
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kb][s], qf[s], sacc[kb], 0, 0, 0);

      // V^T fragments: keys in the accumulator order of P (two 8-byte reads each)
      bf16x8 vf[2][2][2];
#pragma unroll
      for (int d = 0; d < 2; ++d)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const int lo = 4 * kb + 2 * c;
            const unsigned char* row = Vs + (d * 32 + frow) * ROWB + 8 * half;
            const bf16x4 a = *reinterpret_cast<const bf16x4*>(row + ((lo ^ fs) * 16));
            const bf16x4 bq = *reinterpret_cast<const bf16x4*>(row + (((lo + 1) ^ fs) * 16));
            bf16x8 v;
            v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
            v[4] = bq[0]; v[5] = bq[1]; v[6] = bq[2]; v[7] = bq[3];
            vf[d][kb][c] = v;
          }

      if (k0 + kKT > p.Skv) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (k0 + kb * 32 + acc_row(r, lane) >= p.Skv) sacc[kb][r] = -INFINITY;
      }

      // row max: four independent partial maxima, then the partner lane
      float mp[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        mp[i] = fmaxf(fmaxf(fmaxf(sacc[0][i], sacc[0][4 + i]), fmaxf(sacc[0][8 + i], sacc[0][12 + i])),
                      fmaxf(fmaxf(sacc[1][i], sacc[1][4 + i]), fmaxf(sacc[1][8 + i], sacc[1][12 + i])));
      float mx = fmaxf(fmaxf(mp[0], mp[1]), fmaxf(mp[2], mp[3]));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * p.scale_log2;
      if (__any(mx > m_ref + kLazy)) {
        const float m_new = fmaxf(m_ref, mx);
        const float alpha = fast_exp2(m_ref - m_new);
        l_run *= alpha;
#pragma unroll
        for (int d = 0; d < 2; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[d][r] *= alpha;
        m_ref = m_new;
      }
      bf16x8 pf[2][2];
      float sp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          bf16x8 pv;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float ex = fast_exp2(sacc[kb][8 * c + e] * p.scale_log2 - m_ref);
            sp[e & 3] += ex;
            pv[e] = static_cast<bf16>(ex);
          }
          pf[kb][c] = pv;
        }
      const float rs = (sp[0] + sp[1]) + (sp[2] + sp[3]);
      l_run += rs + __shfl_xor(rs, 32, 64);

      // O^T += V^T P^T
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int d = 0; d < 2; ++d)
            o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[d][kb][c], pf[kb][c], o[d], 0, 0, 0);
    }

    // hand-over: group grp + 1 (the last one issued) must have landed; after the barrier
    // every wave is done with group grp's slots, which take group grp + kRing
    __builtin_amdgcn_s_waitcnt(attn_wait_vm_lgkm0((kRing - 2) * PW));
    __builtin_amdgcn_s_barrier();
    issue(grp + kRing, gslot);
    gslot = gslot + 1 == kRing ? 0 : gslot + 1;
  }
  __builtin_amdgcn_s_waitcnt(attn_wait_vm_lgkm0(0));
  __builtin_amdgcn_s_barrier();

  // ---- merge the NK partial states of each query group (slots reused as scratch:
  // per wave 64 lanes x 34 floats)
  float* xch = reinterpret_cast<float*>(smem);
  if (NK > 1) {
    if (wk > 0) {
      float* dst = xch + ((wk - 1) * NQ + wq) * 64 * 34 + lane;
#pragma unroll
      for (int d = 0; d < 2; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) dst[(d * 16 + r) * 64] = o[d][r];
      dst[32 * 64] = m_ref;
      dst[33 * 64] = l_run;
    }
    __syncthreads();
    if (wk == 0) {
#pragma unroll
      for (int k = 1; k < NK; ++k) {
        const float* src = xch + ((k - 1) * NQ + wq) * 64 * 34 + lane;
        const float m2 = src[32 * 64], l2 = src[33 * 64];
        const float m_new = fmaxf(m_ref, m2);
        const float a1 = m_ref == -INFINITY ? 0.f : fast_exp2(m_ref - m_new);
        const float a2 = m2 == -INFINITY ? 0.f : fast_exp2(m2 - m_new);
        l_run = l_run * a1 + l2 * a2;
#pragma unroll
        for (int d = 0; d < 2; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[d][r] = o[d][r] * a1 + src[(d * 16 + r) * 64] * a2;
        m_ref = m_new;
      }
    }
  }

  const int qi = q0 + (lane & 31);
  if (wk == 0 && qi < p.Sq) {
    const float inv = 1.f / l_run;
    bf16* op = static_cast<bf16*>(p.o) + b * p.o_bs + (long long)qi * p.ldo + h * D;
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(o[d][4 * g + e] * inv);
        *reinterpret_cast<bf16x4*>(op + d * 32 + 8 * g + 4 * half) = v;
      }
  }
}

template <int NQ, int NK> void launch_dma(const AttnParams& p, hipStream_t s) {
  constexpr int TILE = 2 * kKT * 128;
  const size_t lds = std::max(size_t(kRing) * NK * TILE, size_t(NK - 1) * NQ * 64 * 34 * 4);
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_dma_kernel<NQ, NK>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  const int qtiles = (p.Sq + 32 * NQ - 1) / (32 * NQ);
  hipLaunchKernelGGL((attn_dma_kernel<NQ, NK>), dim3(qtiles * p.heads * p.B), dim3(64 * NQ * NK), lds, s, p, qtiles);
}

template <typename T, int D, int NW> void launch(dim3 grid, const AttnParams& p, hipStream_t s) {
  constexpr int VEC = 16 / sizeof(T);
  const size_t lds = size_t(2) * (kKT * (D + VEC) + D * (kKT + VEC)) * sizeof(T);
  static bool attr_set = false;
  if (!attr_set) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<T, D, NW>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr_set = true;
  }
  hipLaunchKernelGGL((attn_kernel<T, D, NW>), grid, dim3(64 * NW), lds, s, p);
}

}  // namespace

template <typename T> void attention(const AttnParams& p, int D, hipStream_t s) {
  DN_CHECK(p.B >= 1 && p.heads >= 1 && p.Sq >= 1 && p.Skv >= 1, "attention: empty problem");
  DN_CHECK(D == 32 || D == 64, "attention: padded head dim must be 32 or 64");
  DN_CHECK(p.q && p.k && p.vt && p.o, "attention: null operand");
  constexpr int VEC = 16 / sizeof(T);
  DN_CHECK(p.ldq % VEC == 0 && p.ldk % VEC == 0 && p.vt_ld % VEC == 0, "attention: strides must be 16-byte multiples");
  DN_CHECK(p.vt_ld >= (p.Skv + kKT - 1) / kKT * kKT, "attention: V^T rows must cover whole 64-key tiles");
  // bf16 self-attention over long key ranges: the direct-to-LDS kernel with the key
  // range split over two wave groups (4 x 32 queries per workgroup for long query
  // ranges, 2 x 32 otherwise); short key ranges (cross-attention) keep the
  // register-staged kernel below, whose single pass has no merge step.
  if (sizeof(T) == 2 && D == 64 && p.Skv >= 256) {
    if (p.Sq >= 2048)
      launch_dma<4, 2>(p, s);
    else
      launch_dma<2, 2>(p, s);
    DN_HIP(hipGetLastError());
    return;
  }
  // Fewer, wider workgroups when there are many queries; two waves per workgroup
  // otherwise, so that short sequences still spread over every CU.
  const long long wg4 = (long long)((p.Sq + 127) / 128) * p.heads * p.B;
  if (wg4 >= 512) {
    dim3 grid((p.Sq + 127) / 128, p.heads, p.B);
    if (D == 64)
      launch<T, 64, 4>(grid, p, s);
    else
      launch<T, 32, 4>(grid, p, s);
  } else {
    dim3 grid((p.Sq + 63) / 64, p.heads, p.B);
    if (D == 64)
      launch<T, 64, 2>(grid, p, s);
    else
      launch<T, 32, 2>(grid, p, s);
  }
  DN_HIP(hipGetLastError());
}

template void attention<float>(const AttnParams&, int, hipStream_t);
template void attention<bf16>(const AttnParams&, int, hipStream_t);

}  // namespace dn
