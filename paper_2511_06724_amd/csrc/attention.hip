// Flash-style multi-head attention for the UNet transformer blocks (gfx950).
//
// O = softmax(Q K^T * scale) V per (sample, head), never materialising the
// score matrix: one workgroup = 4 waves = 128 queries of one (sample, head);
// key/value tiles of 64 rows are staged in LDS (K row-major, V transposed) and
// each wave runs an online softmax in fp32 over its 32 queries.
//
// The wave computes S^T = K Q^T with 32x32 MFMA so that each lane owns one
// query column of the score tile; the softmax row statistics are then a
// per-lane reduction plus one exchange with the partner lane (lane ^ 32), and
// the probabilities already sit in the B-operand layout of O^T = V^T P^T. The
// V^T operand is read with the key permutation that matches the accumulator
// layout, so no shuffle of P is needed.
#include "kernels.h"

namespace dn {
namespace {

constexpr int kKT = 64;  // keys per LDS tile

template <typename T> struct PvFrag;
template <> struct PvFrag<bf16> {
  // Keys of P registers [8c, 8c + 8) of a 32-key block for lane half h are
  // 16c + 4h + {0..3} and 16c + 8 + 4h + {0..3}: two 8-byte LDS reads.
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

template <typename T, int D>
__global__ __launch_bounds__(256) void attn_kernel(AttnParams p) {
  using MM = Mma<T>;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SK = D + VEC;                      // K tile row stride
  constexpr int SV = kKT + 8;                      // V^T row stride (keys)
  constexpr int NS = D / MM::KS;                   // MFMA steps over the head dim
  constexpr int DB = D / 32;                       // 32-row blocks of O^T
  constexpr int PCH = 16 / MM::KPL;                // MFMAs per 32-key block (P side)
  constexpr int VPR = D / VEC;                     // 16-byte vectors per key row

  __shared__ __align__(16) T Ks[kKT * SK];
  __shared__ __align__(16) T Vt[D * SV];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  const int b = blockIdx.z, h = blockIdx.y;
  const int q0 = blockIdx.x * 128 + wave * 32;

  const T* qp = static_cast<const T*>(p.q) + b * p.q_bs + h * D;
  const T* kp = static_cast<const T*>(p.k) + b * p.kv_bs + h * D;
  const T* vp = static_cast<const T*>(p.v) + b * p.kv_bs + h * D;

  const int qrow = min(q0 + (lane & 31), p.Sq - 1);
  typename MM::frag qf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) qf[s] = MM::load(qp + (long long)qrow * p.ldq + s * MM::KS + half * MM::KPL);

  f32x16 o[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int ntiles = (p.Skv + kKT - 1) / kKT;
  for (int t = 0; t < ntiles; ++t) {
    const int k0 = t * kKT;
    for (int i = tid; i < kKT * VPR; i += 256) {
      const int kr = i / VPR, vcol = i - (i / VPR) * VPR;
      const long long key = min(k0 + kr, p.Skv - 1);
      st16(&Ks[kr * SK + vcol * VEC], ld16(kp + key * p.ldk + vcol * VEC));
      const uint4 vv = ld16(vp + key * p.ldv + vcol * VEC);
      const T* ve = reinterpret_cast<const T*>(&vv);
#pragma unroll
      for (int e = 0; e < VEC; ++e) Vt[(vcol * VEC + e) * SV + kr] = ve[e];
    }
    __syncthreads();

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
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx * p.scale_log2);
    const float alpha = exp2f(m_run - m_new);
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = exp2f(sacc[kb][r] * p.scale_log2 - m_new);
        sacc[kb][r] = e;
        rs += e;
      }
    rs += __shfl_xor(rs, 32, 64);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[d][r] *= alpha;

#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        const typename MM::frag pf = PvFrag<T>::p(sacc[kb], c);
#pragma unroll
        for (int d = 0; d < DB; ++d)
          o[d] = MM::mma(PvFrag<T>::v(&Vt[(d * 32 + (lane & 31)) * SV], kb, c, half), pf, o[d]);
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
      for (int r = 0; r < 16; ++r) op[d * 32 + acc_row(r, lane)] = from_f32<T>(o[d][r] * inv);
  }
}

}  // namespace

template <typename T> void attention(const AttnParams& p, int D, hipStream_t s) {
  DN_CHECK(p.B >= 1 && p.heads >= 1 && p.Sq >= 1 && p.Skv >= 1, "attention: empty problem");
  DN_CHECK(D == 32 || D == 64, "attention: padded head dim must be 32 or 64");
  DN_CHECK(p.q && p.k && p.v && p.o, "attention: null operand");
  constexpr int VEC = 16 / sizeof(T);
  DN_CHECK(p.ldq % VEC == 0 && p.ldk % VEC == 0 && p.ldv % VEC == 0, "attention: strides must be 16-byte multiples");
  dim3 grid((p.Sq + 127) / 128, p.heads, p.B);
  if (D == 64)
    hipLaunchKernelGGL((attn_kernel<T, 64>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((attn_kernel<T, 32>), grid, dim3(256), 0, s, p);
  DN_HIP(hipGetLastError());
}

template void attention<float>(const AttnParams&, int, hipStream_t);
template void attention<bf16>(const AttnParams&, int, hipStream_t);

}  // namespace dn
