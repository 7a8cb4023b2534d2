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
#include "kernels.h"

namespace dn {
namespace {

constexpr int kKT = 64;          // keys per LDS tile
constexpr float kLazy = 8.0f;    // log2 headroom before the reference max moves

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
      const float alpha = exp2f(m_ref - m_new);
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
        const float e = exp2f(sacc[kb][r] * p.scale_log2 - m_ref);
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
