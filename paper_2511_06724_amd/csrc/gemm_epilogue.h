// Shared GEMM epilogue: bias, per-sample row vector, residual, output dtype,
// and the per-head transposed V output of the attention projections.
#pragma once

#include "kernels.h"

namespace dn {

template <typename T> struct OutVec;
template <> struct OutVec<bf16> {
  __device__ static __forceinline__ void store(bf16* p, const float v[4]) {
    bf16x4 o;
    o[0] = static_cast<bf16>(v[0]);
    o[1] = static_cast<bf16>(v[1]);
    o[2] = static_cast<bf16>(v[2]);
    o[3] = static_cast<bf16>(v[3]);
    *reinterpret_cast<bf16x4*>(p) = o;
  }
  __device__ static __forceinline__ void load(const bf16* p, float v[4]) {
    const bf16x4 i = *reinterpret_cast<const bf16x4*>(p);
    v[0] = static_cast<float>(i[0]);
    v[1] = static_cast<float>(i[1]);
    v[2] = static_cast<float>(i[2]);
    v[3] = static_cast<float>(i[3]);
  }
};
template <> struct OutVec<float> {
  __device__ static __forceinline__ void store(float* p, const float v[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
  __device__ static __forceinline__ void load(const float* p, float v[4]) {
    const float4 i = *reinterpret_cast<const float4*>(p);
    v[0] = i.x;
    v[1] = i.y;
    v[2] = i.z;
    v[3] = i.w;
  }
};

// Stores 4 consecutive output columns [n, n + 4) of row m (n % 4 == 0), masking
// columns >= n_store element-wise when the group straddles the edge.
template <typename T>
__device__ __forceinline__ void store4(const GemmParams& p, int m, int n, const float v[4], int n_store) {
  const long long o = (long long)m * p.ldo + n;
  const bool vec = n + 4 <= n_store && (p.ldo & 3) == 0;
  if (p.out_f32) {
    float* out = static_cast<float*>(p.out);
    if (vec) {
      OutVec<float>::store(out + o, v);
    } else {
      for (int e = 0; e < 4; ++e)
        if (n + e < n_store) out[o + e] = v[e];
    }
  } else {
    T* out = static_cast<T*>(p.out);
    if (vec) {
      OutVec<T>::store(out + o, v);
    } else {
      for (int e = 0; e < 4; ++e)
        if (n + e < n_store) out[o + e] = from_f32<T>(v[e]);
    }
  }
}

// v holds acc[m][n .. n + 3]: adds bias, the per-sample row vector and the
// residual, then stores; columns >= vt_col0 go to the transposed V buffer
// vt[sample][head][d][token] (row stride vt_ld) instead of `out`.
template <typename T> __device__ __forceinline__ void epilogue_group(const GemmParams& p, int m, int n, float v[4]) {
  if (n >= p.n_store) return;
  const bool full = n + 4 <= p.n_store;
  if (p.bias)
    for (int e = 0; e < 4; ++e) v[e] += (full || n + e < p.n_store) ? p.bias[n + e] : 0.f;
  if (p.rowvec) {
    const float* rv = p.rowvec + (long long)(m / p.rows_per_sample) * p.rowvec_ld + n;
    for (int e = 0; e < 4; ++e) v[e] += (full || n + e < p.n_store) ? rv[e] : 0.f;
  }
  if (p.resid) {
    const long long ro = (long long)m * p.ldr + n;
    if (full && (p.ldr & 3) == 0) {
      float r[4];
      if (p.resid_f32)
        OutVec<float>::load(static_cast<const float*>(p.resid) + ro, r);
      else
        OutVec<T>::load(static_cast<const T*>(p.resid) + ro, r);
      for (int e = 0; e < 4; ++e) v[e] += r[e];
    } else {
      for (int e = 0; e < 4; ++e)
        if (n + e < p.n_store)
          v[e] += p.resid_f32 ? static_cast<const float*>(p.resid)[ro + e]
                              : to_f32(static_cast<const T*>(p.resid)[ro + e]);
    }
  }
  if (p.vt && n >= p.vt_col0) {
    const int nn = n - p.vt_col0;
    const int h = nn / p.vt_dp, d = nn - h * p.vt_dp;
    const int b = m / p.vt_seq, s = m - b * p.vt_seq;
    T* dst = static_cast<T*>(p.vt) + (((long long)b * p.vt_heads + h) * p.vt_dp + d) * p.vt_ld + s;
    for (int e = 0; e < 4; ++e)
      if (n + e < p.n_store) dst[(long long)e * p.vt_ld] = from_f32<T>(v[e]);
    return;
  }
  store4<T>(p, m, n, v, p.n_store);
}

}  // namespace dn
