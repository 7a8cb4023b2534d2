// Shared device/host helpers of the denoise-loop library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <stdexcept>
#include <string>

namespace dn {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Library error carrying a dn_status code; caught at the C ABI.
struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};

#define DN_HIP(expr)                                                                          \
  do {                                                                                        \
    hipError_t e_ = (expr);                                                                   \
    if (e_ != hipSuccess)                                                                     \
      throw ::dn::Error(-3, std::string(#expr) + ": " + hipGetErrorString(e_) + " at " +      \
                                __FILE__ + ":" + std::to_string(__LINE__));                   \
  } while (0)

#define DN_CHECK(cond, msg)                                    \
  do {                                                         \
    if (!(cond)) throw ::dn::Error(-1, std::string(msg));      \
  } while (0)

// ---------------------------------------------------------------- element-type traits

template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kVec = 4;  // elements per 16-byte vector
};
template <> struct Elem<bf16> {
  static constexpr int kVec = 8;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }

// x * sigmoid(x) with the hardware reciprocal (about 1 ulp; no IEEE division sequence).
__device__ __forceinline__ float silu_f(float x) { return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }

// Exact-form GELU, x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)), with erf from
// Abramowitz & Stegun (1964) formula 7.1.26: |error| <= 1.5e-7 on the real line
// (one hardware reciprocal, one exponential, five FMAs instead of a library erf).
__device__ __forceinline__ float gelu_erf(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * z);
  const float poly = t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  const float e = 1.0f - poly * __expf(-z * z);  // erf(|x| / sqrt 2)
  return 0.5f * x * (1.0f + copysignf(e, x));
}

// Four floats -> four OCP E4M3 codes (nearest even) in one 32-bit word, byte e = value e.
// The hardware conversion turns magnitudes beyond the format into NaN codes, so values
// are clamped to +-448 first: the conversion then saturates.
__device__ __forceinline__ unsigned fp8x4(float a, float b, float c, float d) {
  const float lo = -448.f, hi = 448.f;
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(fminf(fmaxf(a, lo), hi), fminf(fmaxf(b, lo), hi), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(fminf(fmaxf(c, lo), hi), fminf(fmaxf(d, lo), hi), w, true);
  return static_cast<unsigned>(w);
}

// 16-byte vector load/store helpers.
__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

// Wave-wide (64 lanes) reductions.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// The same sum with DPP lane moves (no LDS crossbar round trips), wave-uniform result:
// quad butterflies, then the half-row and row mirrors give every lane its 16-lane row
// sum; row broadcasts of lane 15 and lane 31 fold the rows into lane 63, which is read
// back. A fixed association, so the result is deterministic.
template <int CTRL, int ROW_MASK> __device__ __forceinline__ float dpp_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK,
                                                                       0xf, false));
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
  v = dpp_add<0xb1, 0xf>(v);   // quad_perm [1, 0, 3, 2]
  v = dpp_add<0x4e, 0xf>(v);   // quad_perm [2, 3, 0, 1]
  v = dpp_add<0x141, 0xf>(v);  // row_half_mirror
  v = dpp_add<0x140, 0xf>(v);  // row_mirror
  v = dpp_add<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
  v = dpp_add<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

inline int ceil_div(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

}  // namespace dn

namespace dn {

// 32x32 MFMA tile operations for one element type. A wave computes
// C[32][32] += A[32][KS] * B[KS][32]; lane l supplies A row (l % 32) and
// B column (l % 32), k = KPL * (l / 32) .. + KPL - 1, and holds C column (l % 32),
// rows 8 * (r / 4) + 4 * (l / 32) + (r % 4) in accumulator register r.
template <typename T> struct Mma;
template <> struct Mma<bf16> {
  static constexpr int KS = 16;
  static constexpr int KPL = 8;
  typedef bf16x8 frag;
  __device__ static __forceinline__ frag load(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
  __device__ static __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  static constexpr int KS = 2;
  static constexpr int KPL = 1;
  typedef float frag;
  __device__ static __forceinline__ frag load(const float* p) { return *p; }
  __device__ static __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

}  // namespace dn
