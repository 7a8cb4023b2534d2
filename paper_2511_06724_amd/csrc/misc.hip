// Small kernels of the denoise loop: noise schedule, timestep embedding,
// guidance + DDIM update, layout conversions and weight packing (gfx950).
#include "kernels.h"

namespace dn {
namespace {

// abar_t = prod_{i <= t} (1 - beta_i) in fp64; linear or scaled-linear betas.
__global__ void abar_kernel(double* abar, int T, double b0, double b1, int schedule) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double prod = 1.0;
  for (int i = 0; i < T; ++i) {
    const double f = T > 1 ? (double)i / (double)(T - 1) : 0.0;
    double beta;
    if (schedule == 0) {
      beta = b0 + (b1 - b0) * f;
    } else {
      const double r = sqrt(b0) + (sqrt(b1) - sqrt(b0)) * f;
      beta = r * r;
    }
    prod *= 1.0 - beta;
    abar[i] = prod;
  }
}

// Sinusoidal timestep features: with half = dim / 2 and f_j = exp(-ln(10000) j / half),
// out[s] = [cos(t_s f_j) for j] ++ [sin(t_s f_j) for j]; evaluated in fp64.
__global__ void sinusoid_kernel(float* out, TsChunk ts, int dim) {
  const int half = dim / 2;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= ts.count * half) return;
  const int s = i / half, j = i - (i / half) * half;
  const double f = exp(-log(10000.0) * (double)j / (double)half);
  const double a = (double)ts.t[s] * f;
  out[(long long)s * dim + j] = (float)cos(a);
  out[(long long)s * dim + half + j] = (float)sin(a);
}

// out[s][j] = sum_k act(in[s][k]) * w[j][k] + b[j]: one wave per output row j,
// the row of w held in registers while the S input rows stream past.
constexpr int kSkinnyMaxK = 64 * 32;
__global__ __launch_bounds__(256) void skinny_kernel(const float* in, int S, int K, const float* w, const float* b,
                                                     int J, float* out, int ld_out, int silu) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= J) return;
  float wr[kSkinnyMaxK / 64];
#pragma unroll
  for (int i = 0; i < kSkinnyMaxK / 64; ++i) {
    const int k = lane + 64 * i;
    wr[i] = k < K ? w[(long long)j * K + k] : 0.f;
  }
  const float bj = b ? b[j] : 0.f;
  for (int s = 0; s < S; ++s) {
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < kSkinnyMaxK / 64; ++i) {
      const int k = lane + 64 * i;
      if (k < K) {
        float v = in[(long long)s * K + k];
        if (silu) v = silu_f(v);
        acc += v * wr[i];
      }
    }
    acc = wave_sum(acc);
    if (lane == 0) out[(long long)s * ld_out + j] = acc + bj;
  }
}

// latent NCHW fp32 [B][C][HW] -> UNet input NHWC [2B][HW][Cpad] (both guidance
// halves get the same latent; channels >= C are zero).
template <typename T>
__global__ void latent_to_input_kernel(const float* lat, T* xin, int B, int C, int HW, int Cpad) {
  const long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (i >= (long long)B * HW) return;
  const int b = static_cast<int>(i / HW), px = static_cast<int>(i - (long long)(i / HW) * HW);
  T* o0 = xin + ((long long)b * HW + px) * Cpad;
  T* o1 = xin + ((long long)(B + b) * HW + px) * Cpad;
  for (int c = 0; c < Cpad; ++c) {
    const T v = from_f32<T>(c < C ? lat[((long long)b * C + c) * HW + px] : 0.f);
    o0[c] = v;
    o1[c] = v;
  }
}

// Guidance + DDIM (eta = 0) on one latent pixel, all channels. eps is the UNet
// output NHWC fp32 [2B][HW][C] (unconditional rows first). abar_t and abar_prev
// come from the fp64 table (t = -1: abar = 1) and the update is evaluated as
//   x0 = (x - sqrt(1 - abar_t) eps) / sqrt(abar_t);  x = sqrt(abar_prev) x0 + sqrt(1 - abar_prev) eps
// with the coefficients in fp64 and the arithmetic on x and eps in fp32.
template <typename T>
__global__ void cfg_ddim_kernel(const float* eps, float* lat, T* xin, const double* abar, int t, int t_prev,
                                float scale, int B, int C, int HW, int Cpad) {
  const long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (i >= (long long)B * HW) return;
  const int b = static_cast<int>(i / HW), px = static_cast<int>(i - (long long)(i / HW) * HW);
  const double at = t < 0 ? 1.0 : abar[t];
  const double ap = t_prev < 0 ? 1.0 : abar[t_prev];
  const float s1t = (float)sqrt(1.0 - at), rst = (float)(1.0 / sqrt(at));
  const float sp = (float)sqrt(ap), s1p = (float)sqrt(1.0 - ap);
  for (int c = 0; c < C; ++c) {
    const float eu = eps[((long long)b * HW + px) * C + c];
    const float ec = eps[((long long)(B + b) * HW + px) * C + c];
    const float e = eu + scale * (ec - eu);
    float* xp = lat + ((long long)b * C + c) * HW + px;
    const float x0 = (*xp - s1t * e) * rst;
    const float xn = sp * x0 + s1p * e;
    *xp = xn;
    if (xin) {
      const T v = from_f32<T>(xn);
      xin[((long long)b * HW + px) * Cpad + c] = v;
      xin[((long long)(B + b) * HW + px) * Cpad + c] = v;
    }
  }
}

// UNet output NHWC [2B][HW][C] -> raw NCHW [2B][C][HW] and guided NCHW [B][C][HW].
__global__ void export_eps_kernel(const float* eps, float* raw, float* guided, float scale, int B, int C, int HW) {
  const long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (i >= (long long)2 * B * HW) return;
  const int n = static_cast<int>(i / HW), px = static_cast<int>(i - (long long)(i / HW) * HW);
  for (int c = 0; c < C; ++c) {
    const float v = eps[((long long)n * HW + px) * C + c];
    raw[((long long)n * C + c) * HW + px] = v;
    if (guided && n < B) {
      const float vc = eps[((long long)(B + n) * HW + px) * C + c];
      guided[((long long)n * C + c) * HW + px] = v + scale * (vc - v);
    }
  }
}

template <typename T> __global__ void convert_kernel(const float* src, T* dst, long long n) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x)
    dst[i] = from_f32<T>(src[i]);
}

__global__ void bf16_to_f32_kernel(const uint16_t* src, float* dst, long long n) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x)
    dst[i] = __uint_as_float(static_cast<uint32_t>(src[i]) << 16);
}

// Source row of packed row r (or -1 for a zero row).
__device__ __forceinline__ long long pack_src_row(const PackParams& p, int r) {
  if (p.row_mode == 1) {  // GEGLU: 32-row blocks alternate value / gate
    const int half = p.src_rows / 2;
    const int blk = r / 64, w = r - blk * 64;
    return w < 32 ? (long long)blk * 32 + w : (long long)half + blk * 32 + (w - 32);
  }
  if (p.row_mode == 2) {  // head padding: head h rows [h*Dp, h*Dp + D) <- source [h*D, h*D + D)
    const int h = r / p.Dp, d = r - h * p.Dp;
    return d < p.D ? (long long)h * p.D + d : -1;
  }
  return r < p.src_rows ? r : -1;
}

template <typename T> __global__ void pack_kernel(PackParams p) {
  const long long total = (long long)p.rows * p.cols;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const int r = static_cast<int>(i / p.cols), c = static_cast<int>(i - (long long)(i / p.cols) * p.cols);
    const long long sr = pack_src_row(p, r);
    float v = 0.f;
    if (sr >= 0) {
      if (p.col_mode == 0) {
        if (c < p.src_cols) v = p.src[sr * p.src_cols + c];
      } else if (p.col_mode == 1) {
        const int h = c / p.Dp, d = c - h * p.Dp;
        if (d < p.D) v = p.src[sr * p.src_cols + (long long)h * p.D + d];
      } else {  // conv3x3: packed column = tap * Cinp + ci <- source [r][ci][ky][kx]
        const int tap = c / p.Cinp, ci = c - tap * p.Cinp;
        if (ci < p.Cin) v = p.src[(sr * p.Cin + ci) * 9 + tap];
      }
    }
    long long o = (long long)r * p.ld_dst + c;
    if (p.frag) {  // fragment order of a [rows][cols] matrix, see gemm_frag.hip
      const int lane = (r & 31) + 32 * ((c & 15) >> 3);
      o = ((long long)(r >> 5) * (p.cols >> 4) + (c >> 4)) * 512 + lane * 8 + (c & 7);
    }
    static_cast<T*>(p.dst)[o] = from_f32<T>(v);
  }
}

// One workgroup per destination row r of the fp8 matrix: the row's largest magnitude,
// its scale, then every code at its fragment position (see pack_fp8 in kernels.h):
// byte ((r / 32) * (cols / 64) + c / 64) * 2048 + (r % 32 + 32 * ((c % 64) / 32)) * 32 + c % 32.
__global__ __launch_bounds__(256) void pack_fp8_kernel(PackParams p, float* scales, int rows_pad) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const long long sr = r < p.rows ? pack_src_row(p, r) : -1;
  const float* src = sr >= 0 ? p.src + sr * p.src_cols : nullptr;
  float m = 0.f;
  if (src)
    for (int c = threadIdx.x; c < p.src_cols; c += 256) m = fmaxf(m, fabsf(src[c]));
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float s = m > 0.f ? m / 448.f : 1.f;  // IEEE division, as the scale is defined
  if (threadIdx.x == 0) scales[r] = s;
  uint8_t* dst = static_cast<uint8_t*>(p.dst);
  const long long kst = p.cols / 64;
  for (int c4 = threadIdx.x * 4; c4 < p.cols; c4 += 1024) {
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (src)
      for (int e = 0; e < 4; ++e)
        if (c4 + e < p.src_cols) v[e] = src[c4 + e] / s;
    const long long o = ((long long)(r >> 5) * kst + c4 / 64) * 2048 + ((r & 31) + 32 * ((c4 & 63) >> 5)) * 32 + (c4 & 31);
    *reinterpret_cast<unsigned*>(dst + o) = fp8x4(v[0], v[1], v[2], v[3]);
  }
}

__global__ void pack_bias_kernel(float* dst, int n, const float* src, int src_n, int row_mode, int D, int Dp) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  PackParams p;
  p.row_mode = row_mode;
  p.src_rows = src_n;
  p.D = D;
  p.Dp = Dp;
  const long long sr = pack_src_row(p, r);
  dst[r] = sr >= 0 ? src[sr] : 0.f;
}

inline int blocks_for(long long n, int per = 256, int cap = 16384) {
  const long long b = (n + per - 1) / per;
  return static_cast<int>(b < 1 ? 1 : (b > cap ? cap : b));
}

}  // namespace

void abar_table(double* abar, int T, double beta_start, double beta_end, int schedule, hipStream_t s) {
  hipLaunchKernelGGL(abar_kernel, dim3(1), dim3(64), 0, s, abar, T, beta_start, beta_end, schedule);
  DN_HIP(hipGetLastError());
}

void sinusoid(float* out, const TsChunk& c, int dim, hipStream_t s) {
  const int n = c.count * (dim / 2);
  hipLaunchKernelGGL(sinusoid_kernel, dim3(blocks_for(n)), dim3(256), 0, s, out, c, dim);
  DN_HIP(hipGetLastError());
}

void skinny_linear(const float* in, int S, int K, const float* w, const float* b, int J, float* out, int ld_out,
                   int silu, hipStream_t s) {
  DN_CHECK(K <= kSkinnyMaxK, "skinny_linear: K too large");
  hipLaunchKernelGGL(skinny_kernel, dim3((J + 3) / 4), dim3(256), 0, s, in, S, K, w, b, J, out, ld_out, silu);
  DN_HIP(hipGetLastError());
}

template <typename T>
void latent_to_input(const float* latent, T* xin, int B, int C, int HW, int Cpad, hipStream_t s) {
  hipLaunchKernelGGL(latent_to_input_kernel<T>, dim3(blocks_for((long long)B * HW)), dim3(256), 0, s, latent, xin, B,
                     C, HW, Cpad);
  DN_HIP(hipGetLastError());
}

template <typename T>
void cfg_ddim(const float* eps, float* latent, T* xin, const double* abar, int t, int t_prev, float scale, int B,
              int C, int HW, int Cpad, hipStream_t s) {
  hipLaunchKernelGGL(cfg_ddim_kernel<T>, dim3(blocks_for((long long)B * HW)), dim3(256), 0, s, eps, latent, xin, abar,
                     t, t_prev, scale, B, C, HW, Cpad);
  DN_HIP(hipGetLastError());
}

void export_eps(const float* eps, float* raw, float* guided, float scale, int B, int C, int HW, hipStream_t s) {
  hipLaunchKernelGGL(export_eps_kernel, dim3(blocks_for(2ll * B * HW)), dim3(256), 0, s, eps, raw, guided, scale, B, C,
                     HW);
  DN_HIP(hipGetLastError());
}

template <typename T> void convert_from_f32(const float* src, T* dst, long long n, hipStream_t s) {
  hipLaunchKernelGGL(convert_kernel<T>, dim3(blocks_for(n)), dim3(256), 0, s, src, dst, n);
  DN_HIP(hipGetLastError());
}

void bf16_latent_to_f32(const uint16_t* src, float* dst, long long n, hipStream_t s) {
  hipLaunchKernelGGL(bf16_to_f32_kernel, dim3(blocks_for(n)), dim3(256), 0, s, src, dst, n);
  DN_HIP(hipGetLastError());
}

template <typename T> void pack(const PackParams& p, hipStream_t s) {
  hipLaunchKernelGGL(pack_kernel<T>, dim3(blocks_for((long long)p.rows * p.cols)), dim3(256), 0, s, p);
  DN_HIP(hipGetLastError());
}

void pack_fp8(const PackParams& p, float* scales, hipStream_t s) {
  DN_CHECK(p.col_mode == 0 && p.cols % 128 == 0 && p.src_cols <= p.cols, "pack_fp8: columns must be a multiple of 128");
  const int rows_pad = (p.rows + 31) / 32 * 32;
  hipLaunchKernelGGL(pack_fp8_kernel, dim3(rows_pad), dim3(256), 0, s, p, scales, rows_pad);
  DN_HIP(hipGetLastError());
}

void pack_bias(float* dst, int n, const float* src, int src_n, int row_mode, int D, int Dp, hipStream_t s) {
  hipLaunchKernelGGL(pack_bias_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, n, src, src_n, row_mode, D, Dp);
  DN_HIP(hipGetLastError());
}

template void latent_to_input<float>(const float*, float*, int, int, int, int, hipStream_t);
template void latent_to_input<bf16>(const float*, bf16*, int, int, int, int, hipStream_t);
template void cfg_ddim<float>(const float*, float*, float*, const double*, int, int, float, int, int, int, int,
                              hipStream_t);
template void cfg_ddim<bf16>(const float*, float*, bf16*, const double*, int, int, float, int, int, int, int,
                             hipStream_t);
template void convert_from_f32<float>(const float*, float*, long long, hipStream_t);
template void convert_from_f32<bf16>(const float*, bf16*, long long, hipStream_t);
template void pack<float>(const PackParams&, hipStream_t);
template void pack<bf16>(const PackParams&, hipStream_t);

}  // namespace dn
