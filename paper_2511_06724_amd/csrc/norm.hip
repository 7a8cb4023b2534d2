// GroupNorm (+SiLU) and LayerNorm kernels (HBM-bound; gfx950).
//
// GroupNorm on NHWC activations runs in three launches:
//   1. partial: each workgroup reduces a chunk of pixels of one sample and a slice of
//      up to 256 channel vectors into fp32 sums of x and x^2 per group (16-byte
//      coalesced loads; a thread owns one 16-byte channel vector, so its accumulators
//      never mix channels; per-channel sums meet in LDS, then one thread per group adds
//      the group's channels in that slice, zero for groups outside it);
//   2. finalize: one workgroup per (sample, group) merges the (chunk, slice) partials
//      in fp64 in a fixed order (per thread, over the wave, over the four waves) and
//      writes per-(sample, channel) scale and shift
//      (gamma * rstd, beta - mean * gamma * rstd);
//   3. apply: y = x * scale + shift (then SiLU), one FMA per element, 16-byte
//      vectors, a (pixel block, sample) grid; up to 256 vectors per pixel a thread
//      keeps one channel vector's scale and shift and walks pixels, beyond that the
//      threads walk (pixel, vector) pairs.
// The input may be the channel concatenation of two tensors (the up path's
// [h, skip]); the output is always one contiguous tensor.
//
// LayerNorm: one wave per token row in registers, two-pass mean / variance,
// 16-byte loads and 8-byte (bf16) stores.
#include "kernels.h"

namespace dn {
namespace {

constexpr int kPixPerThread = 8;

struct GnGeom {
  int C, V, vslices, chunks, pix_per_chunk;
};

template <typename T> GnGeom gn_geom(int HW, int C) {
  constexpr int VEC = Elem<T>::kVec;
  GnGeom g;
  g.C = C;
  g.V = C / VEC;
  g.vslices = (g.V + 255) / 256;
  const int vz = g.V < 256 ? g.V : 256;
  const int pl = 256 / vz;
  g.pix_per_chunk = pl * kPixPerThread;
  g.chunks = (HW + g.pix_per_chunk - 1) / g.pix_per_chunk;
  return g;
}

template <typename T>
__global__ __launch_bounds__(256) void gn_partial_kernel(GroupNormParams p, GnGeom g) {
  constexpr int VEC = Elem<T>::kVec;
  __shared__ float red[256 * VEC * 2];
  const int tid = threadIdx.x;
  const int chunk = blockIdx.x, n = blockIdx.y, z = blockIdx.z;
  const int v_begin = z * 256;
  const int vz = min(g.V - v_begin, 256);
  const int pl_count = 256 / vz;
  const int pl = tid / vz;
  const int vl = tid - pl * vz;
  const bool active = pl < pl_count;

  float s[VEC], q[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) s[e] = q[e] = 0.f;
  if (active) {
    int c = (v_begin + vl) * VEC;
    const T* src;
    int ld;
    if (c < p.c0) {
      src = static_cast<const T*>(p.x0);
      ld = p.c0;
    } else {
      src = static_cast<const T*>(p.x1);
      ld = p.c1;
      c -= p.c0;
    }
    // all of the thread's pixels are loaded first (clamped to the image), then summed
    // in pixel order
    const int pbeg = chunk * g.pix_per_chunk;
    const int pend = min(pbeg + g.pix_per_chunk, p.HW);
    uint4 raw[kPixPerThread];
#pragma unroll
    for (int t = 0; t < kPixPerThread; ++t) {
      const int px = min(pbeg + pl + t * pl_count, p.HW - 1);
      raw[t] = ld16(src + ((long long)n * p.HW + px) * ld + c);
    }
#pragma unroll
    for (int t = 0; t < kPixPerThread; ++t) {
      // pixels past the chunk add an exact zero (a select, so that no branch sinks the
      // loads back to their uses)
      const bool in = pbeg + pl + t * pl_count < pend;
      const T* xv = reinterpret_cast<const T*>(&raw[t]);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float x = in ? to_f32(xv[e]) : 0.f;
        s[e] += x;
        q[e] += x * x;
      }
    }
  }
  if (active) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      red[((pl * vz + vl) * VEC + e) * 2 + 0] = s[e];
      red[((pl * vz + vl) * VEC + e) * 2 + 1] = q[e];
    }
  }
  __syncthreads();
  // per-channel sums over the pixel lanes (in place, lane 0's slots), then per group
  const int nch = vz * VEC;
  for (int j = tid; j < nch; j += 256) {
    float ss = 0.f, qq = 0.f;
    for (int l = 0; l < pl_count; ++l) {
      ss += red[(l * nch + j) * 2 + 0];
      qq += red[(l * nch + j) * 2 + 1];
    }
    red[j * 2 + 0] = ss;
    red[j * 2 + 1] = qq;
  }
  __syncthreads();
  const int cg = g.C / p.G;
  const int c_begin = v_begin * VEC;
  for (int grp = tid; grp < p.G; grp += 256) {
    const int lo = max(grp * cg, c_begin) - c_begin, hi = min((grp + 1) * cg, c_begin + nch) - c_begin;
    float ss = 0.f, qq = 0.f;
    for (int j = lo; j < hi; ++j) {
      ss += red[j * 2 + 0];
      qq += red[j * 2 + 1];
    }
    float* out = p.partial + ((((long long)n * g.chunks + chunk) * g.vslices + z) * p.G + grp) * 2;
    out[0] = ss;
    out[1] = qq;
  }
}

__global__ __launch_bounds__(256) void gn_finalize_kernel(GroupNormParams p, GnGeom g) {
  __shared__ double ws[4], wq[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = blockIdx.x, n = blockIdx.y;
  const int cg = g.C / p.G;
  const int items = g.chunks * g.vslices;
  double s = 0.0, q = 0.0;
  for (int i = tid; i < items; i += 256) {
    const float* in = p.partial + (((long long)n * items + i) * p.G + grp) * 2;
    s += in[0];
    q += in[1];
  }
  // a butterfly over the wave (lane 0's order of additions is fixed), then the four
  // waves in order
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    s += __shfl_xor(s, o, 64);
    q += __shfl_xor(q, o, 64);
  }
  if (lane == 0) {
    ws[wave] = s;
    wq[wave] = q;
  }
  __syncthreads();
  const double S = (ws[0] + ws[1]) + (ws[2] + ws[3]);
  const double Q = (wq[0] + wq[1]) + (wq[2] + wq[3]);
  const double cnt = (double)cg * p.HW;
  const double mean = S / cnt;
  const double var = fmax(Q / cnt - mean * mean, 0.0);
  const double rstd = 1.0 / sqrt(var + (double)p.eps);
  for (int j = tid; j < cg; j += 256) {
    const int c = grp * cg + j;
    const double sc = (double)p.gamma[c] * rstd;
    p.stats[(long long)n * g.C + c] = (float)sc;
    p.stats[(long long)(p.n + n) * g.C + c] = (float)((double)p.beta[c] - mean * sc);
  }
}

// Apply: grid (pixel blocks, samples); a block covers kApplyPix pixels of one sample,
// its threads walk the (pixel, 16-byte channel vector) pairs with an incremental
// quotient / remainder (no division in the loop).
constexpr int kApplyVecs = 2048;  // 16-byte vectors per apply workgroup (8 per thread)

template <typename T>
__global__ __launch_bounds__(256) void gn_apply_kernel(GroupNormParams p, GnGeom g, int pix_per_block) {
  constexpr int VEC = Elem<T>::kVec;
  const int V = g.V;
  const int n = blockIdx.y;
  const int pix0 = blockIdx.x * pix_per_block;
  const int npix = min(pix_per_block, p.HW - pix0);
  const int step_q = 256 / V, step_r = 256 - (256 / V) * V;
  int q = threadIdx.x / V, r = threadIdx.x - (threadIdx.x / V) * V;
  const float* scale = p.stats + (long long)n * g.C;
  const float* shift = p.stats + (long long)(p.n + n) * g.C;
  const long long rowbase = (long long)n * p.HW + pix0;
  // the block's (pixel, vector) pairs, 256 at a time, in batches of kBatch per thread
  // whose loads are all issued before the batch is computed and stored
  constexpr int kBatch = 4;
  const int nit = (npix * V + 255) / 256;  // pairs per thread, rounded up
  for (int b0 = 0; b0 < nit; b0 += kBatch) {
    uint4 raw[kBatch];
    float4 sc[kBatch][VEC / 4], sh[kBatch][VEC / 4];
    int qq[kBatch], cc[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      qq[u] = q;
      cc[u] = r * VEC;
      const long long pix = rowbase + min(q, npix - 1);
      const int c = r * VEC;
      raw[u] = c < p.c0 ? ld16(static_cast<const T*>(p.x0) + pix * p.c0 + c)
                        : ld16(static_cast<const T*>(p.x1) + pix * p.c1 + (c - p.c0));
#pragma unroll
      for (int e = 0; e < VEC / 4; ++e) {
        sc[u][e] = *reinterpret_cast<const float4*>(scale + c + 4 * e);
        sh[u][e] = *reinterpret_cast<const float4*>(shift + c + 4 * e);
      }
      q += step_q;
      r += step_r;
      if (r >= V) {
        r -= V;
        ++q;
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (qq[u] >= npix) continue;
      const T* xv = reinterpret_cast<const T*>(&raw[u]);
      uint4 outv;
      T* ov = reinterpret_cast<T*>(&outv);
#pragma unroll
      for (int e = 0; e < VEC; e += 4) {
        const float4 a = sc[u][e / 4], bsh = sh[u][e / 4];
        float v0 = to_f32(xv[e + 0]) * a.x + bsh.x, v1 = to_f32(xv[e + 1]) * a.y + bsh.y;
        float v2 = to_f32(xv[e + 2]) * a.z + bsh.z, v3 = to_f32(xv[e + 3]) * a.w + bsh.w;
        if (p.silu) {
          v0 = silu_f(v0);
          v1 = silu_f(v1);
          v2 = silu_f(v2);
          v3 = silu_f(v3);
        }
        ov[e + 0] = from_f32<T>(v0);
        ov[e + 1] = from_f32<T>(v1);
        ov[e + 2] = from_f32<T>(v2);
        ov[e + 3] = from_f32<T>(v3);
      }
      st16(static_cast<T*>(p.y) + (rowbase + qq[u]) * g.C + cc[u], outv);
    }
  }
}

// Apply with one channel vector per thread, for V <= 256 vectors per pixel: the 256
// threads are 256 / V pixel lanes of V channel vectors; a thread loads the scale and shift
// of its vector once, then its pixel lane's kApplyBatch pixels of the block, every load
// issued before the first is used. Same arithmetic per element as gn_apply_kernel.
constexpr int kApplyBatch = 8;

template <typename T>
__global__ __launch_bounds__(256) void gn_apply_cv_kernel(GroupNormParams p, GnGeom g, int pix_per_block) {
  constexpr int VEC = Elem<T>::kVec;
  const int V = g.V;
  const int lanes = 256 / V;
  const int pl = threadIdx.x / V, r = threadIdx.x - (threadIdx.x / V) * V;
  if (pl >= lanes) return;
  const int n = blockIdx.y;
  const int pix0 = blockIdx.x * pix_per_block;
  const int npix = min(pix_per_block, p.HW - pix0);
  const int c = r * VEC;
  const float* scale = p.stats + (long long)n * g.C;
  const float* shift = p.stats + (long long)(p.n + n) * g.C;
  float4 sc[VEC / 4], sh[VEC / 4];
#pragma unroll
  for (int e = 0; e < VEC / 4; ++e) {
    sc[e] = *reinterpret_cast<const float4*>(scale + c + 4 * e);
    sh[e] = *reinterpret_cast<const float4*>(shift + c + 4 * e);
  }
  const bool first = c < p.c0;
  const T* src = first ? static_cast<const T*>(p.x0) : static_cast<const T*>(p.x1);
  const int ld = first ? p.c0 : p.c1;
  const int cs = first ? c : c - p.c0;
  const long long rowbase = (long long)n * p.HW + pix0;
  for (int q0 = pl; q0 < npix; q0 += lanes * kApplyBatch) {
    uint4 raw[kApplyBatch];
#pragma unroll
    for (int u = 0; u < kApplyBatch; ++u) {
      const int q = min(q0 + u * lanes, npix - 1);
      raw[u] = ld16(src + (rowbase + q) * ld + cs);
    }
#pragma unroll
    for (int u = 0; u < kApplyBatch; ++u) {
      const int q = q0 + u * lanes;
      if (q >= npix) continue;
      const T* xv = reinterpret_cast<const T*>(&raw[u]);
      uint4 outv;
      T* ov = reinterpret_cast<T*>(&outv);
#pragma unroll
      for (int e = 0; e < VEC; e += 4) {
        const float4 a = sc[e / 4], bsh = sh[e / 4];
        float v0 = to_f32(xv[e + 0]) * a.x + bsh.x, v1 = to_f32(xv[e + 1]) * a.y + bsh.y;
        float v2 = to_f32(xv[e + 2]) * a.z + bsh.z, v3 = to_f32(xv[e + 3]) * a.w + bsh.w;
        if (p.silu) {
          v0 = silu_f(v0);
          v1 = silu_f(v1);
          v2 = silu_f(v2);
          v3 = silu_f(v3);
        }
        ov[e + 0] = from_f32<T>(v0);
        ov[e + 1] = from_f32<T>(v1);
        ov[e + 2] = from_f32<T>(v2);
        ov[e + 3] = from_f32<T>(v3);
      }
      st16(static_cast<T*>(p.y) + (rowbase + q) * g.C + c, outv);
    }
  }
}

constexpr int kLnMaxVec = 8;  // float4 vectors per lane: C <= 2048

template <typename T> struct Store4;
template <> struct Store4<uint8_t> {  // E4M3 codes
  __device__ static __forceinline__ void st(uint8_t* p, float a, float b, float c, float d) {
    *reinterpret_cast<unsigned*>(p) = fp8x4(a, b, c, d);
  }
};
template <> struct Store4<bf16> {
  __device__ static __forceinline__ void st(bf16* p, float a, float b, float c, float d) {
    bf16x4 o;
    o[0] = static_cast<bf16>(a);
    o[1] = static_cast<bf16>(b);
    o[2] = static_cast<bf16>(c);
    o[3] = static_cast<bf16>(d);
    *reinterpret_cast<bf16x4*>(p) = o;
  }
};
template <> struct Store4<float> {
  __device__ static __forceinline__ void st(float* p, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
  }
};

// One wave per row. With NS > 0 the row is first rebuilt from the residual stream:
// x[row] = (resid ? x[row] : 0) + bias + sum_s part[s][row] in that order (the reduction of
// a split-K GEMM that wrote fp32 partial slabs), and written back; then
// y = (x - mean) * rstd * gamma + beta with two-pass mean / variance. Every load of the
// row (x, the slabs, the bias; gamma and beta too when NS = 0) is issued before the first
// use, so a row waits on one memory latency; the two wave sums use DPP lane moves;
// vector columns past C are skipped wave-uniformly, lanes past C read a valid column and
// are masked.
template <typename T, int NS>
__global__ __launch_bounds__(256) void ln_kernel(float* x, T* y, long long M, int C, const float* gamma,
                                                 const float* beta, float eps, const float* part, long long slab,
                                                 const float* bias, int resid) {
  const int lane = threadIdx.x & 63;
  const long long row = blockIdx.x * 4ll + (threadIdx.x >> 6);
  if (row >= M) return;
  const int nv = C / 4;
  float4* xr = reinterpret_cast<float4*>(x + row * C);
  const float4 zero4 = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 v[kLnMaxVec];
  float4 sl[NS > 0 ? NS : 1][kLnMaxVec];
  float4 bv[kLnMaxVec];
  // the plain LayerNorm also loads gamma and beta with the row (the slab-summing
  // variant keeps its registers for the slabs and loads them after the statistics)
  float4 gv[NS == 0 ? kLnMaxVec : 1], btv[NS == 0 ? kLnMaxVec : 1];
  const float4* g4 = reinterpret_cast<const float4*>(gamma);
  const float4* b4 = reinterpret_cast<const float4*>(beta);
#pragma unroll
  for (int j = 0; j < kLnMaxVec; ++j) {
    v[j] = bv[j] = zero4;
    if constexpr (NS == 0) gv[j] = btv[j] = zero4;
#pragma unroll
    for (int k = 0; k < (NS > 0 ? NS : 1); ++k) sl[k][j] = zero4;
    if (64 * j < nv) {
      const int i = min(lane + 64 * j, nv - 1);
      if (NS == 0 || resid) v[j] = xr[i];
      if constexpr (NS == 0) {
        gv[j] = g4[i];
        btv[j] = b4[i];
      }
      if constexpr (NS > 0) {
        if (bias) bv[j] = reinterpret_cast<const float4*>(bias)[i];
        const float4* pr = reinterpret_cast<const float4*>(part + row * C);
#pragma unroll
        for (int k = 0; k < NS; ++k) sl[k][j] = pr[k * (slab / 4) + i];
      }
    }
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kLnMaxVec; ++j) {
    const int i = lane + 64 * j;
    if (64 * j < nv) {
      if constexpr (NS > 0) {
        float4 a = v[j];
        if (bias) {
          a.x += bv[j].x;
          a.y += bv[j].y;
          a.z += bv[j].z;
          a.w += bv[j].w;
        }
#pragma unroll
        for (int k = 0; k < NS; ++k) {
          a.x += sl[k][j].x;
          a.y += sl[k][j].y;
          a.z += sl[k][j].z;
          a.w += sl[k][j].w;
        }
        v[j] = a;
        if (i < nv) xr[i] = a;
      }
      if (i < nv) s += (v[j].x + v[j].y) + (v[j].z + v[j].w);
    }
  }
  const float mean = wave_sum_dpp(s) / C;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < kLnMaxVec; ++j) {
    const int i = lane + 64 * j;
    if (64 * j < nv && i < nv) {
      const float a = v[j].x - mean, b = v[j].y - mean, c = v[j].z - mean, d = v[j].w - mean;
      q += (a * a + b * b) + (c * c + d * d);
    }
  }
  const float rstd = rsqrtf(wave_sum_dpp(q) / C + eps);
  T* yr = y + row * C;
#pragma unroll
  for (int j = 0; j < kLnMaxVec; ++j) {
    const int i = lane + 64 * j;
    if (64 * j < nv && i < nv) {
      float4 g, bb;
      if constexpr (NS == 0) {
        g = gv[j];
        bb = btv[j];
      } else {
        g = g4[i];
        bb = b4[i];
      }
      Store4<T>::st(yr + 4 * i, (v[j].x - mean) * rstd * g.x + bb.x, (v[j].y - mean) * rstd * g.y + bb.y,
                    (v[j].z - mean) * rstd * g.z + bb.z, (v[j].w - mean) * rstd * g.w + bb.w);
    }
  }
}

template <typename T, int NS>
void launch_ln(float* x, T* y, long long M, int C, const float* gamma, const float* beta, float eps, const float* part,
               const float* bias, bool resid, hipStream_t s) {
  hipLaunchKernelGGL((ln_kernel<T, NS>), dim3(static_cast<unsigned>((M + 3) / 4)), dim3(256), 0, s, x, y, M, C, gamma,
                     beta, eps, part, M * C, bias, resid ? 1 : 0);
}

}  // namespace

size_t groupnorm_workspace_floats(int n, int HW, int C, int G) {
  // [n][chunk][slice][G] (sum, sum of squares); the larger of the fp32 and bf16 geometries
  const GnGeom g = gn_geom<float>(HW, C);
  const GnGeom g2 = gn_geom<bf16>(HW, C);
  const size_t a = size_t(g.chunks) * g.vslices, b = size_t(g2.chunks) * g2.vslices;
  return size_t(n) * (a > b ? a : b) * G * 2;
}

template <typename T> void groupnorm(const GroupNormParams& p, hipStream_t s) {
  constexpr int VEC = Elem<T>::kVec;
  const int C = p.c0 + p.c1;
  DN_CHECK(p.n >= 1 && p.HW >= 1 && C >= 1 && p.G >= 1, "groupnorm: empty problem");
  DN_CHECK(C % p.G == 0, "groupnorm: channels must divide into groups");
  DN_CHECK(p.c0 % VEC == 0 && p.c1 % VEC == 0, "groupnorm: channel counts must be multiples of 16 bytes");
  DN_CHECK(p.x0 && p.y && p.partial && p.stats && p.gamma && p.beta && (p.c1 == 0 || p.x1), "groupnorm: null");
  const GnGeom g = gn_geom<T>(p.HW, C);
  hipLaunchKernelGGL(gn_partial_kernel<T>, dim3(g.chunks, p.n, g.vslices), dim3(256), 0, s, p, g);
  hipLaunchKernelGGL(gn_finalize_kernel, dim3(p.G, p.n), dim3(256), 0, s, p, g);
  if (g.V <= 256) {
    const int ppb = (256 / g.V) * kApplyBatch;
    hipLaunchKernelGGL(gn_apply_cv_kernel<T>, dim3((p.HW + ppb - 1) / ppb, p.n), dim3(256), 0, s, p, g, ppb);
  } else {
    const int ppb = (kApplyVecs + g.V - 1) / g.V;
    hipLaunchKernelGGL(gn_apply_kernel<T>, dim3((p.HW + ppb - 1) / ppb, p.n), dim3(256), 0, s, p, g, ppb);
  }
  DN_HIP(hipGetLastError());
}

template <typename T>
void layernorm(const float* x, T* y, long long M, int C, const float* gamma, const float* beta, float eps,
               hipStream_t s) {
  layernorm_reduce<T>(const_cast<float*>(x), y, M, C, gamma, beta, eps, nullptr, 0, nullptr, true, s);
}

template <typename T>
void layernorm_reduce(float* x, T* y, long long M, int C, const float* gamma, const float* beta, float eps,
                      const float* part, int nsplit, const float* bias, bool resid, hipStream_t s) {
  DN_CHECK(M >= 1 && C >= 4 && C % 4 == 0 && C <= 4 * 64 * kLnMaxVec, "layernorm: C must be a multiple of 4, <= 2048");
  DN_CHECK(x && y && gamma && beta, "layernorm: null");
  DN_CHECK(((uintptr_t)x | (uintptr_t)gamma | (uintptr_t)beta | (uintptr_t)part | (uintptr_t)bias) % 16 == 0 &&
               (uintptr_t)y % (4 * sizeof(T)) == 0,
           "layernorm: x, gamma, beta, partials and bias must be 16-byte aligned, y aligned to 4 elements");
  DN_CHECK(nsplit == 0 || part, "layernorm: partial slabs missing");
  switch (nsplit) {
    case 0: launch_ln<T, 0>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 1: launch_ln<T, 1>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 2: launch_ln<T, 2>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 3: launch_ln<T, 3>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 4: launch_ln<T, 4>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 5: launch_ln<T, 5>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 6: launch_ln<T, 6>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 7: launch_ln<T, 7>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    case 8: launch_ln<T, 8>(x, y, M, C, gamma, beta, eps, part, bias, resid, s); break;
    default: throw Error(-1, "layernorm: at most 8 partial slabs");
  }
  DN_HIP(hipGetLastError());
}

template void groupnorm<float>(const GroupNormParams&, hipStream_t);
template void groupnorm<bf16>(const GroupNormParams&, hipStream_t);
template void layernorm<float>(const float*, float*, long long, int, const float*, const float*, float, hipStream_t);
template void layernorm<bf16>(const float*, bf16*, long long, int, const float*, const float*, float, hipStream_t);
template void layernorm_reduce<float>(float*, float*, long long, int, const float*, const float*, float, const float*,
                                      int, const float*, bool, hipStream_t);
template void layernorm_reduce<bf16>(float*, bf16*, long long, int, const float*, const float*, float, const float*,
                                     int, const float*, bool, hipStream_t);
template void layernorm_reduce<uint8_t>(float*, uint8_t*, long long, int, const float*, const float*, float,
                                        const float*, int, const float*, bool, hipStream_t);
template void layernorm<uint8_t>(const float*, uint8_t*, long long, int, const float*, const float*, float,
                                 hipStream_t);

}  // namespace dn
