// Top-1 cosine search over the prompt-embedding cache (HBM-bound; gfx950).
//
// Pass 1: every half-wave (32 lanes) scores one cache row at a time — 16-byte
// coalesced fp16 loads, fp32 products and sums of q.c and c.c, a 5-step
// butterfly — and keeps its best (score, index); each workgroup writes the
// best of its 8 half-waves. Pass 2: one workgroup reduces the per-workgroup
// winners. Ties go to the lowest index at every stage, so the result is the
// first maximum, independent of the launch shape.
#include "kernels.h"

namespace dn {
namespace {

constexpr int kScanBlocks = 2048;
constexpr int kQMaxVec = 4;  // fast path: dim <= 32 lanes * 4 vectors * 8 = 1024

struct Cand {
  float s;
  long long i;
};

__device__ __forceinline__ bool better(float s, long long i, float bs, long long bi) {
  return s > bs || (s == bs && i < bi);
}

__device__ __forceinline__ float h2f(uint16_t h) { return static_cast<float>(__builtin_bit_cast(_Float16, h)); }

__device__ __forceinline__ float half_sum(float v) {
#pragma unroll
  for (int o = 16; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Score of one row (cosine up to the positive factor 1/|q|); -inf for a zero row.
__device__ __forceinline__ float row_score(float dot, float cc) { return cc > 0.f ? dot * rsqrtf(cc) : -INFINITY; }

template <int NQ>
__global__ __launch_bounds__(256) void scan_vec_kernel(const uint16_t* q, const uint16_t* cache, long long n, int dim,
                                                       Cand* part) {
  const int lane = threadIdx.x & 63;
  const int li = lane & 31;
  const int hw = threadIdx.x >> 5;  // half-wave in block, 0..7
  const int V = dim / 8;
  float qv[NQ][8];
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const int v = li + 32 * j;
    uint4 raw = v < V ? ld16(q + v * 8) : make_uint4(0u, 0u, 0u, 0u);
    const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
    for (int e = 0; e < 8; ++e) qv[j][e] = h2f(h[e]);
  }
  float best_s = -INFINITY;
  long long best_i = n;
  const long long stride = (long long)gridDim.x * 8;
  for (long long row = (long long)blockIdx.x * 8 + hw; row < n; row += stride) {
    const uint16_t* c = cache + row * dim;
    float dot = 0.f, cc = 0.f;
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      const int v = li + 32 * j;
      if (v < V) {
        const uint4 raw = ld16(c + v * 8);
        const uint16_t* h = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = h2f(h[e]);
          dot += qv[j][e] * x;
          cc += x * x;
        }
      }
    }
    dot = half_sum(dot);
    cc = half_sum(cc);
    const float s = row_score(dot, cc);
    if (better(s, row, best_s, best_i)) {
      best_s = s;
      best_i = row;
    }
  }
  __shared__ Cand red[8];
  if (li == 0) red[hw] = Cand{best_s, best_i};
  __syncthreads();
  if (threadIdx.x == 0) {
    Cand b = red[0];
    for (int k = 1; k < 8; ++k)
      if (better(red[k].s, red[k].i, b.s, b.i)) b = red[k];
    part[blockIdx.x] = b;
  }
}

// Any dim / alignment: element-wise loads, q staged in LDS.
__global__ __launch_bounds__(256) void scan_scalar_kernel(const uint16_t* q, const uint16_t* cache, long long n,
                                                          int dim, Cand* part) {
  extern __shared__ float qs[];
  for (int e = threadIdx.x; e < dim; e += 256) qs[e] = h2f(q[e]);
  __syncthreads();
  const int li = threadIdx.x & 31;
  const int hw = threadIdx.x >> 5;
  float best_s = -INFINITY;
  long long best_i = n;
  const long long stride = (long long)gridDim.x * 8;
  for (long long row = (long long)blockIdx.x * 8 + hw; row < n; row += stride) {
    const uint16_t* c = cache + row * dim;
    float dot = 0.f, cc = 0.f;
    for (int e = li; e < dim; e += 32) {
      const float x = h2f(c[e]);
      dot += qs[e] * x;
      cc += x * x;
    }
    dot = half_sum(dot);
    cc = half_sum(cc);
    const float s = row_score(dot, cc);
    if (better(s, row, best_s, best_i)) {
      best_s = s;
      best_i = row;
    }
  }
  __shared__ Cand red[8];
  if (li == 0) red[hw] = Cand{best_s, best_i};
  __syncthreads();
  if (threadIdx.x == 0) {
    Cand b = red[0];
    for (int k = 1; k < 8; ++k)
      if (better(red[k].s, red[k].i, b.s, b.i)) b = red[k];
    part[blockIdx.x] = b;
  }
}

__global__ __launch_bounds__(256) void reduce_kernel(const Cand* part, int nb, const uint16_t* q, int dim,
                                                     long long* idx, float* score) {
  __shared__ float ss[256];
  __shared__ long long si[256];
  __shared__ float qn[256];
  const int t = threadIdx.x;
  float bs = -INFINITY;
  long long bi = 0x7fffffffffffffffll;
  for (int k = t; k < nb; k += 256)
    if (better(part[k].s, part[k].i, bs, bi)) {
      bs = part[k].s;
      bi = part[k].i;
    }
  float qq = 0.f;
  for (int e = t; e < dim; e += 256) {
    const float x = h2f(q[e]);
    qq += x * x;
  }
  ss[t] = bs;
  si[t] = bi;
  qn[t] = qq;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) {
      if (better(ss[t + w], si[t + w], ss[t], si[t])) {
        ss[t] = ss[t + w];
        si[t] = si[t + w];
      }
      qn[t] += qn[t + w];
    }
    __syncthreads();
  }
  if (t == 0) {
    // A zero query (or a cache of zero rows) has no defined cosine: report no row.
    *idx = (qn[0] > 0.f && ss[0] > -INFINITY) ? si[0] : -1;
    *score = ss[0] * rsqrtf(qn[0]);
  }
}

}  // namespace

size_t lookup_workspace_bytes() { return sizeof(Cand) * kScanBlocks; }

void lookup(const uint16_t* q, const uint16_t* cache, long long n, int dim, void* ws, long long* idx_dev,
            float* score_dev, hipStream_t s) {
  DN_CHECK(n >= 1 && dim >= 1, "lookup: empty cache");
  Cand* part = static_cast<Cand*>(ws);
  const long long want = (n + 7) / 8;
  const int nb = static_cast<int>(want < kScanBlocks ? want : kScanBlocks);
  const bool aligned = (reinterpret_cast<uintptr_t>(cache) % 16 == 0) && (reinterpret_cast<uintptr_t>(q) % 16 == 0);
  const int V = dim / 8;
  if (aligned && dim % 8 == 0 && V <= 32 * kQMaxVec) {
    const int nq = (V + 31) / 32;
    if (nq == 1)
      hipLaunchKernelGGL(scan_vec_kernel<1>, dim3(nb), dim3(256), 0, s, q, cache, n, dim, part);
    else if (nq == 2)
      hipLaunchKernelGGL(scan_vec_kernel<2>, dim3(nb), dim3(256), 0, s, q, cache, n, dim, part);
    else if (nq == 3)
      hipLaunchKernelGGL(scan_vec_kernel<3>, dim3(nb), dim3(256), 0, s, q, cache, n, dim, part);
    else
      hipLaunchKernelGGL(scan_vec_kernel<4>, dim3(nb), dim3(256), 0, s, q, cache, n, dim, part);
  } else {
    DN_CHECK(dim <= 16384, "lookup: dim too large for the scalar path");
    hipLaunchKernelGGL(scan_scalar_kernel, dim3(nb), dim3(256), dim * sizeof(float), s, q, cache, n, dim, part);
  }
  hipLaunchKernelGGL(reduce_kernel, dim3(1), dim3(256), 0, s, part, nb, q, dim, idx_dev, score_dev);
  DN_HIP(hipGetLastError());
}

}  // namespace dn
