// Top-1 cosine search over the prompt-embedding cache (HBM-bound; gfx950).
//
// Pass 1: every half-wave (32 lanes) scores two cache rows per iteration — all
// 16-byte coalesced fp16 loads of both rows issued before any arithmetic, packed
// fp16 dot products accumulating in fp32 (v_dot2_f32_f16: the fp16 x fp16 products
// are exact in fp32) for q.c and c.c, then 5-step butterflies — and keeps its best
// (score, index); each workgroup writes the best of its 8 half-waves. Pass 2: one
// workgroup reduces the per-workgroup winners. Ties go to the lowest index at every
// stage, so the result is the first maximum, independent of the launch shape.
//
// Batched search (up to 64 queries per pass): the scores of a 16-row tile against all
// queries are one [16 x dim] x [dim x 64] contraction on the matrix cores
// (v_mfma_f32_16x16x32_f16: fp16 operands, exact products, fp32 sums), so the table is
// read from HBM once per 64 queries instead of once per query. Each lane loads its
// A operand (row l % 16, 8 consecutive dims at 8 * (l / 16)) straight from the table:
// one 16-byte load per 32-dim k-step, 64 contiguous bytes per row per instruction.
// The queries sit in LDS in B-fragment order (one conflict-free 16-byte read per lane
// and k-step). Row norms come from the same A registers (packed fp16 dot products),
// and the top-1 per query is kept in registers while the wave walks its tiles.
#include "kernels.h"

namespace dn {
namespace {

constexpr int kScanBlocks = 2048;  // a multiple of 256 (the reduction's per-thread share)
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

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ h2 as_h2(unsigned u) { return __builtin_bit_cast(h2, u); }

// q . x and x . x over one 16-byte vector (8 fp16 values), accumulated in fp32.
__device__ __forceinline__ void dot8(const h2 (&qv)[4], const uint4 x, float& dot, float& cc) {
  const unsigned w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const h2 v = as_h2(w[k]);
    dot = __builtin_amdgcn_fdot2(qv[k], v, dot, false);
    cc = __builtin_amdgcn_fdot2(v, v, cc, false);
  }
}

template <int NQ>
__global__ __launch_bounds__(256) void scan_vec_kernel(const uint16_t* q, const uint16_t* cache, long long n, int dim,
                                                       Cand* part) {
  const int lane = threadIdx.x & 63;
  const int li = lane & 31;
  const int hw = threadIdx.x >> 5;  // half-wave in block, 0..7
  const int V = dim / 8;
  h2 qv[NQ][4];
  bool act[NQ];
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const int v = li + 32 * j;
    act[j] = v < V;
    const uint4 raw = act[j] ? ld16(q + v * 8) : make_uint4(0u, 0u, 0u, 0u);
    qv[j][0] = as_h2(raw.x);
    qv[j][1] = as_h2(raw.y);
    qv[j][2] = as_h2(raw.z);
    qv[j][3] = as_h2(raw.w);
  }
  float best_s = -INFINITY;
  long long best_i = n;
  const long long stride = (long long)gridDim.x * 16;
  // rows r and r + 1 per half-wave; past the end the second row re-reads row r and is not scored
  for (long long r = (long long)blockIdx.x * 16 + 2 * hw; r < n; r += stride) {
    const bool two = r + 1 < n;
    const uint16_t* c0 = cache + r * dim;
    const uint16_t* c1 = two ? c0 + dim : c0;
    uint4 x0[NQ], x1[NQ];
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      const int v = act[j] ? li + 32 * j : 0;
      x0[j] = ld16(c0 + v * 8);
      x1[j] = ld16(c1 + v * 8);
    }
    float d0 = 0.f, s0 = 0.f, d1 = 0.f, s1 = 0.f;
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      if (!act[j]) continue;
      dot8(qv[j], x0[j], d0, s0);
      dot8(qv[j], x1[j], d1, s1);
    }
#pragma unroll
    for (int o = 16; o > 0; o >>= 1) {
      d0 += __shfl_xor(d0, o, 64);
      s0 += __shfl_xor(s0, o, 64);
      d1 += __shfl_xor(d1, o, 64);
      s1 += __shfl_xor(s1, o, 64);
    }
    const float sc0 = row_score(d0, s0);
    if (better(sc0, r, best_s, best_i)) {
      best_s = sc0;
      best_i = r;
    }
    const float sc1 = row_score(d1, s1);
    if (two && better(sc1, r + 1, best_s, best_i)) {
      best_s = sc1;
      best_i = r + 1;
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

// Level of the table for a result (index -1: nothing retrieved, level 0).
__device__ __forceinline__ int select_level(const KTable& kt, long long idx, float score) {
  if (idx < 0) return 0;
  int j = 0;
  for (int i = 0; i < kt.n; ++i)
    if (score >= kt.thr[i]) j = i + 1;
  return kt.level[j];
}

// Pass 2, one workgroup: every thread loads its (up to kScanBlocks / 256) winners
// before comparing them; waves reduce with shuffles, then the 4 wave winners in order.
// The squared norm of q (for the reported cosine) is summed alongside. The result may
// be written to pinned host memory.
__global__ __launch_bounds__(256) void reduce_kernel(const Cand* part, int nb, const uint16_t* q, int dim,
                                                     long long* idx, float* score, KTable kt, int* kout) {
  constexpr int kPer = kScanBlocks / 256;
  __shared__ float ws_s[4], ws_q[4];
  __shared__ long long ws_i[4];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  Cand c[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int j = t + 256 * k;
    c[k] = j < nb ? part[j] : Cand{-INFINITY, 0x7fffffffffffffffll};
  }
  float qq = 0.f;
  for (int e = t; e < dim; e += 256) {
    const float x = h2f(q[e]);
    qq += x * x;
  }
  float bs = c[0].s;
  long long bi = c[0].i;
#pragma unroll
  for (int k = 1; k < kPer; ++k)
    if (better(c[k].s, c[k].i, bs, bi)) {
      bs = c[k].s;
      bi = c[k].i;
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float s2 = __shfl_xor(bs, o, 64);
    const long long i2 = __shfl_xor(bi, o, 64);
    if (better(s2, i2, bs, bi)) {
      bs = s2;
      bi = i2;
    }
    qq += __shfl_xor(qq, o, 64);
  }
  if (lane == 0) {
    ws_s[w] = bs;
    ws_i[w] = bi;
    ws_q[w] = qq;
  }
  __syncthreads();
  if (t == 0) {
    float qn = ws_q[0];
    for (int k = 1; k < 4; ++k) {
      if (better(ws_s[k], ws_i[k], bs, bi)) {
        bs = ws_s[k];
        bi = ws_i[k];
      }
      qn += ws_q[k];
    }
    // A zero query (or a cache of zero rows) has no defined cosine: report no row.
    const long long r = (qn > 0.f && bs > -INFINITY) ? bi : -1;
    const float sc = bs * rsqrtf(qn);
    *idx = r;
    *score = sc;
    if (kout) *kout = select_level(kt, r, sc);
  }
}


// ---------------------------------------------------------------- batched search

constexpr int kBatchQ = 64;          // queries per pass: 4 column tiles of 16
constexpr int kBatchBlocks = 256;    // at most one workgroup per CU (the queries take up to 128 KB of LDS)

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// Two register sets of a tile's rows (4 KS VGPRs each) when they fit beside three
// (KS = 8) or two waves per SIMD: the next tile's loads are then in flight while the
// current tile is scored. dim 1024 keeps one set (two waves per SIMD).
template <int KS> struct BatchCfg {
  static constexpr bool kTwoSets = KS <= 24;
  static constexpr int kWaves = KS <= 8 ? 12 : 8;
};

// dim = 32 * KS. q [nq][dim] (nq <= 64), cache [n][dim]; part [gridDim.x][64] receives
// each workgroup's best (score, index) per query (queries >= nq score zero and are ignored).
template <int KS>
__global__ __launch_bounds__(BatchCfg<KS>::kWaves * 64) void scan_mfma_kernel(const uint16_t* q, int nq,
                                                                            const uint16_t* cache, int n,
                                                                            Cand* part) {
  constexpr int NW = BatchCfg<KS>::kWaves;
  constexpr int dim = 32 * KS;
  extern __shared__ __align__(16) uint4 qf[];  // [4 column tiles][KS k-steps][64 lanes]
  __shared__ Cand red[NW][kBatchQ];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int r16 = lane & 15, grp = lane >> 4;
  for (int u = t; u < 4 * KS * 64; u += NW * 64) {
    const int ln = u & 63, ks = (u >> 6) % KS, qt = (u >> 6) / KS;
    const int qi = qt * 16 + (ln & 15);
    qf[u] = qi < nq ? ld16(q + (long long)qi * dim + ks * 32 + 8 * (ln >> 4)) : make_uint4(0u, 0u, 0u, 0u);
  }
  __syncthreads();
  float best_s[4];
  int best_i[4];
#pragma unroll
  for (int qt = 0; qt < 4; ++qt) {
    best_s[qt] = -INFINITY;
    best_i[qt] = n;
  }
  const int tiles = (n + 15) / 16;
  const int stride = gridDim.x * NW;

  // the lane's 16-byte slices of row tile * 16 + r16 (past the end: the last row, not scored);
  // tile < tiles + 2 * stride keeps tile * 16 + 15 below 2^31 for n < 2^31 - 64
  auto load = [&](uint4 (&a)[KS], int tile) {
    const int row = tile * 16 + r16;
    const uint16_t* src = cache + (long long)(row < n ? row : n - 1) * dim + 8 * grp;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) a[ks] = ld16(src + 32 * ks);
  };
  auto score = [&](const uint4 (&a)[KS], int tile) {
    f32x4 acc[4];
#pragma unroll
    for (int qt = 0; qt < 4; ++qt) acc[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float cc = 0.f;
    // opaque to the optimiser, so the query fragments are re-read from LDS per tile
    // instead of being hoisted out of the loop into 16 KS registers
    int ql = lane;
    asm volatile("" : "+v"(ql));
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const f16x8 av = __builtin_bit_cast(f16x8, a[ks]);
#pragma unroll
      for (int qt = 0; qt < 4; ++qt)
        acc[qt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, __builtin_bit_cast(f16x8, qf[(qt * KS + ks) * 64 + ql]),
                                                         acc[qt], 0, 0, 0);
      const unsigned wd[4] = {a[ks].x, a[ks].y, a[ks].z, a[ks].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) cc = __builtin_amdgcn_fdot2(as_h2(wd[k]), as_h2(wd[k]), cc, false);
    }
    // |c|^2 of row r16: the four lane groups hold its four 8-dim slices of every k-step
    cc += __shfl_xor(cc, 16, 64);
    cc += __shfl_xor(cc, 32, 64);
    // acc[qt][i] = c_(tile*16 + 4 grp + i) . q_(16 qt + r16)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = 4 * grp + i;
      const float c2 = __shfl(cc, rr, 64);
      const int ri = tile * 16 + rr;
      if (ri >= n) continue;
#pragma unroll
      for (int qt = 0; qt < 4; ++qt) {
        const float sc = row_score(acc[qt][i], c2);
        if (better(sc, ri, best_s[qt], best_i[qt])) {
          best_s[qt] = sc;
          best_i[qt] = ri;
        }
      }
    }
  };

  const int first = blockIdx.x * NW + w;
  if constexpr (BatchCfg<KS>::kTwoSets) {
    // The look-ahead loads are unconditional (a tile past the end reads the last row,
    // in bounds, and is never scored): inside a branch they would make the compiler's
    // wait counts assume the worst case, so scoring a tile would wait for the next one.
    uint4 a0[KS], a1[KS];
    load(a0, first);
    for (int tile = first; tile < tiles; tile += 2 * stride) {
      const int t1 = tile + stride;
      load(a1, t1);
      score(a0, tile);
      if (t1 >= tiles) break;
      load(a0, t1 + stride);
      score(a1, t1);
    }
  } else {
    uint4 a0[KS];
    for (int tile = first; tile < tiles; tile += stride) {
      load(a0, tile);
      score(a0, tile);
    }
  }
  // the four lane groups of a query column, then the waves in order
#pragma unroll
  for (int qt = 0; qt < 4; ++qt) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float s2 = __shfl_xor(best_s[qt], o, 64);
      const int i2 = __shfl_xor(best_i[qt], o, 64);
      if (better(s2, i2, best_s[qt], best_i[qt])) {
        best_s[qt] = s2;
        best_i[qt] = i2;
      }
    }
    if (grp == 0) red[w][qt * 16 + r16] = Cand{best_s[qt], best_i[qt]};
  }
  __syncthreads();
  if (t < kBatchQ) {
    Cand b = red[0][t];
    for (int k = 1; k < NW; ++k)
      if (better(red[k][t].s, red[k][t].i, b.s, b.i)) b = red[k][t];
    part[(long long)blockIdx.x * kBatchQ + t] = b;
  }
}

// One workgroup per query: the nb workgroup winners of its column, and |q|^2 for the
// reported cosine. Writes idx[j] = -1 where the query has no defined cosine.
__global__ __launch_bounds__(256) void reduce_batch_kernel(const Cand* part, int nb, const uint16_t* q, int dim,
                                                           long long* idx, float* score, KTable kt, int* kout) {
  __shared__ float ws_s[4], ws_q[4];
  __shared__ long long ws_i[4];
  const int j = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  Cand c = t < nb ? part[(long long)t * kBatchQ + j] : Cand{-INFINITY, 0x7fffffffffffffffll};
  float qq = 0.f;
  for (int e = t; e < dim; e += 256) {
    const float x = h2f(q[(long long)j * dim + e]);
    qq += x * x;
  }
  float bs = c.s;
  long long bi = c.i;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float s2 = __shfl_xor(bs, o, 64);
    const long long i2 = __shfl_xor(bi, o, 64);
    if (better(s2, i2, bs, bi)) {
      bs = s2;
      bi = i2;
    }
    qq += __shfl_xor(qq, o, 64);
  }
  if (lane == 0) {
    ws_s[w] = bs;
    ws_i[w] = bi;
    ws_q[w] = qq;
  }
  __syncthreads();
  if (t == 0) {
    float qn = ws_q[0];
    for (int k = 1; k < 4; ++k) {
      if (better(ws_s[k], ws_i[k], bs, bi)) {
        bs = ws_s[k];
        bi = ws_i[k];
      }
      qn += ws_q[k];
    }
    const long long r = (qn > 0.f && bs > -INFINITY) ? bi : -1;
    const float sc = bs * rsqrtf(qn);
    idx[j] = r;
    score[j] = sc;
    if (kout) kout[j] = select_level(kt, r, sc);
  }
}

// Launches the scan over min(256, tiles / waves) workgroups; returns that count.
template <int KS>
int launch_batch(const uint16_t* q, int nq, const uint16_t* cache, int n, Cand* part, hipStream_t s) {
  constexpr int NW = BatchCfg<KS>::kWaves;
  const long long want = ((n + 15) / 16 + NW - 1) / NW;
  const int nb = static_cast<int>(want < kBatchBlocks ? want : kBatchBlocks);
  const size_t lds = sizeof(uint4) * 4 * KS * 64;
  static bool attr = false;  // per process: the attribute belongs to the code object
  if (!attr) {
    DN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&scan_mfma_kernel<KS>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
    attr = true;
  }
  hipLaunchKernelGGL(scan_mfma_kernel<KS>, dim3(nb), dim3(NW * 64), lds, s, q, nq, cache, n, part);
  return nb;
}

}  // namespace

size_t lookup_workspace_bytes() { return sizeof(Cand) * kScanBlocks; }

void lookup(const uint16_t* q, const uint16_t* cache, long long n, int dim, void* ws, long long* idx_out,
            float* score_out, hipStream_t s, const KTable* kt, int* k_out) {
  DN_CHECK(n >= 1 && dim >= 1, "lookup: empty cache");
  Cand* part = static_cast<Cand*>(ws);
  const long long want = (n + 15) / 16;
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
  const KTable tab = kt ? *kt : KTable();
  hipLaunchKernelGGL(reduce_kernel, dim3(1), dim3(256), 0, s, part, nb, q, dim, idx_out, score_out, tab,
                     kt ? k_out : nullptr);
  DN_HIP(hipGetLastError());
}

}  // namespace dn

namespace dn {

size_t lookup_batch_workspace_bytes() { return sizeof(Cand) * kBatchBlocks * kBatchQ; }

int lookup_batch_max_queries() { return kBatchQ; }

bool lookup_batch_supported(const uint16_t* q, const uint16_t* cache, long long n, int dim) {
  if (n > (1ll << 31) - 64) return false;  // 32-bit row indices in the scan
  const bool aligned = (reinterpret_cast<uintptr_t>(cache) % 16 == 0) && (reinterpret_cast<uintptr_t>(q) % 16 == 0);
  return aligned && (dim == 256 || dim == 512 || dim == 768 || dim == 1024);
}

void lookup_batch(const uint16_t* q, int nq, const uint16_t* cache, long long n, int dim, void* ws,
                  long long* idx_out, float* score_out, hipStream_t s, const KTable* kt, int* k_out) {
  DN_CHECK(n >= 1 && dim >= 1, "lookup_batch: empty cache");
  DN_CHECK(nq >= 1 && nq <= kBatchQ, "lookup_batch: 1 to 64 queries per pass");
  DN_CHECK(lookup_batch_supported(q, cache, n, dim),
           "lookup_batch: dim must be 256, 512, 768 or 1024, 16-byte aligned, n < 2^31 - 64");
  const int n32 = static_cast<int>(n);
  Cand* part = static_cast<Cand*>(ws);
  int nb = 0;
  switch (dim) {
    case 256: nb = launch_batch<8>(q, nq, cache, n32, part, s); break;
    case 512: nb = launch_batch<16>(q, nq, cache, n32, part, s); break;
    case 768: nb = launch_batch<24>(q, nq, cache, n32, part, s); break;
    default: nb = launch_batch<32>(q, nq, cache, n32, part, s); break;
  }
  const KTable tab = kt ? *kt : KTable();
  hipLaunchKernelGGL(reduce_batch_kernel, dim3(nq), dim3(256), 0, s, part, nb, q, dim, idx_out, score_out, tab,
                     kt ? k_out : nullptr);
  DN_HIP(hipGetLastError());
}

}  // namespace dn
