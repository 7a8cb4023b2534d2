// Kernel parameter blocks and host launchers (internal to the library).
#pragma once

#include "common.h"

namespace dn {

// ---------------------------------------------------------------- GEMM / implicit-GEMM conv
//
// C[m][n] = sum_k A[m][k] * B[n][k], then the epilogue. B is a packed weight
// matrix [N][ldb] (K contiguous). A is gathered on the fly:
//  - linear (taps == 1): row m of the source(s), channels [0, c0) from a0 and
//    [c0, c0 + c1) from a1 (channel concatenation);
//  - conv3x3 (taps == 9): NHWC source(s); output pixel m = (s, oy, ox) and
//    k = tap * (c0 + c1) + c read input pixel (oy*stride + ky - 1, ox*stride + kx - 1)
//    of the logical input (nearest x2 upsampled when up = 1), zero outside.
// Epilogue: v = acc + bias[n] + rowvec[m / rows_per_sample][n] + resid[m][n];
// geglu: columns come in 32-wide (value, gate) block pairs and the output
// column j of pair p is (acc_v + bias_v) * GELU(acc_g + bias_g).
struct GemmParams {
  const void* a0 = nullptr;
  const void* a1 = nullptr;
  int c0 = 0, c1 = 0;
  int lda0 = 0, lda1 = 0;
  int taps = 1;
  int in_h = 1, in_w = 1, up = 0;
  int out_h = 1, out_w = 1, stride = 1;
  const void* b = nullptr;
  int ldb = 0;
  int M = 0, N = 0, K = 0;
  const float* bias = nullptr;
  const float* rowvec = nullptr;
  int rowvec_ld = 0, rows_per_sample = 1;
  const void* resid = nullptr;
  int ldr = 0, resid_f32 = 0;
  void* out = nullptr;
  int ldo = 0, out_f32 = 0;
  int n_store = 0;  // output columns written
  int geglu = 0;
  const void* zero16 = nullptr;  // >= 16 zero bytes (implicit-conv padding reads of the fragment-B kernel)
  // Transposed V output: columns n >= vt_col0 (the V projection of an attention,
  // heads of vt_dp columns) are written to vt[sample][head][d][token] with token
  // stride 1 and d stride vt_ld; rows are tokens, vt_seq per sample.
  void* vt = nullptr;
  int vt_col0 = 0, vt_dp = 0, vt_heads = 0, vt_seq = 1, vt_ld = 0;
  // Split-K workspace (fragment-B kernel): fp32 partial slabs [split][M][n_store].
  float* part = nullptr;
  size_t part_floats = 0;
  // Raw partial output: write the slabs (even unsplit) and skip the reduction and the
  // epilogue; a later kernel (layernorm_reduce) completes them.
  int raw_partial = 0;
  // fp8 kernel (gemm_fp8): per-output-row fp32 weight scales (the accumulator of column n
  // is multiplied by wscale[n]); out_fp8: the output is E4M3 codes.
  const float* wscale = nullptr;
  int out_fp8 = 0;
};

// Block tile (bm x bn) of one GEMM launch and the kernel that runs it.
struct GemmPlan {
  int bm, bn;
  int stages = 2;        // fragment-B kernel variant: 3 the default (three LDS stages), 2 the 128 x 256
                         // tile at one workgroup per CU, 5 the 160-column tile on four waves,
                         // 13 / 14 stage read-ahead with three / four stages
  int frag = 0;          // 1: bf16 fragment-B kernel (gemm_frag.hip), else the register-staged kernel
  int split = 1;         // fragment-B kernel: K split in this many ranges (fp32 partials + reduce)
  int tail_bands = 0;    // fragment-B 128 x 256 tiles: the last column bands as 64-row tiles
};
constexpr int kMaxSplit = 8;
// allow_split = false for epilogues split-K does not support (the per-head V^T output);
// fused_reduce: the partial slabs are summed by the consumer (layernorm_reduce), so a
// split costs only the extra slab reads.
template <typename T>
GemmPlan gemm_plan(int M, int N, int K, int geglu, int cus, bool allow_split = true, bool fused_reduce = false,
                   bool conv = false);
template <typename T> void gemm(const GemmParams& p, const GemmPlan& g, hipStream_t s);
// The fragment-B kernel's tile plan (cost model fitted to measured SD-XL GEMM times).
GemmPlan frag_plan(int M, int N, int K, int geglu, int cus, bool allow_split, bool fused_reduce, bool conv);
void gemm_bf16_frag(const GemmParams& p, const GemmPlan& g, hipStream_t s);
// bf16 weight matrices [N][K] with gemm_frag_layout(N, K) are stored in MFMA fragment
// order (gemm_frag.hip) and multiplied by the fragment-B kernel; every other shape,
// and fp32, keeps the row-major [N][K] layout.
bool gemm_frag_layout(int N, int K);
// fp8 (E4M3) GEMM: A fp8 codes [M][lda], B a matrix packed by pack_fp8 (codes in the
// fragment order of the 32x32x64 fp8 matrix-core step, fp32 row scales in p.wscale);
// N % 32 == 0, K % 128 == 0. Tile plans 128 x 256 and 128 x 128, split-K as gemm_plan.
GemmPlan gemm_plan_fp8(int M, int N, int K, int geglu, int cus, bool allow_split, bool fused_reduce);
void gemm_fp8(const GemmParams& p, const GemmPlan& g, hipStream_t s);
bool gemm_fp8_layout(int N, int K);
size_t gemm_fp8_code_bytes(int N, int K);  // N rounded up to 32, times K
size_t gemm_frag_elems(int N, int K);  // N rounded up to 32, times K
void to_frag(const bf16* src, int N, int K, int ld_src, bf16* dst, hipStream_t s);
// fp32 workspace floats the plan needs (split-K partial slabs), 0 when none.
inline size_t gemm_workspace_floats(const GemmPlan& g, int M, int N, bool raw_partial = false) {
  return g.frag && (g.split > 1 || raw_partial) ? (size_t)g.split * M * N : 0;
}
template <typename T> constexpr int gemm_bk() { return sizeof(T) == 2 ? 64 : 32; }

// ---------------------------------------------------------------- attention
// O = softmax(Q K^T * scale) V per (sample, head). Head h occupies columns
// [h*D, h*D + D) of q, k and o (D = 32 or 64); V is given transposed per head:
// vt[((b * heads + h) * D + d) * vt_ld + key], vt_ld >= Skv rounded up to 64
// (keys past Skv must hold finite values; they get zero weight).
struct AttnParams {
  const void* q = nullptr;
  const void* k = nullptr;
  const void* vt = nullptr;
  void* o = nullptr;
  int ldq = 0, ldk = 0, ldo = 0, vt_ld = 0;
  long long q_bs = 0, k_bs = 0, o_bs = 0;  // per-sample strides (elements)
  int B = 0, heads = 0, Sq = 0, Skv = 0;
  float scale_log2 = 0.f;  // scale * log2(e)
};
template <typename T> void attention(const AttnParams& p, int D, hipStream_t s);

// ---------------------------------------------------------------- norms
// GroupNorm over NHWC [n][HW][c0 + c1] (two channel sources). Statistics in
// fp32 partial sums merged in fp64; apply writes y (contiguous [n][HW][C]).
struct GroupNormParams {
  const void* x0 = nullptr;
  const void* x1 = nullptr;
  int c0 = 0, c1 = 0;
  int n = 0, HW = 0, G = 0;
  const float* gamma = nullptr;
  const float* beta = nullptr;
  float eps = 1e-5f;
  int silu = 0;
  void* y = nullptr;
  float* partial = nullptr;  // workspace, groupnorm_workspace_floats()
  float* stats = nullptr;    // workspace [2][n][C]: per-channel scale, then shift
};
size_t groupnorm_workspace_floats(int n, int HW, int C, int G);
template <typename T> void groupnorm(const GroupNormParams& p, hipStream_t s);

template <typename T>
void layernorm(const float* x, T* y, long long M, int C, const float* gamma, const float* beta, float eps,
               hipStream_t s);
// LayerNorm that first completes a residual update: x = (resid ? x : 0) + bias +
// sum_s part[s] (nsplit fp32 slabs [M][C], summed in order), written back to x.
template <typename T>
void layernorm_reduce(float* x, T* y, long long M, int C, const float* gamma, const float* beta, float eps,
                      const float* part, int nsplit, const float* bias, bool resid, hipStream_t s);

// ---------------------------------------------------------------- misc
void abar_table(double* abar, int T, double beta_start, double beta_end, int schedule, hipStream_t s);
constexpr int kTsChunk = 256;
struct TsChunk {
  int count;
  int t[kTsChunk];
};
// out[s][.] = sinusoidal features of timestep c.t[s], s < c.count (fp64 evaluation)
void sinusoid(float* out, const TsChunk& c, int dim, hipStream_t s);
// out[s][j] = sum_k act(in[s][k]) * w[j][k] + b[j] (fp32; act = SiLU if silu)
void skinny_linear(const float* in, int S, int K, const float* w, const float* b, int J, float* out, int ld_out,
                   int silu, hipStream_t s);
template <typename T>
void latent_to_input(const float* latent, T* xin, int B, int C, int HW, int Cpad, hipStream_t s);
template <typename T>
void cfg_ddim(const float* eps, float* latent, T* xin, const double* abar, int t, int t_prev, float scale, int B,
              int C, int HW, int Cpad, hipStream_t s);
void export_eps(const float* eps, float* raw, float* guided, float scale, int B, int C, int HW, hipStream_t s);
template <typename T> void convert_from_f32(const float* src, T* dst, long long n, hipStream_t s);
void bf16_latent_to_f32(const uint16_t* src, float* dst, long long n, hipStream_t s);

// Weight packing: dst[r][c] (ld_dst) from an fp32 PyTorch-layout source.
struct PackParams {
  void* dst = nullptr;
  int rows = 0, cols = 0, ld_dst = 0;
  const float* src = nullptr;
  int row_mode = 0;  // 0 identity, 1 GEGLU interleave, 2 head padding
  int col_mode = 0;  // 0 identity, 1 head padding, 2 conv3x3 tap-major
  int src_rows = 0, src_cols = 0;  // source matrix [src_rows][src_cols]
  int D = 0, Dp = 0;               // head dim and padded head dim
  int Cin = 0, Cinp = 0;           // conv input channels and padded count
  int frag = 0;                    // 1: write dst in fragment order (gemm_frag.hip; ld_dst unused)
};
template <typename T> void pack(const PackParams& p, hipStream_t s);
// E4M3 quantisation of a [rows][cols] fp32 source (the same row mapping as pack; column
// mode 0 only): per destination row r, scale[r] = max_c |src| / 448 (1 for a zero row)
// and code = round(src / scale) (nearest even, saturating), written in the fp8
// fragment order to p.dst (bytes); rows past the source (up to a multiple of 32) are zero.
void pack_fp8(const PackParams& p, float* scales, hipStream_t s);
void pack_bias(float* dst, int n, const float* src, int src_n, int row_mode, int D, int Dp, hipStream_t s);

// ---------------------------------------------------------------- cache lookup
// Similarity-driven approximation level: a retrieved cosine s gets level[j],
// j = #{i < n : s >= thr[i]} (fp32 comparisons); a query that retrieved nothing gets 0.
constexpr int kMaxKLevels = 16;
struct KTable {
  int n = 0;
  float thr[kMaxKLevels - 1] = {};
  int level[kMaxKLevels] = {};
};
// Top-1 cosine row of cache [n][dim] (fp16) for q [dim]: writes the index (-1 when no
// row has a defined cosine) and the cosine to idx_out / score_out, which may be device
// memory or pinned host memory. ws: lookup_workspace_bytes() of device memory.
size_t lookup_workspace_bytes();
// With k_out != nullptr the reduction also writes the level of kt for the result.
void lookup(const uint16_t* q, const uint16_t* cache, long long n, int dim, void* ws, long long* idx_out,
            float* score_out, hipStream_t s, const KTable* kt = nullptr, int* k_out = nullptr);
// Top-1 rows of cache [n][dim] for nq <= lookup_batch_max_queries() queries q [nq][dim]
// in one pass over the table (matrix-core scores). idx_out / score_out [nq] (device or
// pinned host memory); idx -1 for a query with no defined cosine. Needs
// lookup_batch_supported(q, cache, dim); ws: lookup_batch_workspace_bytes().
size_t lookup_batch_workspace_bytes();
int lookup_batch_max_queries();
bool lookup_batch_supported(const uint16_t* q, const uint16_t* cache, long long n, int dim);
void lookup_batch(const uint16_t* q, int nq, const uint16_t* cache, long long n, int dim, void* ws,
                  long long* idx_out, float* score_out, hipStream_t s, const KTable* kt = nullptr,
                  int* k_out = nullptr);

}  // namespace dn
