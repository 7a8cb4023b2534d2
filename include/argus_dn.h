/*
 * argus_dn.h — C ABI of the MI355X (gfx950) denoise-loop library.
 *
 * Hot path of the Argus serving method (arXiv 2511.06724): the GPU worker of
 * Sec. 4.5 / Sec. 4.7 either starts from Gaussian noise or, under approximate
 * caching (AC, Sec. 2.1), finds the most similar cached prompt by embedding
 * similarity, takes that prompt's intermediate latent at iteration K and runs
 * the remaining N-K denoising iterations conditioned on the new prompt. Each
 * iteration is one UNet evaluation (the compute-bound component of Table 3 and
 * Observation 5, Sec. 3.2) with classifier-free guidance, then a DDIM update.
 *
 * Calls:
 *   dn_weight_count / dn_weight_table  size and describe the canonical weight blob
 *   dn_create                          build a denoiser (pack weights for the GPU)
 *   dn_denoise                         run iterations [start_step, start_step + n_steps)
 *   dn_denoise_capture                 the same, writing the latent after chosen iterations (cache write)
 *   ac_lookup                          top-1 cosine search over the prompt-embedding cache
 *   ac_lookup_batch                    the same search for many queries in one pass over the cache
 *   ac_lookup_batch_k                  ac_lookup_batch + the approximation level K chosen from the similarity
 *   ac_lookup_batch_noalloc            ac_lookup_batch on a stream, results in device memory, no allocation
 *   ac_fetch_latent                    copy cached latent #idx into an fp32 latent buffer
 *   dn_unet_eps                        one UNet evaluation + guidance (per-step check hook)
 *   dn_vae_*                           the latent decoder after the loop (Table 3's VAE Decoder)
 *   dn_op_*                            single-kernel entry points (kernel checks, timing)
 *   dn_probe_mfma_rate                 measurement: the matrix-core rate the device sustains
 *   dn_destroy, dn_last_error
 *   argus_oda, argus_route, argus_select_worker   routing control plane on the host (Sec. 4.3-4.4)
 *
 * Conventions (every call):
 *   - Pointers marked "device" are HIP device allocations owned by the caller;
 *     they must stay valid until the work enqueued on `stream` has finished.
 *     Pointers marked "host" are read or written during the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Calls that take a stream only enqueue work and return; calls that do not
 *     take one are synchronous.
 *   - Every argument is checked before any work is enqueued: on DN_EINVAL
 *     nothing was enqueued and no output was touched. HIP runtime failures
 *     return DN_EHIP. dn_last_error() gives a message for the calling thread.
 *   - Floating-point data: fp32 = IEEE binary32; fp16 and bf16 buffers are
 *     passed as uint16_t bit patterns (IEEE binary16 / bfloat16).
 *   - All results are deterministic: the same inputs give bitwise equal outputs
 *     (no floating-point atomics; all reductions run in a fixed order).
 */
#ifndef ARGUS_DN_H
#define ARGUS_DN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DN_ABI_VERSION 1
#define DN_MAX_LEVELS 4

typedef struct dn_handle dn_handle; /* opaque: packed device weights + workspace */

typedef enum {
  DN_OK = 0,
  DN_EINVAL = -1,       /* invalid argument or configuration */
  DN_ENOMEM = -2,       /* device or host allocation failed */
  DN_EHIP = -3,         /* HIP runtime error */
  DN_EUNSUPPORTED = -4  /* valid but not supported by the library as built (e.g. no gfx950 device) */
} dn_status;

typedef enum { DN_FP32 = 0, DN_BF16 = 1, DN_FP8 = 2 } dn_dtype;
typedef enum { DN_WEIGHTS_HOST = 0, DN_WEIGHTS_DEVICE = 1 } dn_weights_location;
typedef enum { DN_BETA_LINEAR = 0, DN_BETA_SCALED_LINEAR = 1 } dn_beta_schedule;

/* One resolution level of the UNet. depth = transformer blocks per attention
 * stage (0 = ResNet blocks only). heads * head_dim must equal channels. */
typedef struct {
  int32_t channels;
  int32_t depth;
  int32_t heads;
  int32_t head_dim;
} dn_level;

/* A latent-diffusion UNet and its sampler schedule. The parameter counts of
 * this topology reproduce Table 3's SD-XL and SD 2.0 UNets exactly (SD-XL's
 * added-condition MLP aside, which the denoise loop does not use).
 *
 * dtype          DN_BF16: weights and activations bf16 with fp32 accumulation;
 *                norm statistics, softmax, the time embedding, the transformer
 *                residual stream, the latent and the DDIM update stay fp32.
 *                DN_FP32: everything fp32.
 *                DN_FP8: the quantized variant (quantized models are approximation
 *                levels, Sec. 4.2): DN_BF16 except the GEGLU feed-forward of every
 *                transformer block, whose two matrices are OCP E4M3 codes with one
 *                fp32 scale per output row (row max / 448) and whose two inputs (the
 *                third LayerNorm's output, the GEGLU output) are E4M3 at scale 1
 *                (nearest even, saturating at 448), multiplied on the fp8 matrix cores.
 * batch          images B; the UNet runs on 2B rows (B unconditional, then B
 *                conditional) for classifier-free guidance.
 * latent_*       latent channels (<= 64) and spatial size; H and W must be
 *                divisible by 2^(n_levels-1).
 * model_channels C0: width of conv_in and of the sinusoidal timestep features;
 *                the time embedding has 4*C0 features.
 * level[]        n_levels (1..4) levels, coarsening by 2 between levels.
 * layers_per_block  ResNet(+transformer) layers per down level; up levels have one more.
 * mid_depth      -1: no middle block; 0: ResBlock, ResBlock; >0: ResBlock,
 *                transformer of mid_depth blocks, ResBlock (at the last level's width).
 * tiny_topology  1: conv_in -> ResBlock -> transformer(level[0].depth) -> out head
 *                (level 0 only; no skips, no middle block, no up path).
 * ctx_len, ctx_dim  text-encoder context tokens and width (cross-attention keys).
 * ff_mult        GEGLU feed-forward width multiplier (inner width ff_mult*C).
 * gn_groups      GroupNorm groups (channel counts must be divisible by it).
 * gn_eps         GroupNorm epsilon of ResBlocks and the out head; tx_gn_eps of
 *                the transformer's input GroupNorm; ln_eps of its LayerNorms.
 * n_train_steps, beta_start, beta_end, beta_schedule   the training noise
 *                schedule; abar_t = prod_{i<=t} (1 - beta_i).
 */
typedef struct {
  int32_t abi_version; /* must be DN_ABI_VERSION */
  int32_t dtype;
  int32_t batch;
  int32_t latent_c, latent_h, latent_w;
  int32_t model_channels;
  int32_t n_levels;
  dn_level level[DN_MAX_LEVELS];
  int32_t layers_per_block;
  int32_t mid_depth;
  int32_t tiny_topology;
  int32_t ctx_len, ctx_dim, ff_mult, gn_groups;
  float gn_eps, tx_gn_eps, ln_eps;
  int32_t n_train_steps;
  float beta_start, beta_end;
  int32_t beta_schedule;
} dn_config;

/* Number of fp32 values in the canonical weight blob of `cfg`.
 * The blob is every tensor of the model back to back, in PyTorch layouts
 * (conv [Cout][Cin][kh][kw], linear [out][in]), in this order:
 *  1. time MLP: lin1.w [4C0][C0], lin1.b, lin2.w [4C0][4C0], lin2.b
 *  2. conv_in.w [C0][latent_c][3][3], conv_in.b
 *  3. down levels l = 0..L-1: layers_per_block x (ResBlock, then transformer if
 *     depth_l > 0), then for l < L-1 a stride-2 downsample conv [C_l][C_l][3][3] + bias
 *  4. middle block (mid_depth >= 0): ResBlock, transformer(mid_depth) if > 0, ResBlock
 *  5. up levels l = L-1..0: (layers_per_block + 1) x (ResBlock on the channel
 *     concatenation [h, skip], transformer if depth_l > 0), then for l > 0 a
 *     nearest-x2 upsample followed by conv [C_l][C_l][3][3] + bias
 *  6. out head: GroupNorm scale, shift [C0]; conv_out.w [latent_c][C0][3][3], conv_out.b
 * ResBlock(Cin -> Cout): gn1 scale, shift [Cin]; conv1.w [Cout][Cin][3][3], conv1.b;
 *   temb.w [Cout][4C0], temb.b; gn2 scale, shift [Cout]; conv2.w [Cout][Cout][3][3],
 *   conv2.b; if Cin != Cout a 1x1 skip conv skip.w [Cout][Cin][1][1], skip.b.
 * Transformer(C, depth): gn scale, shift; proj_in.w [C][C], proj_in.b; depth x
 *   { ln1 scale, shift; attn1 q, k, v [C][C] (no bias); attn1 out.w [C][C], out.b;
 *     ln2 scale, shift; attn2 q [C][C], k [C][ctx_dim], v [C][ctx_dim]; attn2 out.w, out.b;
 *     ln3 scale, shift; ff1.w [2*F*C][C], ff1.b (first half value, second half gate);
 *     ff2.w [C][F*C], ff2.b }; proj_out.w [C][C], proj_out.b.
 * Returns DN_EINVAL for an invalid configuration. */
dn_status dn_weight_count(const dn_config* cfg, size_t* n_floats);

/* Describes the blob tensor by tensor: for tensor i (canonical order),
 * numel[i] elements, fan_in[i] = the layer's input size (Cin*kh*kw or
 * in_features; also given for its bias; 0 for norm parameters) and kind[i] =
 * 0 weight, 1 bias, 2 norm scale, 3 norm shift. Arrays are host memory with
 * room for `capacity` entries (NULL arrays with capacity 0 query the count);
 * *n_tensors receives the tensor count. DN_EINVAL if capacity is too small. */
dn_status dn_weight_table(const dn_config* cfg, int64_t* numel, int32_t* fan_in, int32_t* kind,
                          size_t capacity, size_t* n_tensors);

/* Builds a denoiser, i.e. one loaded model of a GPU worker (Sec. 4.5: a worker
 * serves one model variant at a time; Table 3 sizes the UNets): validates cfg,
 * copies the fp32 blob (n_floats values, host or device memory per
 * `weights_location`; n_floats must equal dn_weight_count) and repacks it on the
 * GPU into kernel layouts in the configured dtype. The caller keeps ownership of
 * the blob. Synchronous. On success *out receives the handle, which owns the
 * packed weights and the per-call workspace (freed by dn_destroy); on error
 * *out is untouched and nothing stays allocated. DN_EUNSUPPORTED when the
 * current device is not gfx950. */
dn_status dn_create(const dn_config* cfg, const float* weights, size_t n_floats, int32_t weights_location,
                    dn_handle** out);

/* Denoise loop (Sec. 2.1, Sec. 4.7): for i = start_step .. start_step+n_steps-1,
 *   eps_raw = UNet([x; x], t_i, text_ctx)             (2B rows)
 *   eps     = eps_u + cfg_scale * (eps_c - eps_u)     (classifier-free guidance)
 *   x       = sqrt(abar_prev) * x0 + sqrt(1 - abar_prev) * eps,
 *             x0 = (x - sqrt(1 - abar_t) * eps) / sqrt(abar_t)   (DDIM, eta = 0)
 * with t_i = timesteps[i], abar_t = abar[t_i], abar_prev = abar[timesteps[i+1]]
 * and timestep -1 meaning the clean sample (abar = 1).
 * latent     device fp32 [B][latent_c][H][W], read and updated in place: on entry
 *            it is x at timesteps[start_step] (for AC, the cached intermediate
 *            latent of iteration K = start_step), on return x at
 *            timesteps[start_step + n_steps].
 * text_ctx   device fp32 [2B][ctx_len][ctx_dim]: B unconditional rows, then B conditional.
 * timesteps  host int32, n_timesteps >= start_step + n_steps + 1 entries, each in
 *            [-1, n_train_steps).
 * n_steps = 0 enqueues nothing. Asynchronous on `stream`. One handle serves one
 * stream at a time (its workspace is reused by every call). */
dn_status dn_denoise(dn_handle* h, float* latent, const float* text_ctx, const int32_t* timesteps,
                     int32_t n_timesteps, int32_t start_step, int32_t n_steps, float cfg_scale, void* stream);

/* Denoise loop that also writes the cache (Sec. 4.7: every prompt stores its
 * intermediate states at K, which later prompts resume from, Sec. 2.1): runs
 * exactly dn_denoise(h, latent, text_ctx, timesteps, n_timesteps, start_step,
 * n_steps, cfg_scale, stream) and, for each j < n_capture, writes the latent
 * after capture_at[j] iterations, i.e. x at timesteps[capture_at[j]], rounded to
 * bf16 (nearest, ties to even), to out_latents + j * B*latent_c*H*W.
 * capture_at   host int32 [n_capture], each in [start_step, start_step + n_steps]
 *              (start_step captures the input latent); read during the call only.
 * out_latents  device bf16 [n_capture][B][latent_c][H][W], the layout of the cache's
 *              latent table (a slot is what ac_fetch_latent reads back).
 * n_capture = 0 is dn_denoise. Capture arguments are checked with the others,
 * before anything is enqueued. Asynchronous on `stream`; the result latent and
 * the final state are bitwise those of dn_denoise. */
dn_status dn_denoise_capture(dn_handle* h, float* latent, const float* text_ctx, const int32_t* timesteps,
                             int32_t n_timesteps, int32_t start_step, int32_t n_steps, float cfg_scale,
                             const int32_t* capture_at, int32_t n_capture, uint16_t* out_latents, void* stream);

/* One UNet evaluation + guidance at timestep t (no DDIM update), for checking a
 * single iteration. x device fp32 [B][latent_c][H][W]; text_ctx as in dn_denoise;
 * out_raw device fp32 [2B][latent_c][H][W] (UNet output on [x; x]);
 * out_guided device fp32 [B][latent_c][H][W] (eps after guidance) or NULL.
 * Asynchronous on `stream`. */
dn_status dn_unet_eps(dn_handle* h, const float* x, int32_t t, const float* text_ctx, float cfg_scale,
                      float* out_raw, float* out_guided, void* stream);

/* Nearest cached prompt (Sec. 2.1; Sec. 4.7): argmax_i of the cosine similarity
 * (q . c_i) / (|q| |c_i|) over the n rows of the cache, ties going to the
 * lowest index. query_emb device fp16 [dim]; cache_embs device fp16 [n][dim]
 * (row-major). Products and sums in fp32. On success *out_idx (host) receives
 * the index and, if out_score (host) is not NULL, *out_score the cosine.
 * Synchronous (default stream). n >= 1, dim >= 1; the query must be non-zero.
 * On error *out_idx is left untouched (the caller falls back to K = 0).
 * The first call on a device allocates that device's scan workspace (32 KB) and a
 * 256-byte pinned host buffer the result is written to; both are kept until the
 * process ends, and calls that overlap on one device (from several threads) race
 * on them. */
dn_status ac_lookup(const uint16_t* query_emb, const uint16_t* cache_embs, int64_t n, int32_t dim,
                    int64_t* out_idx, float* out_score);

/* Batched nearest cached prompt (Sec. 2.1; Sec. 4.7): for each of the nq queries
 * of query_embs (device fp16 [nq][dim], row-major) the same search as ac_lookup
 * over cache_embs (device fp16 [n][dim]): out_idx[j] (host int64 [nq]) receives
 * the first row of maximal cosine with query j, or -1 when query j is zero (or
 * every row is), and out_score[j] (host float [nq], may be NULL) that cosine.
 * For dim 256, 512, 768 or 1024, 16-byte aligned pointers and n < 2^31 - 64, the table is read
 * once per 64 queries and the scores are matrix-core products (fp16 operands,
 * fp32 sums); other widths run one ac_lookup scan per query. Synchronous (default
 * stream). nq >= 1, n >= 1, dim >= 1; on an argument error nothing is written.
 * The first call on a device allocates that device's workspace (256 KB) and a
 * 768-byte pinned host result buffer, kept until the process ends; calls that
 * overlap on one device race on them. */
dn_status ac_lookup_batch(const uint16_t* query_embs, int32_t nq, const uint16_t* cache_embs, int64_t n, int32_t dim,
                          int64_t* out_idx, float* out_score);

/* Similarity-driven approximation level (Sec. 2.1: the retrieved prompt's similarity
 * decides the approximation level K, i.e. how many of the N iterations the cached
 * state lets the new prompt skip; more similar prompts tolerate a larger K). The
 * paper gives no rule; the table is an input of the caller (e.g. derived from
 * offline quality profiles): n_thresholds = L in [0, 15] strictly increasing finite
 * cosines t_1 < ... < t_L and L + 1 non-decreasing levels K_0 <= ... <= K_L (>= 0).
 * A retrieved cosine s (the fp32 value reported in out_score) gets K_j with
 * j = #{i : s >= t_i}; a query that retrieved nothing (index -1) gets K = 0. */
#define AC_MAX_K_LEVELS 16
typedef struct {
  int32_t n_thresholds;
  float threshold[AC_MAX_K_LEVELS - 1];
  int32_t level[AC_MAX_K_LEVELS];
} ac_k_table;

/* ac_lookup_batch that also returns the approximation level of every query
 * (out_k host int32 [nq]) from `table` (host, read during the call), computed on
 * the GPU from the same fp32 cosine it reports. The caller then resumes query j
 * from cached slot K = out_k[j] of row out_idx[j] (dn_denoise with start_step = K).
 * Synchronous; DN_EINVAL for a malformed table before anything runs. */
dn_status ac_lookup_batch_k(const uint16_t* query_embs, int32_t nq, const uint16_t* cache_embs, int64_t n,
                            int32_t dim, const ac_k_table* table, int64_t* out_idx, float* out_score,
                            int32_t* out_k);

/* For callers that cannot allocate — code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation: the search of ac_lookup_batch (same
 * kernels, same results bit for bit) enqueued on `stream`, with the results in
 * device memory and the per-workgroup winners in a fixed scratch array of the
 * library (256 KiB per GPU, held until the process ends). The call allocates
 * nothing (no hipMalloc, hipFree or pinned host memory) and does not synchronise.
 * out_idx    device int64 [nq]: first row of maximal cosine per query, -1 when the
 *            query is zero (or every row is).
 * out_score  device float [nq] (the cosines) or NULL.
 * Any nq >= 1 (passes of 64 queries run one after another on `stream`), n >= 1,
 * dim >= 1 (dim <= 16384 off the matrix-core widths 256/512/768/1024).
 * Every call on one GPU shares that GPU's scratch: calls that overlap on one GPU
 * (several streams or threads) race and must be serialised by the caller. Returns
 * DN_EINVAL before enqueuing anything if the scan would need more scratch than
 * the library holds. */
dn_status ac_lookup_batch_noalloc(const uint16_t* query_embs, int32_t nq, const uint16_t* cache_embs, int64_t n,
                                  int32_t dim, int64_t* out_idx, float* out_score, void* stream);

/* Copies cached latent #idx of a device bf16 table [n][numel] into the device
 * fp32 latent buffer [numel] (the resume state of Sec. 4.7). Asynchronous. */
dn_status ac_fetch_latent(const uint16_t* cache_latents, int64_t n, int64_t numel, int64_t idx, float* latent,
                          void* stream);

/* ---------------------------------------------------------------------------
 * Single-kernel entry points. They run exactly the kernels dn_denoise runs and
 * exist for element-wise checks at full size and for timing one kernel. A GEMM
 * whose tile plan splits K also runs the split-K reduction kernel; its partial
 * sums live in a per-device workspace the library allocates on first need and
 * keeps, so calls on one device must not overlap.
 * All buffers are device memory, row-major, in the element type `dtype`
 * (DN_BF16 -> bf16 bits, DN_FP32 -> fp32) unless stated otherwise.
 * ------------------------------------------------------------------------- */

/* Weight layout of the GEMM entry points below. A weight matrix w[N][K] (row n =
 * output column n; for the 3x3 convolution K = 9 * Cin, tap-major) is passed in
 * the library's packed layout, which depends only on (dtype, N, K): bf16 matrices
 * with N % 32 == 0 and K % 64 == 0 are stored in MFMA fragment order (for each
 * block of 32 rows and each 16 columns, the 64 16-byte operands of one matrix-core
 * instruction lie in 1 KB of contiguous memory); every other matrix, and every fp32
 * matrix, is row-major unchanged.
 * dn_packed_weight_elems: *elems = elements the packed matrix occupies (N rounded
 *   up to 32, times K, for the fragment order; N * K otherwise).
 * dn_pack_weight: packs a row-major device matrix w [N][K] (dtype elements) into
 *   `out` (device, dn_packed_weight_elems elements, not overlapping w). K must be a
 *   multiple of 16. Asynchronous on `stream`.
 * DN_FP8: w is fp32 [N][K] (N % 32 == 0, K % 128 == 0); `out` receives N * K bytes of
 *   E4M3 codes in the fragment order of the 32x32x64 fp8 matrix-core step (per 32 rows
 *   and 64-deep step, the lanes' 32-byte operands in 2 KB), code = round(w / scale_n),
 *   then N fp32 scales scale_n = max_k |w[n][k]| / 448 (1 for a zero row);
 *   dn_packed_weight_elems gives the total in bytes. */
dn_status dn_packed_weight_elems(int32_t dtype, int32_t N, int32_t K, int64_t* elems);
dn_status dn_pack_weight(int32_t dtype, const void* w, int32_t N, int32_t K, void* out, void* stream);

/* Dense layer (the transformer's projections and feed-forward):
 * y[m][n] = sum_k x[m][k] * w[n][k] + bias[n] (+ resid[m][n]).
 * x [M][K], w [N][K] packed by dn_pack_weight, bias fp32 [N] or NULL, resid
 * [M][N] or NULL, y [M][N].
 * K must be a multiple of 64 (bf16) / 32 (fp32). Output fp32 when y_f32 != 0,
 * else `dtype`; resid fp32 when resid_f32 != 0, else `dtype`.
 * geglu != 0 (GEGLU feed-forward, Shazeer 2020): w has 2N rows and bias 2N
 * entries, interleaved in blocks of 32 — rows [64j, 64j+32) are value rows
 * [32j, 32j+32) and rows [64j+32, 64j+64) the matching gate rows — and
 * y[m][n] = a * GELU(g) with a, g the value and gate outputs of column n
 * (exact erf GELU); N % 32 == 0 and resid must be NULL. Asynchronous.
 * DN_FP8: x E4M3 codes [M][K], w packed for DN_FP8 (K % 128 == 0; GEGLU value / gate
 *   rows interleaved as above before packing), accumulator column n scaled by scale_n;
 *   y fp32 when y_f32 != 0, else E4M3 codes when geglu != 0 (the input of the next fp8
 *   layer), else bf16; resid fp32 or bf16 per resid_f32. */
dn_status dn_op_linear(int32_t dtype, const void* x, const void* w, const float* bias, const void* resid,
                       int32_t resid_f32, void* y, int32_t y_f32, int64_t M, int32_t N, int32_t K, int32_t geglu,
                       void* stream);

/* 3x3 convolution (cross-correlation, zero padding 1, bias) as an implicit GEMM
 * on NHWC activations: x [n][H][W][Cin]; with up = 1 the input is first
 * nearest-neighbour upsampled to 2H x 2W (never materialised); stride 1 or 2.
 * w [Cout][3][3][Cin] (tap-major: PyTorch [Cout][Cin][3][3] permuted; packed by
 * dn_pack_weight as an N = Cout, K = 9 * Cin matrix), bias fp32
 * [Cout] or NULL, temb fp32 [n][Cout] or NULL (added per sample, as a ResBlock
 * adds its time-embedding projection), resid [n][Ho][Wo][Cout] or NULL,
 * y [n][Ho][Wo][Cout] with Ho = (Hl - 1) / stride + 1 for the logical input
 * height Hl (same for W); fp32 output when y_f32 != 0. Cin must be a multiple
 * of 64 (bf16) / 32 (fp32). Asynchronous. */
dn_status dn_op_conv3x3(int32_t dtype, const void* x, int32_t n, int32_t H, int32_t W, int32_t Cin, int32_t up,
                        int32_t stride, const void* w, const float* bias, const float* temb, const void* resid,
                        void* y, int32_t Cout, int32_t y_f32, void* stream);

/* Attention core O = softmax(Q K^T * scale) V for each (sample, head), the
 * score matrix never materialised (flash-style, fp32 softmax):
 * q [B][Sq][ldq], k [B][Skv][ldk], o [B][Sq][ldo]; head h occupies columns
 * [h * head_stride, (h + 1) * head_stride) of each, head_stride 32 or 64.
 * V is given transposed per head, as the projection GEMM writes it (see
 * dn_op_linear_vt): vt [B][heads][head_stride][vt_ld], keys contiguous, with
 * vt_ld >= Skv rounded up to 64 and finite values (e.g. zeros) in keys
 * [Skv, vt_ld). A head of d < head_stride real dimensions must hold zeros in its
 * padding columns of q and k. Asynchronous. */
dn_status dn_op_attention(int32_t dtype, const void* q, int32_t ldq, const void* k, int32_t ldk, const void* vt,
                          int32_t vt_ld, void* o, int32_t ldo, int32_t B, int32_t heads, int32_t Sq, int32_t Skv,
                          int32_t head_stride, float scale, void* stream);

/* Attention input projection with the V part written transposed per head:
 * acc[m][n] = sum_k x[m][k] * w[n][k] + bias[n] for n < N; columns n < vt_col0
 * go to y [M][vt_col0] (e.g. Q and K), columns n >= vt_col0 (heads * head_stride
 * of them) go to vt [M / seq][heads][head_stride][vt_ld] at token m % seq.
 * w packed by dn_pack_weight. Same kernels and tile plan as dn_op_linear.
 * Asynchronous. */
dn_status dn_op_linear_vt(int32_t dtype, const void* x, const void* w, const float* bias, void* y, int64_t M,
                          int32_t N, int32_t K, int32_t vt_col0, void* vt, int32_t heads, int32_t head_stride,
                          int32_t seq, int32_t vt_ld, void* stream);

/* GroupNorm (Wu & He 2018) over NHWC x [n][HW][C] with G groups: biased
 * variance, statistics from fp32 partial sums merged in fp64,
 * y = x_hat * gamma[c] + beta[c], then SiLU if silu != 0. gamma, beta fp32 [C];
 * C % G == 0 and C a multiple of 16 bytes of elements. Asynchronous. Its partial sums
 * live in the per-device workspace of the single-kernel entry points (grown on
 * first need; growing it synchronises the device). */
dn_status dn_op_groupnorm(int32_t dtype, const void* x, void* y, int32_t n, int32_t HW, int32_t C, int32_t G,
                          const float* gamma, const float* beta, float eps, int32_t silu, void* stream);

/* LayerNorm over the last axis: x fp32 [M][C] (the residual stream), y [M][C]
 * in `dtype` (E4M3 codes for DN_FP8, nearest even, saturating); C a multiple of 4, at
 * most 2048. Asynchronous. */
dn_status dn_op_layernorm(int32_t dtype, const float* x, void* y, int64_t M, int32_t C, const float* gamma,
                          const float* beta, float eps, void* stream);

/* LayerNorm that first completes a residual-stream update whose GEMM split K into
 * nsplit fp32 partial slabs (the transformer block's out-projection or FF-out feeding
 * the next LayerNorm, Table 3's SD-XL blocks): for every row,
 *   x = (resid ? x : 0) + bias + slabs[0] + ... + slabs[nsplit-1]   (fp32, in this order)
 * is written back to x, then y = LayerNorm(x) * gamma + beta as in dn_op_layernorm.
 * x fp32 [M][C] (in/out), slabs fp32 [nsplit][M][C], bias fp32 [C] or NULL, y [M][C]
 * in `dtype`; 1 <= nsplit <= 8; C a multiple of 4, at most 2048; x, slabs, bias, gamma
 * and beta 16-byte aligned. Asynchronous. */
dn_status dn_op_layernorm_slabs(int32_t dtype, float* x, void* y, int64_t M, int32_t C, const float* gamma,
                                const float* beta, float eps, const float* slabs, int32_t nsplit, const float* bias,
                                int32_t resid, void* stream);

/* Measurement entry point, not a step of the method: the bf16 rate the matrix cores of
 * the current device sustain and the shader clock they hold meanwhile, the ceiling the
 * GEMM and attention rooflines are read against beside the published peak. One
 * workgroup of four waves per CU issues `iters` (1 .. 2^20) rounds of eight independent
 * 32x32x16 bf16 MFMAs per wave; *tflops (host) = MFMA FLOPs / event time of the launch
 * (after one untimed launch), *clock_ghz (host) = the waves' cycle counts over the 100 MHz
 * constant counter. Synchronous (default stream); allocates and frees a few KB. */
dn_status dn_probe_mfma_rate(int32_t iters, double* tflops, double* clock_ghz);

/* ---------------------------------------------------------------------------
 * Latent decoder: the VAE Decoder of Table 3 (0.050 B parameters, 2481 GFLOP for a
 * 512 x 512 image), run once per image after the denoise loop to turn the final
 * latent into the RGB image. KL-autoencoder decoder of latent diffusion:
 *   z / scaling_factor -> 1x1 conv (latent_c -> latent_c) -> conv3x3 (-> C_top)
 *   -> ResBlock, single-head self-attention over all positions, ResBlock (at C_top)
 *   -> up levels l = n_levels-1 .. 0: (layers_per_block + 1) ResBlocks at width
 *      channels[l] (a 1x1 skip conv where the width changes), then for l > 0 a
 *      nearest-x2 upsample followed by conv3x3
 *   -> GroupNorm, SiLU, conv3x3 (channels[0] -> out_c).
 * ResBlock(x) = skip(x) + conv2(SiLU(GN2(conv1(SiLU(GN1(x)))))) (no time input);
 * every GroupNorm has gn_groups groups and epsilon gn_eps; the attention's q, k, v and
 * output projections are linear layers with bias, softmax scale 1/sqrt(C_top).
 * ------------------------------------------------------------------------- */
typedef struct dn_vae dn_vae; /* opaque: packed device weights + workspace of one decoder */

/* dtype as in dn_config; batch images; latent_c (<= 64), latent_h x latent_w
 * (a multiple of 64 positions, at most 65536); n_levels (1..4) widths channels[]
 * (multiples of 64, <= 2048, divisible by gn_groups), slowest resolution last; the
 * image is 2^(n_levels-1) times the latent in each direction (at most 4 M pixels). */
typedef struct {
  int32_t abi_version; /* must be DN_ABI_VERSION */
  int32_t dtype;
  int32_t batch;
  int32_t latent_c, latent_h, latent_w;
  int32_t n_levels;
  int32_t channels[DN_MAX_LEVELS];
  int32_t layers_per_block;
  int32_t gn_groups;
  float gn_eps;
  float scaling_factor;
  int32_t out_c;
} dn_vae_config;

/* Canonical fp32 blob of a decoder (PyTorch layouts, conv [Cout][Cin][kh][kw],
 * linear [out][in]): post_quant.w [latent_c][latent_c][1][1], .b; conv_in.w, .b;
 * mid.res0; mid.attn: gn scale, shift, q.w [C][C], q.b, k.w, k.b, v.w, v.b, o.w, o.b;
 * mid.res1; up levels l = n_levels-1 .. 0: (layers_per_block + 1) ResBlocks, then
 * (l > 0) up.w [C_l][C_l][3][3], up.b; out GroupNorm scale, shift; conv_out.w, .b.
 * ResBlock(Cin -> Cout): gn1 scale, shift [Cin]; conv1.w, .b; gn2 scale, shift
 * [Cout]; conv2.w, .b; if Cin != Cout skip.w [Cout][Cin][1][1], skip.b.
 * dn_vae_weight_table describes it tensor by tensor as dn_weight_table does. */
dn_status dn_vae_weight_count(const dn_vae_config* cfg, size_t* n_floats);
dn_status dn_vae_weight_table(const dn_vae_config* cfg, int64_t* numel, int32_t* fan_in, int32_t* kind,
                              size_t capacity, size_t* n_tensors);

/* Builds a decoder: validates cfg, copies and packs the blob (host or device memory
 * per weights_location; the caller keeps it) in the configured dtype and allocates
 * the workspace of one decode (for a 128 x 128 latent about 4 GB in bf16, including
 * the 16384 x 16384 fp32 attention scores). Synchronous. DN_EUNSUPPORTED when the
 * current device is not gfx950. */
dn_status dn_vae_create(const dn_vae_config* cfg, const float* weights, size_t n_floats, int32_t weights_location,
                        dn_vae** out);

/* Decodes latent (device fp32 [batch][latent_c][H][W], e.g. the latent dn_denoise
 * leaves) into image (device fp32 [batch][out_c][H'][W'], H' = 2^(n_levels-1) H).
 * Asynchronous on `stream`; one decoder serves one stream at a time. */
dn_status dn_vae_decode(dn_vae* v, const float* latent, float* image, void* stream);

void dn_vae_destroy(dn_vae* v); /* NULL-safe; synchronizes the device first */

/* ---------------------------------------------------------------------------
 * Routing control plane (host only, no GPU work; Sec. 4.3-4.4). Approximation levels
 * are indexed 0 .. n-1 from the slowest / most accurate to the fastest / most
 * approximate (for approximate caching: increasing K). All arrays are host memory
 * read or written during the call. These calls report errors through
 * argus_last_error(), not dn_last_error().
 * ------------------------------------------------------------------------- */
#define ARGUS_MAX_LEVELS 64

/* Optimized Distribution Aligner (Sec. 4.3, Alg. 1): from the classifier's demand
 * histogram H[n] (share of prompts whose optimal level is i) and the solver's load
 * split F[n] (share of the load each level serves; sum F = sum H > 0, both
 * non-negative), writes the Probabilistic Approximation Shift Map pasm[n][n]
 * (row-major): pasm[i][j] = probability that a prompt whose optimal level is i is
 * served at level j. Levels are visited from the fastest to the slowest: excess
 * demand moves to the next slower level (proportionally for all prompts present
 * there), a shortfall is filled from the nearest slower levels first. Every row sums
 * to 1 and sum_i H[i] pasm[i][j] = F[j]. A row with H[i] = 0 is the identity. */
dn_status argus_oda(const double* H, const double* F, int32_t n, double* pasm);

/* Prompt Scheduler (Sec. 4.4): the level a prompt whose optimal level is `level` is
 * sent to, drawn from PASM row `level` with a uniform number u in [0, 1) supplied by
 * the caller: the first j whose cumulative probability (from level 0) exceeds u, or
 * the last level of positive probability if rounding leaves the row sum <= u. */
dn_status argus_route(const double* pasm, int32_t n, int32_t level, double u, int32_t* out_level);

/* Worker selector, Eq. 3 (Sec. 4.4): among the n_workers workers whose
 * worker_level[w] equals `level`, the one minimising queue_len[w] * t_proc[w] (queued
 * requests times its generation time at that level), lowest w on ties; *out_worker =
 * -1 when no worker runs the level. */
dn_status argus_select_worker(const int32_t* queue_len, const double* t_proc, const int32_t* worker_level,
                              int32_t n_workers, int32_t level, int32_t* out_worker);

const char* argus_last_error(void); /* message of the calling thread's last control-plane error */

void dn_destroy(dn_handle* h); /* NULL-safe; synchronizes the device first */

const char* dn_last_error(void); /* message of the calling thread's last error, "" if none */

#ifdef __cplusplus
}
#endif

#endif /* ARGUS_DN_H */
