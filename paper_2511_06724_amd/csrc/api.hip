// C ABI of the denoise-loop library: argument checks, error mapping and the
// single-kernel entry points. Every entry point catches all C++ exceptions.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "model.h"

// Scratch of the no-allocation batched lookup: the per-workgroup winners of one pass
// (at most lookup_batch_workspace_bytes(), 256 KiB, which also covers the per-query
// scan's lookup_workspace_bytes()), then 64 floats that receive the cosines when the
// caller asks for none. Every GPU the library runs on holds its own copy until the
// process ends; its device address comes from hipGetSymbolAddress, once per device.
constexpr size_t kScratchWinnerBytes = 256 * 1024;
constexpr size_t kScratchBytes = kScratchWinnerBytes + 64 * sizeof(float);
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace dn {
// probe.hip: the bf16 matrix-core rate (TFLOP/s) every CU sustains on back-to-back
// 32x32x16 MFMAs and the shader clock (GHz) meanwhile. Synchronous.
void mfma_rate(int iters, double* tflops, double* clock_ghz);
}  // namespace dn

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device (looked up on the first call on
// that device, with the device current; later calls reuse it).
void* scratch_ptr() {
  int dev = 0;
  DN_HIP(hipGetDevice(&dev));
  DN_CHECK(dev >= 0 && dev < kMaxDevices, "scratch: device ordinal beyond 64");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    DN_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    DN_CHECK(p != nullptr, "scratch: no device address");
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

thread_local std::string g_last_error;

dn_status fail(int code, const std::string& msg) {
  g_last_error = msg;
  return static_cast<dn_status>(code);
}

template <typename F> dn_status guarded(F&& f) {
  try {
    g_last_error.clear();
    f();
    return DN_OK;
  } catch (const dn::Error& e) {
    return fail(e.code, e.what());
  } catch (const std::bad_alloc&) {
    return fail(DN_ENOMEM, "host allocation failed");
  } catch (const std::exception& e) {
    return fail(DN_EHIP, e.what());
  } catch (...) {
    return fail(DN_EHIP, "unknown error");
  }
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// Per-device state of the cache lookup, allocated once: the device workspace of the
// per-workgroup winners, and a pinned host buffer the reduction writes the result to
// (index at byte 0, score at byte 8), so no copy follows the kernels.
struct LookupRes {
  long long idx;
  float score;
  int k;
};
struct LookupWs {
  std::mutex mu;
  std::vector<void*> ws;
  std::vector<LookupRes*> res;
  std::vector<void*> batch_ws;        // per-workgroup winners of the batched scan
  std::vector<long long*> batch_res;  // pinned: 64 indices, then 64 scores, then 64 levels
};
LookupWs g_lookup;

void lookup_state(int dev, void** ws, LookupRes** res) {
  std::lock_guard<std::mutex> lk(g_lookup.mu);
  if ((int)g_lookup.ws.size() <= dev) {
    g_lookup.ws.resize(dev + 1, nullptr);
    g_lookup.res.resize(dev + 1, nullptr);
  }
  if (!g_lookup.ws[dev]) DN_HIP(hipMalloc(&g_lookup.ws[dev], dn::lookup_workspace_bytes()));
  if (!g_lookup.res[dev]) DN_HIP(hipHostMalloc(reinterpret_cast<void**>(&g_lookup.res[dev]), 256));
  *ws = g_lookup.ws[dev];
  *res = g_lookup.res[dev];
}

void lookup_batch_state(int dev, void** ws, long long** idx, float** score, int** lev) {
  std::lock_guard<std::mutex> lk(g_lookup.mu);
  if ((int)g_lookup.batch_ws.size() <= dev) {
    g_lookup.batch_ws.resize(dev + 1, nullptr);
    g_lookup.batch_res.resize(dev + 1, nullptr);
  }
  const int mq = dn::lookup_batch_max_queries();
  if (!g_lookup.batch_ws[dev]) DN_HIP(hipMalloc(&g_lookup.batch_ws[dev], dn::lookup_batch_workspace_bytes()));
  if (!g_lookup.batch_res[dev])
    DN_HIP(hipHostMalloc(reinterpret_cast<void**>(&g_lookup.batch_res[dev]),
                         mq * (sizeof(long long) + sizeof(float) + sizeof(int))));
  *ws = g_lookup.batch_ws[dev];
  *idx = g_lookup.batch_res[dev];
  *score = reinterpret_cast<float*>(g_lookup.batch_res[dev] + mq);
  *lev = reinterpret_cast<int*>(*score + mq);
}

// Checks a similarity-to-level table and converts it for the kernels.
dn::KTable k_table(const ac_k_table* t) {
  DN_CHECK(t, "ac_k_table: null table");
  DN_CHECK(t->n_thresholds >= 0 && t->n_thresholds < AC_MAX_K_LEVELS,
           "ac_k_table: n_thresholds must be in [0, " + std::to_string(AC_MAX_K_LEVELS - 1) + "]");
  dn::KTable k;
  k.n = t->n_thresholds;
  for (int i = 0; i < k.n; ++i) {
    DN_CHECK(std::isfinite(t->threshold[i]), "ac_k_table: thresholds must be finite");
    DN_CHECK(i == 0 || t->threshold[i] > t->threshold[i - 1], "ac_k_table: thresholds must increase strictly");
    k.thr[i] = t->threshold[i];
  }
  for (int j = 0; j <= k.n; ++j) {
    DN_CHECK(t->level[j] >= 0, "ac_k_table: levels must be >= 0");
    DN_CHECK(j == 0 || t->level[j] >= t->level[j - 1], "ac_k_table: levels must not decrease");
    k.level[j] = t->level[j];
  }
  return k;
}

// The batched search of ac_lookup_batch / ac_lookup_batch_k (host results; level per
// query when kt is given).
void lookup_batch_host(const uint16_t* query_embs, int32_t nq, const uint16_t* cache_embs, int64_t n, int32_t dim,
                       int64_t* out_idx, float* out_score, const dn::KTable* kt, int32_t* out_k, const char* who) {
  const std::string w(who);
  DN_CHECK(query_embs && cache_embs && out_idx, w + ": null pointer");
  DN_CHECK(nq >= 1, w + ": nq must be >= 1");
  DN_CHECK(n >= 1, w + ": n must be >= 1");
  DN_CHECK(dim >= 1, w + ": dim must be >= 1");
  DN_CHECK(!kt || out_k, w + ": null level output");
  int dev = 0;
  DN_HIP(hipGetDevice(&dev));
  if (!dn::lookup_batch_supported(query_embs, cache_embs, n, dim)) {
    // other widths or alignments: one scan per query
    void* ws = nullptr;
    LookupRes* res = nullptr;
    lookup_state(dev, &ws, &res);
    for (int j = 0; j < nq; ++j) {
      res->idx = -1;
      res->score = 0.f;
      res->k = -1;
      dn::lookup(query_embs + (size_t)j * dim, cache_embs, n, dim, ws, &res->idx, &res->score, nullptr, kt,
                 &res->k);
      DN_HIP(hipStreamSynchronize(nullptr));
      out_idx[j] = *static_cast<volatile long long*>(&res->idx);
      if (out_score) out_score[j] = *static_cast<volatile float*>(&res->score);
      if (kt) out_k[j] = *static_cast<volatile int*>(&res->k);
    }
    return;
  }
  void* ws = nullptr;
  long long* ridx = nullptr;
  float* rscore = nullptr;
  int* rk = nullptr;
  lookup_batch_state(dev, &ws, &ridx, &rscore, &rk);
  const int mq = dn::lookup_batch_max_queries();
  for (int j0 = 0; j0 < nq; j0 += mq) {
    const int m = nq - j0 < mq ? nq - j0 : mq;
    for (int j = 0; j < m; ++j) ridx[j] = -2;
    dn::lookup_batch(query_embs + (size_t)j0 * dim, m, cache_embs, n, dim, ws, ridx, rscore, nullptr, kt, rk);
    DN_HIP(hipStreamSynchronize(nullptr));
    for (int j = 0; j < m; ++j) {
      const long long idx = static_cast<volatile long long*>(ridx)[j];
      DN_CHECK(idx >= -1 && idx < n, w + ": result not written");
      out_idx[j0 + j] = idx;
      if (out_score) out_score[j0 + j] = static_cast<volatile float*>(rscore)[j];
      if (kt) out_k[j0 + j] = static_cast<volatile int*>(rk)[j];
    }
  }
}

bool is_dtype(int32_t d) { return d == DN_FP32 || d == DN_BF16; }
bool is_dtype8(int32_t d) { return is_dtype(d) || d == DN_FP8; }

// Per-device state of the single-kernel GEMM entry points: CU count (tile
// planning) and a zero block for implicit-conv padding reads.
struct OpDev {
  int cus = 0;
  void* zero = nullptr;
  float* part = nullptr;  // split-K partial slabs, grown on demand
  size_t part_floats = 0;
  float* gn = nullptr;    // GroupNorm partial sums and per-channel scale / shift, grown on demand
  size_t gn_floats = 0;
};
std::mutex g_op_mu;
std::vector<OpDev> g_op_dev;

// Grows a per-device buffer of the single-kernel entry points. Work already enqueued
// may still read the old buffer, so the device is synchronised before it is freed.
void grow(float** buf, size_t* have, size_t need) {
  if (need <= *have) return;
  if (*buf) {
    DN_HIP(hipDeviceSynchronize());
    DN_HIP(hipFree(*buf));
    *buf = nullptr;
    *have = 0;
  }
  DN_HIP(hipMalloc(reinterpret_cast<void**>(buf), need * 4));
  *have = need;
}

OpDev& op_dev_locked(int dev) {
  if ((int)g_op_dev.size() <= dev) g_op_dev.resize(dev + 1);
  OpDev& d = g_op_dev[dev];
  if (!d.cus) {
    hipDeviceProp_t prop;
    DN_HIP(hipGetDeviceProperties(&prop, dev));
    DN_HIP(hipMalloc(&d.zero, 256));
    DN_HIP(hipMemset(d.zero, 0, 256));
    d.cus = prop.multiProcessorCount;
  }
  return d;
}

template <typename T> dn::GemmPlan op_plan(const dn::GemmParams& p, int cus) {
  return p.wscale ? dn::gemm_plan_fp8(p.M, p.N, p.K, p.geglu, cus, true, false)
                  : dn::gemm_plan<T>(p.M, p.N, p.K, p.geglu, cus, p.vt == nullptr, false, p.taps == 9);
}

template <typename T> void op_gemm(dn::GemmParams& p, hipStream_t s) {
  int dev = 0;
  DN_HIP(hipGetDevice(&dev));
  OpDev w;
  {
    std::lock_guard<std::mutex> lk(g_op_mu);
    OpDev& d = op_dev_locked(dev);
    const dn::GemmPlan g0 = op_plan<T>(p, d.cus);
    grow(&d.part, &d.part_floats, dn::gemm_workspace_floats(g0, p.M, p.N));
    w = d;
  }
  const dn::GemmPlan g = op_plan<T>(p, w.cus);
  p.zero16 = w.zero;
  p.part = w.part;
  p.part_floats = w.part_floats;
  if (p.wscale)
    dn::gemm_fp8(p, g, s);
  else
    dn::gemm<T>(p, g, s);
}

}  // namespace

struct dn_handle {
  dn::Model* m = nullptr;
};
struct dn_vae {
  dn::Vae* v = nullptr;
};

extern "C" {

dn_status dn_weight_count(const dn_config* cfg, size_t* n_floats) {
  return guarded([&] {
    DN_CHECK(cfg && n_floats, "dn_weight_count: null pointer");
    const auto t = dn::weight_table(*cfg);
    *n_floats = t.empty() ? 0 : static_cast<size_t>(t.back().offset + t.back().numel);
  });
}

dn_status dn_weight_table(const dn_config* cfg, int64_t* numel, int32_t* fan_in, int32_t* kind, size_t capacity,
                          size_t* n_tensors) {
  return guarded([&] {
    DN_CHECK(cfg && n_tensors, "dn_weight_table: null pointer");
    const auto t = dn::weight_table(*cfg);
    DN_CHECK(capacity == 0 || capacity >= t.size(), "dn_weight_table: capacity too small");
    DN_CHECK(capacity == 0 || (numel && fan_in && kind), "dn_weight_table: null output array");
    if (capacity) {
      for (size_t i = 0; i < t.size(); ++i) {
        numel[i] = t[i].numel;
        fan_in[i] = t[i].fan_in;
        kind[i] = t[i].kind;
      }
    }
    *n_tensors = t.size();
  });
}

dn_status dn_create(const dn_config* cfg, const float* weights, size_t n_floats, int32_t weights_location,
                    dn_handle** out) {
  return guarded([&] {
    DN_CHECK(cfg && weights && out, "dn_create: null pointer");
    DN_CHECK(weights_location == DN_WEIGHTS_HOST || weights_location == DN_WEIGHTS_DEVICE,
             "dn_create: bad weights_location");
    dn::Model* m = dn::model_create(*cfg, weights, n_floats, weights_location == DN_WEIGHTS_DEVICE);
    dn_handle* h = new dn_handle();
    h->m = m;
    *out = h;
  });
}

dn_status dn_denoise(dn_handle* h, float* latent, const float* text_ctx, const int32_t* timesteps,
                     int32_t n_timesteps, int32_t start_step, int32_t n_steps, float cfg_scale, void* stream) {
  return guarded([&] {
    DN_CHECK(h && h->m, "dn_denoise: null handle");
    dn::model_denoise(h->m, latent, text_ctx, timesteps, n_timesteps, start_step, n_steps, cfg_scale,
                      as_stream(stream));
  });
}

dn_status dn_denoise_capture(dn_handle* h, float* latent, const float* text_ctx, const int32_t* timesteps,
                             int32_t n_timesteps, int32_t start_step, int32_t n_steps, float cfg_scale,
                             const int32_t* capture_at, int32_t n_capture, uint16_t* out_latents, void* stream) {
  return guarded([&] {
    DN_CHECK(h && h->m, "dn_denoise_capture: null handle");
    dn::model_denoise(h->m, latent, text_ctx, timesteps, n_timesteps, start_step, n_steps, cfg_scale,
                      as_stream(stream), capture_at, n_capture, out_latents);
  });
}

dn_status dn_unet_eps(dn_handle* h, const float* x, int32_t t, const float* text_ctx, float cfg_scale, float* out_raw,
                      float* out_guided, void* stream) {
  return guarded([&] {
    DN_CHECK(h && h->m, "dn_unet_eps: null handle");
    dn::model_unet_eps(h->m, x, t, text_ctx, cfg_scale, out_raw, out_guided, as_stream(stream));
  });
}

dn_status ac_lookup(const uint16_t* query_emb, const uint16_t* cache_embs, int64_t n, int32_t dim, int64_t* out_idx,
                    float* out_score) {
  return guarded([&] {
    DN_CHECK(query_emb && cache_embs && out_idx, "ac_lookup: null pointer");
    DN_CHECK(n >= 1, "ac_lookup: n must be >= 1");
    DN_CHECK(dim >= 1, "ac_lookup: dim must be >= 1");
    int dev = 0;
    DN_HIP(hipGetDevice(&dev));
    void* ws = nullptr;
    LookupRes* res = nullptr;
    lookup_state(dev, &ws, &res);
    res->idx = -1;
    res->score = 0.f;
    dn::lookup(query_emb, cache_embs, n, dim, ws, &res->idx, &res->score, nullptr);
    DN_HIP(hipStreamSynchronize(nullptr));
    // written by the device: read through volatile so the values set above are not reused
    const long long idx = *static_cast<volatile long long*>(&res->idx);
    const float score = *static_cast<volatile float*>(&res->score);
    DN_CHECK(idx >= 0 && idx < n, "ac_lookup: no row scored (zero query or zero-norm cache)");
    *out_idx = idx;
    if (out_score) *out_score = score;
  });
}

dn_status ac_lookup_batch(const uint16_t* query_embs, int32_t nq, const uint16_t* cache_embs, int64_t n, int32_t dim,
                          int64_t* out_idx, float* out_score) {
  return guarded([&] {
    lookup_batch_host(query_embs, nq, cache_embs, n, dim, out_idx, out_score, nullptr, nullptr, "ac_lookup_batch");
  });
}

dn_status ac_lookup_batch_k(const uint16_t* query_embs, int32_t nq, const uint16_t* cache_embs, int64_t n,
                            int32_t dim, const ac_k_table* table, int64_t* out_idx, float* out_score,
                            int32_t* out_k) {
  return guarded([&] {
    const dn::KTable kt = k_table(table);
    lookup_batch_host(query_embs, nq, cache_embs, n, dim, out_idx, out_score, &kt, out_k, "ac_lookup_batch_k");
  });
}

dn_status ac_lookup_batch_noalloc(const uint16_t* query_embs, int32_t nq, const uint16_t* cache_embs, int64_t n,
                                  int32_t dim, int64_t* out_idx, float* out_score, void* stream) {
  return guarded([&] {
    DN_CHECK(query_embs && cache_embs && out_idx, "ac_lookup_batch_noalloc: null pointer");
    DN_CHECK(nq >= 1, "ac_lookup_batch_noalloc: nq must be >= 1");
    DN_CHECK(n >= 1, "ac_lookup_batch_noalloc: n must be >= 1");
    DN_CHECK(dim >= 1, "ac_lookup_batch_noalloc: dim must be >= 1");
    const bool batched = dn::lookup_batch_supported(query_embs, cache_embs, n, dim);
    const size_t need = batched ? dn::lookup_batch_workspace_bytes() : dn::lookup_workspace_bytes();
    DN_CHECK(need <= kScratchWinnerBytes, "ac_lookup_batch_noalloc: scan needs " + std::to_string(need) +
                                              " bytes of scratch, the library holds " +
                                              std::to_string(kScratchWinnerBytes));
    DN_CHECK(batched || dim <= 16384, "ac_lookup_batch_noalloc: dim too large for the per-query scan");
    char* ws = static_cast<char*>(scratch_ptr());
    float* dummy = reinterpret_cast<float*>(ws + kScratchWinnerBytes);
    const hipStream_t s = as_stream(stream);
    long long* idx = reinterpret_cast<long long*>(out_idx);
    if (batched) {
      const int mq = dn::lookup_batch_max_queries();
      for (int j0 = 0; j0 < nq; j0 += mq) {
        const int m = nq - j0 < mq ? nq - j0 : mq;
        dn::lookup_batch(query_embs + (size_t)j0 * dim, m, cache_embs, n, dim, ws, idx + j0,
                         out_score ? out_score + j0 : dummy, s);
      }
    } else {
      for (int j = 0; j < nq; ++j)
        dn::lookup(query_embs + (size_t)j * dim, cache_embs, n, dim, ws, idx + j, out_score ? out_score + j : dummy,
                   s);
    }
  });
}

dn_status ac_fetch_latent(const uint16_t* cache_latents, int64_t n, int64_t numel, int64_t idx, float* latent,
                          void* stream) {
  return guarded([&] {
    DN_CHECK(cache_latents && latent, "ac_fetch_latent: null pointer");
    DN_CHECK(n >= 1 && numel >= 1, "ac_fetch_latent: empty cache");
    DN_CHECK(idx >= 0 && idx < n, "ac_fetch_latent: index out of range");
    dn::bf16_latent_to_f32(cache_latents + idx * numel, latent, numel, as_stream(stream));
  });
}

dn_status dn_packed_weight_elems(int32_t dtype, int32_t N, int32_t K, int64_t* elems) {
  return guarded([&] {
    DN_CHECK(is_dtype8(dtype), "dn_packed_weight_elems: bad dtype");
    DN_CHECK(elems, "dn_packed_weight_elems: null pointer");
    DN_CHECK(N >= 1 && K >= 1, "dn_packed_weight_elems: bad sizes");
    if (dtype == DN_FP8) {
      DN_CHECK(dn::gemm_fp8_layout(N, K), "dn_packed_weight_elems: DN_FP8 needs N % 32 == 0, K % 128 == 0");
      *elems = (int64_t)dn::gemm_fp8_code_bytes(N, K) + 4ll * N;
      return;
    }
    *elems = dtype == DN_BF16 && dn::gemm_frag_layout(N, K) ? (int64_t)dn::gemm_frag_elems(N, K) : (int64_t)N * K;
  });
}

dn_status dn_pack_weight(int32_t dtype, const void* w, int32_t N, int32_t K, void* out, void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype8(dtype), "dn_pack_weight: bad dtype");
    DN_CHECK(w && out, "dn_pack_weight: null pointer");
    if (dtype == DN_FP8) {
      DN_CHECK(dn::gemm_fp8_layout(N, K), "dn_pack_weight: DN_FP8 needs N % 32 == 0, K % 128 == 0");
      dn::PackParams p;
      p.dst = out;
      p.rows = N;
      p.cols = K;
      p.ld_dst = K;
      p.src = static_cast<const float*>(w);
      p.src_rows = N;
      p.src_cols = K;
      dn::pack_fp8(p, reinterpret_cast<float*>(static_cast<char*>(out) + dn::gemm_fp8_code_bytes(N, K)),
                   as_stream(stream));
      return;
    }
    DN_CHECK(N >= 1 && K >= 1 && K % 16 == 0, "dn_pack_weight: bad sizes (K must be a multiple of 16)");
    if (dtype == DN_BF16 && dn::gemm_frag_layout(N, K)) {
      dn::to_frag(static_cast<const dn::bf16*>(w), N, K, K, static_cast<dn::bf16*>(out), as_stream(stream));
    } else {
      const size_t bytes = (size_t)N * K * (dtype == DN_BF16 ? 2 : 4);
      DN_HIP(hipMemcpyAsync(out, w, bytes, hipMemcpyDeviceToDevice, as_stream(stream)));
    }
  });
}

dn_status dn_op_linear(int32_t dtype, const void* x, const void* w, const float* bias, const void* resid,
                       int32_t resid_f32, void* y, int32_t y_f32, int64_t M, int32_t N, int32_t K, int32_t geglu,
                       void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype8(dtype), "dn_op_linear: bad dtype");
    DN_CHECK(x && w && y, "dn_op_linear: null pointer");
    DN_CHECK(M >= 1 && M <= 0x7fffffff && N >= 1 && K >= 1, "dn_op_linear: bad sizes");
    DN_CHECK(!geglu || N % 32 == 0, "dn_op_linear: GEGLU needs N % 32 == 0");
    DN_CHECK(!(geglu && resid), "dn_op_linear: GEGLU takes no residual");
    dn::GemmParams p;
    p.a0 = x;
    p.c0 = K;
    p.lda0 = K;
    p.taps = 1;
    p.b = w;
    p.ldb = K;
    p.M = static_cast<int>(M);
    p.N = geglu ? 2 * N : N;
    p.K = K;
    p.bias = bias;
    p.resid = resid;
    p.ldr = N;
    p.resid_f32 = resid_f32;
    p.out = y;
    p.ldo = N;
    p.out_f32 = y_f32;
    p.n_store = N;
    p.geglu = geglu;
    if (dtype == DN_FP8) {
      const int Nw = geglu ? 2 * N : N;
      DN_CHECK(dn::gemm_fp8_layout(Nw, K), "dn_op_linear: DN_FP8 needs N % 32 == 0 and K % 128 == 0");
      p.wscale = reinterpret_cast<const float*>(static_cast<const char*>(w) + dn::gemm_fp8_code_bytes(Nw, K));
      p.out_fp8 = !y_f32 && geglu;
      op_gemm<dn::bf16>(p, as_stream(stream));
    } else if (dtype == DN_BF16) {
      op_gemm<dn::bf16>(p, as_stream(stream));
    } else {
      op_gemm<float>(p, as_stream(stream));
    }
  });
}

dn_status dn_op_conv3x3(int32_t dtype, const void* x, int32_t n, int32_t H, int32_t W, int32_t Cin, int32_t up,
                        int32_t stride, const void* w, const float* bias, const float* temb, const void* resid,
                        void* y, int32_t Cout, int32_t y_f32, void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype(dtype), "dn_op_conv3x3: bad dtype");
    DN_CHECK(x && w && y, "dn_op_conv3x3: null pointer");
    DN_CHECK(n >= 1 && H >= 1 && W >= 1 && Cin >= 1 && Cout >= 1, "dn_op_conv3x3: bad sizes");
    DN_CHECK(up == 0 || up == 1, "dn_op_conv3x3: up must be 0 or 1");
    DN_CHECK(stride == 1 || stride == 2, "dn_op_conv3x3: stride must be 1 or 2");
    const int hl = up ? 2 * H : H, wl = up ? 2 * W : W;
    const int ho = (hl - 1) / stride + 1, wo = (wl - 1) / stride + 1;
    dn::GemmParams p;
    p.a0 = x;
    p.c0 = Cin;
    p.lda0 = Cin;
    p.taps = 9;
    p.in_h = H;
    p.in_w = W;
    p.up = up;
    p.out_h = ho;
    p.out_w = wo;
    p.stride = stride;
    p.b = w;
    p.ldb = 9 * Cin;
    p.M = n * ho * wo;
    p.N = Cout;
    p.K = 9 * Cin;
    p.bias = bias;
    p.rowvec = temb;
    p.rowvec_ld = Cout;
    p.rows_per_sample = ho * wo;
    p.resid = resid;
    p.ldr = Cout;
    p.out = y;
    p.ldo = Cout;
    p.out_f32 = y_f32;
    p.n_store = Cout;
    if (dtype == DN_BF16)
      op_gemm<dn::bf16>(p, as_stream(stream));
    else
      op_gemm<float>(p, as_stream(stream));
  });
}

dn_status dn_op_attention(int32_t dtype, const void* q, int32_t ldq, const void* k, int32_t ldk, const void* vt,
                          int32_t vt_ld, void* o, int32_t ldo, int32_t B, int32_t heads, int32_t Sq, int32_t Skv,
                          int32_t head_stride, float scale, void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype(dtype), "dn_op_attention: bad dtype");
    DN_CHECK(q && k && vt && o, "dn_op_attention: null pointer");
    DN_CHECK(head_stride == 32 || head_stride == 64, "dn_op_attention: head_stride must be 32 or 64");
    DN_CHECK(B >= 1 && heads >= 1 && Sq >= 1 && Skv >= 1, "dn_op_attention: bad sizes");
    DN_CHECK(ldq >= heads * head_stride && ldk >= heads * head_stride && ldo >= heads * head_stride,
             "dn_op_attention: leading dimension smaller than heads * head_stride");
    DN_CHECK(vt_ld >= (Skv + 63) / 64 * 64, "dn_op_attention: vt_ld must cover Skv rounded up to 64");
    dn::AttnParams a;
    a.q = q;
    a.k = k;
    a.vt = vt;
    a.o = o;
    a.ldq = ldq;
    a.ldk = ldk;
    a.vt_ld = vt_ld;
    a.ldo = ldo;
    a.q_bs = (long long)Sq * ldq;
    a.k_bs = (long long)Skv * ldk;
    a.o_bs = (long long)Sq * ldo;
    a.B = B;
    a.heads = heads;
    a.Sq = Sq;
    a.Skv = Skv;
    a.scale_log2 = scale * 1.4426950408889634f;
    if (dtype == DN_BF16)
      dn::attention<dn::bf16>(a, head_stride, as_stream(stream));
    else
      dn::attention<float>(a, head_stride, as_stream(stream));
  });
}

dn_status dn_op_linear_vt(int32_t dtype, const void* x, const void* w, const float* bias, void* y, int64_t M,
                          int32_t N, int32_t K, int32_t vt_col0, void* vt, int32_t heads, int32_t head_stride,
                          int32_t seq, int32_t vt_ld, void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype(dtype), "dn_op_linear_vt: bad dtype");
    DN_CHECK(x && w && y && vt, "dn_op_linear_vt: null pointer");
    DN_CHECK(M >= 1 && M <= 0x7fffffff && N >= 1 && K >= 1, "dn_op_linear_vt: bad sizes");
    DN_CHECK(vt_col0 >= 4 && vt_col0 % 4 == 0 && vt_col0 < N, "dn_op_linear_vt: vt_col0 must be in [4, N), % 4 == 0");
    DN_CHECK(head_stride >= 4 && head_stride % 4 == 0 && heads >= 1 && (N - vt_col0) == heads * head_stride,
             "dn_op_linear_vt: N - vt_col0 must equal heads * head_stride (a multiple of 4)");
    DN_CHECK(seq >= 1 && M % seq == 0 && vt_ld >= seq, "dn_op_linear_vt: rows must be whole sequences, vt_ld >= seq");
    dn::GemmParams p;
    p.a0 = x;
    p.c0 = K;
    p.lda0 = K;
    p.taps = 1;
    p.b = w;
    p.ldb = K;
    p.M = static_cast<int>(M);
    p.N = N;
    p.K = K;
    p.bias = bias;
    p.out = y;
    p.ldo = vt_col0;
    p.n_store = N;
    p.vt = vt;
    p.vt_col0 = vt_col0;
    p.vt_dp = head_stride;
    p.vt_heads = heads;
    p.vt_seq = seq;
    p.vt_ld = vt_ld;
    if (dtype == DN_BF16)
      op_gemm<dn::bf16>(p, as_stream(stream));
    else
      op_gemm<float>(p, as_stream(stream));
  });
}

dn_status dn_op_groupnorm(int32_t dtype, const void* x, void* y, int32_t n, int32_t HW, int32_t C, int32_t G,
                          const float* gamma, const float* beta, float eps, int32_t silu, void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype(dtype), "dn_op_groupnorm: bad dtype");
    DN_CHECK(x && y && gamma && beta, "dn_op_groupnorm: null pointer");
    DN_CHECK(n >= 1 && HW >= 1 && C >= 1 && G >= 1 && C % G == 0, "dn_op_groupnorm: bad sizes");
    int dev = 0;
    DN_HIP(hipGetDevice(&dev));
    const size_t part = dn::groupnorm_workspace_floats(n, HW, C, G);
    float* ws = nullptr;
    {
      std::lock_guard<std::mutex> lk(g_op_mu);
      OpDev& d = op_dev_locked(dev);
      grow(&d.gn, &d.gn_floats, part + (size_t)2 * n * C);
      ws = d.gn;
    }
    dn::GroupNormParams p;
    p.x0 = x;
    p.c0 = C;
    p.n = n;
    p.HW = HW;
    p.G = G;
    p.gamma = gamma;
    p.beta = beta;
    p.eps = eps;
    p.silu = silu;
    p.y = y;
    p.partial = ws;
    p.stats = ws + part;
    if (dtype == DN_BF16)
      dn::groupnorm<dn::bf16>(p, as_stream(stream));
    else
      dn::groupnorm<float>(p, as_stream(stream));
  });
}

dn_status dn_op_layernorm(int32_t dtype, const float* x, void* y, int64_t M, int32_t C, const float* gamma,
                          const float* beta, float eps, void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype8(dtype), "dn_op_layernorm: bad dtype");
    DN_CHECK(x && y && gamma && beta, "dn_op_layernorm: null pointer");
    if (dtype == DN_FP8)
      dn::layernorm<uint8_t>(x, static_cast<uint8_t*>(y), M, C, gamma, beta, eps, as_stream(stream));
    else if (dtype == DN_BF16)
      dn::layernorm<dn::bf16>(x, static_cast<dn::bf16*>(y), M, C, gamma, beta, eps, as_stream(stream));
    else
      dn::layernorm<float>(x, static_cast<float*>(y), M, C, gamma, beta, eps, as_stream(stream));
  });
}

dn_status dn_op_layernorm_slabs(int32_t dtype, float* x, void* y, int64_t M, int32_t C, const float* gamma,
                                const float* beta, float eps, const float* slabs, int32_t nsplit, const float* bias,
                                int32_t resid, void* stream) {
  return guarded([&] {
    DN_CHECK(is_dtype(dtype), "dn_op_layernorm_slabs: bad dtype");
    DN_CHECK(x && y && gamma && beta && slabs, "dn_op_layernorm_slabs: null pointer");
    DN_CHECK(nsplit >= 1 && nsplit <= 8, "dn_op_layernorm_slabs: nsplit must be in [1, 8]");
    DN_CHECK(resid == 0 || resid == 1, "dn_op_layernorm_slabs: resid must be 0 or 1");
    if (dtype == DN_BF16)
      dn::layernorm_reduce<dn::bf16>(x, static_cast<dn::bf16*>(y), M, C, gamma, beta, eps, slabs, nsplit, bias,
                                     resid != 0, as_stream(stream));
    else
      dn::layernorm_reduce<float>(x, static_cast<float*>(y), M, C, gamma, beta, eps, slabs, nsplit, bias,
                                  resid != 0, as_stream(stream));
  });
}

dn_status dn_probe_mfma_rate(int32_t iters, double* tflops, double* clock_ghz) {
  return guarded([&] {
    DN_CHECK(tflops && clock_ghz, "dn_probe_mfma_rate: null pointer");
    DN_CHECK(iters >= 1 && iters <= (1 << 20), "dn_probe_mfma_rate: iters must be in [1, 2^20]");
    dn::mfma_rate(iters, tflops, clock_ghz);
  });
}

dn_status dn_vae_weight_count(const dn_vae_config* cfg, size_t* n_floats) {
  return guarded([&] {
    DN_CHECK(cfg && n_floats, "dn_vae_weight_count: null pointer");
    const auto t = dn::vae_weight_table(*cfg);
    *n_floats = static_cast<size_t>(t.back().offset + t.back().numel);
  });
}

dn_status dn_vae_weight_table(const dn_vae_config* cfg, int64_t* numel, int32_t* fan_in, int32_t* kind,
                              size_t capacity, size_t* n_tensors) {
  return guarded([&] {
    DN_CHECK(cfg && n_tensors, "dn_vae_weight_table: null pointer");
    const auto t = dn::vae_weight_table(*cfg);
    DN_CHECK(capacity == 0 || capacity >= t.size(), "dn_vae_weight_table: capacity too small");
    DN_CHECK(capacity == 0 || (numel && fan_in && kind), "dn_vae_weight_table: null output array");
    if (capacity)
      for (size_t i = 0; i < t.size(); ++i) {
        numel[i] = t[i].numel;
        fan_in[i] = t[i].fan_in;
        kind[i] = t[i].kind;
      }
    *n_tensors = t.size();
  });
}

dn_status dn_vae_create(const dn_vae_config* cfg, const float* weights, size_t n_floats, int32_t weights_location,
                        dn_vae** out) {
  return guarded([&] {
    DN_CHECK(cfg && weights && out, "dn_vae_create: null pointer");
    DN_CHECK(weights_location == DN_WEIGHTS_HOST || weights_location == DN_WEIGHTS_DEVICE,
             "dn_vae_create: bad weights_location");
    dn::Vae* v = dn::vae_create(*cfg, weights, n_floats, weights_location == DN_WEIGHTS_DEVICE);
    dn_vae* h = new dn_vae();
    h->v = v;
    *out = h;
  });
}

dn_status dn_vae_decode(dn_vae* h, const float* latent, float* image, void* stream) {
  return guarded([&] {
    DN_CHECK(h && h->v, "dn_vae_decode: null handle");
    dn::vae_decode(h->v, latent, image, as_stream(stream));
  });
}

void dn_vae_destroy(dn_vae* h) {
  if (!h) return;
  dn::vae_destroy(h->v);
  delete h;
}

void dn_destroy(dn_handle* h) {
  if (!h) return;
  dn::model_destroy(h->m);
  delete h;
}

const char* dn_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
