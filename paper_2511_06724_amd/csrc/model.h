// Host-side model: configuration checks, canonical weight table, packed
// device weights, workspace and the UNet / denoise-loop executor.
#pragma once

#include <map>
#include <memory>
#include <string>
#include <vector>

#include "argus_dn.h"
#include "kernels.h"

namespace dn {

constexpr int kMaxSteps = 1000;  // most iterations one dn_denoise call may run
constexpr int kCinPad = 64;      // conv input channels are padded to a multiple of this

struct TensorSpec {
  std::string name;
  std::vector<int64_t> shape;
  int64_t numel = 0;
  int64_t offset = 0;  // in floats, within the canonical blob
  int fan_in = 0;
  int kind = 0;  // 0 weight, 1 bias, 2 norm scale, 3 norm shift
};

// Validates cfg (throws Error(-1) with a message) and returns the canonical table.
void validate_config(const dn_config& cfg);
std::vector<TensorSpec> weight_table(const dn_config& cfg);

struct Model;
Model* model_create(const dn_config& cfg, const float* weights, size_t n_floats, bool on_device);
void model_destroy(Model* m);
void model_denoise(Model* m, float* latent, const float* ctx, const int32_t* ts, int n_ts, int start, int n,
                   float scale, hipStream_t s, const int32_t* cap_at = nullptr, int n_cap = 0,
                   uint16_t* cap_out = nullptr);
void model_unet_eps(Model* m, const float* x, int t, const float* ctx, float scale, float* raw, float* guided,
                    hipStream_t s);

// Latent decoder (vae.hip).
struct Vae;
std::vector<TensorSpec> vae_weight_table(const dn_vae_config& cfg);
Vae* vae_create(const dn_vae_config& cfg, const float* weights, size_t n_floats, bool on_device);
void vae_decode(Vae* v, const float* latent, float* image, hipStream_t s);
void vae_destroy(Vae* v);

}  // namespace dn
