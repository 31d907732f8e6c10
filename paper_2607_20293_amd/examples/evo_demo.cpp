// The cached denoising loop driven through the C ABI alone (include/evo.h and
// the HIP runtime; no Python, no torch): a Push-T-shaped policy with
// synthetic weights, one layer lattice refreshing every fourth step, a
// batch of queries on a stream of its own, the bookkeeping checked against
// the host-only count, and the call timed with HIP events.
//
//   evo_demo [batch] [calls]
//
// Prints one JSON line; exits non-zero on any error.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "evo.h"

#define CHECK_EVO(x)                                                                  \
  do {                                                                                \
    int rc_ = (x);                                                                    \
    if (rc_ != EVO_OK) {                                                              \
      std::fprintf(stderr, "%s -> %d: %s\n", #x, rc_, evo_last_error());              \
      return 1;                                                                       \
    }                                                                                 \
  } while (0)
#define CHECK_HIP(x)                                                                  \
  do {                                                                                \
    hipError_t e_ = (x);                                                              \
    if (e_ != hipSuccess) {                                                           \
      std::fprintf(stderr, "%s -> %s\n", #x, hipGetErrorString(e_));                  \
      return 1;                                                                       \
    }                                                                                 \
  } while (0)

// uniform values in [-a, a) from a 64-bit linear congruential generator
struct Lcg {
  uint64_t s;
  float next(float a) {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    return a * (2.0f * (float)((s >> 40) & 0xFFFFFF) / 16777216.0f - 1.0f);
  }
};

int main(int argc, char** argv) {
  const int batch = argc > 1 ? std::atoi(argv[1]) : 4;
  const int calls = argc > 2 ? std::atoi(argv[2]) : 10;
  if (batch < 1 || calls < 1) return 2;

  evo_policy_desc d{};
  d.n_layers = 8; d.d_model = 256; d.n_heads = 4; d.d_ff = 1024; d.horizon = 16; d.action_dim = 2;
  d.n_obs_tokens = 2; d.obs_dim = 20; d.n_steps = 100;
  d.dtype = EVO_BF16; d.cold_policy = EVO_COLD_COMPUTE; d.clip_sample = 1;
  d.max_batch = batch; d.max_schedules = 1;
  CHECK_EVO(evo_check_desc(&d));
  const int64_t nw = evo_weight_count(&d);
  if (nw < 0) return 1;
  Lcg g{12345};
  std::vector<float> w((size_t)nw);
  for (auto& v : w) v = g.next(0.05f);

  evo_policy* p = nullptr;
  CHECK_EVO(evo_create_policy(&d, w.data(), w.size(), &p));
  std::vector<uint8_t> lat((size_t)d.n_layers * d.n_steps, 0);
  for (int l = 0; l < d.n_layers; ++l)
    for (int t = 0; t < d.n_steps; t += 4) lat[(size_t)l * d.n_steps + t] = 1;
  CHECK_EVO(evo_set_schedule(p, 0, lat.data(), d.n_layers, d.n_steps, EVO_GRAN_LAYER));

  const size_t n_obs = (size_t)batch * d.n_obs_tokens * d.obs_dim;
  const size_t n_noise = (size_t)d.n_steps * batch * d.horizon * d.action_dim;
  const size_t n_out = (size_t)batch * d.horizon * d.action_dim;
  std::vector<float> h_obs(n_obs), h_noise(n_noise), h_out(n_out);
  for (auto& v : h_obs) v = g.next(1.0f);
  for (auto& v : h_noise) v = g.next(1.7f);
  float *obs = nullptr, *noise = nullptr, *out = nullptr;
  CHECK_HIP(hipMalloc(&obs, n_obs * sizeof(float)));
  CHECK_HIP(hipMalloc(&noise, n_noise * sizeof(float)));
  CHECK_HIP(hipMalloc(&out, n_out * sizeof(float)));
  CHECK_HIP(hipMemcpy(obs, h_obs.data(), n_obs * sizeof(float), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(noise, h_noise.data(), n_noise * sizeof(float), hipMemcpyHostToDevice));
  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));  // default priority

  CHECK_EVO(evo_denoise(p, batch, obs, noise, nullptr, out, st));  // warm-up
  hipEvent_t e0, e1;
  CHECK_HIP(hipEventCreate(&e0));
  CHECK_HIP(hipEventCreate(&e1));
  CHECK_HIP(hipEventRecord(e0, st));
  for (int i = 0; i < calls; ++i) CHECK_EVO(evo_denoise(p, batch, obs, noise, nullptr, out, st));
  CHECK_HIP(hipEventRecord(e1, st));
  CHECK_EVO(evo_synchronize(p));
  float ms = 0.f;
  CHECK_HIP(hipEventElapsedTime(&ms, e0, e1));
  CHECK_HIP(hipMemcpy(h_out.data(), out, n_out * sizeof(float), hipMemcpyDeviceToHost));
  bool finite = true;
  for (float v : h_out) finite = finite && std::isfinite(v);

  evo_stats got{}, want{};
  CHECK_EVO(evo_get_stats(p, &got));
  std::vector<int32_t> ids((size_t)batch, 0);
  CHECK_EVO(evo_schedule_stats(&d, lat.data(), 1, d.n_layers, EVO_GRAN_LAYER, ids.data(), batch, &want));
  const bool stats_ok = got.refreshes_effective == want.refreshes_effective && got.flops_full == want.flops_full;

  std::printf("{\"batch\": %d, \"calls\": %d, \"ms_per_call\": %.4f, \"chunks_per_s\": %.1f, "
              "\"refreshes_effective\": %llu, \"stats_match_host\": %s, \"finite\": %s, \"first\": %.6f}\n",
              batch, calls, ms / calls, batch * calls / (ms * 1e-3), (unsigned long long)got.refreshes_effective,
              stats_ok ? "true" : "false", finite ? "true" : "false", h_out[0]);
  CHECK_HIP(hipEventDestroy(e0));
  CHECK_HIP(hipEventDestroy(e1));
  CHECK_HIP(hipStreamDestroy(st));
  CHECK_HIP(hipFree(obs));
  CHECK_HIP(hipFree(noise));
  CHECK_HIP(hipFree(out));
  evo_destroy_policy(p);
  return (finite && stats_ok) ? 0 : 1;
}
