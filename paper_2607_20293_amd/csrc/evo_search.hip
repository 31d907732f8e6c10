// Schedule search with fitness on the GPU (Sec. 3.2, Eq. 4, Eq. 8, Eq. 9):
// a population's new schedules run as one batched evo_denoise call, one
// schedule id per candidate, each candidate on the same n_quick episodes;
// the deviation of every chunk from the uncached chunk of its episode is
// reduced on the device and only [batch] floats come back to the host,
// where the GA (evo_ga.cpp) ranks, selects and breeds.  Every call runs
// one workgroup per tile (no small-batch teams), whose results do not
// depend on the batch size, so a schedule's fitness does not depend on how
// many new schedules its generation has.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "evo_host.hpp"
#include "evo_kernels.hpp"

using namespace evo;

namespace {

// dst[o][i][k] = src[o][i % n_src][k], o < outer, i < n_dst, k < inner
__global__ void __launch_bounds__(256) replicate_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                                        int outer, int n_src, int n_dst, int inner) {
  const long long total = (long long)outer * n_dst * inner;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < total; e += (long long)gridDim.x * 256) {
    const long long k = e % inner;
    const long long r = e / inner;
    const long long i = r % n_dst, o = r / n_dst;
    dst[e] = src[(o * n_src + i % n_src) * inner + k];
  }
}

// dev[i] = max_k |out[i][k] - ref[i % n_ref][k]|, one wavefront per episode
__global__ void __launch_bounds__(64) deviation_kernel(const float* __restrict__ out, const float* __restrict__ ref,
                                                       float* __restrict__ dev, int batch, int n_ref, int inner) {
  const int i = blockIdx.x;
  if (i >= batch) return;
  const float* a = out + (size_t)i * inner;
  const float* b = ref + (size_t)(i % n_ref) * inner;
  float m = 0.0f;
  for (int k = threadIdx.x; k < inner; k += 64) m = fmaxf(m, fabsf(a[k] - b[k]));
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  if (threadIdx.x == 0) dev[i] = m;
}

hipError_t replicate(const float* src, float* dst, int outer, int n_src, int n_dst, int inner, hipStream_t s) {
  const long long total = (long long)outer * n_dst * inner;
  if (total <= 0) return hipSuccess;
  const long long blocks = std::min<long long>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(replicate_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, outer, n_src, n_dst, inner);
  return hipGetLastError();
}

struct Workspace {
  float* ref_q = nullptr;   // [n_quick][H][A] uncached chunks
  float* ref_f = nullptr;   // [n_formal][H][A]
  float* out = nullptr;     // [max(P*n_quick, n_formal)][H][A]
  float* obs = nullptr;     // [P*n_quick][n_obs][obs_dim]
  float* noise = nullptr;   // [T][P*n_quick][H][A]
  float* dev = nullptr;     // [max(P*n_quick, n_formal)]
  ~Workspace() {
    (void)hipFree(ref_q);
    (void)hipFree(ref_f);
    (void)hipFree(out);
    (void)hipFree(obs);
    (void)hipFree(noise);
    (void)hipFree(dev);
  }
};

}  // namespace

extern "C" int evo_search(evo_policy* p, const evo_ga_config* cfg, const evo_search_options* opt,
                          const float* obs_quick, const float* noise_quick, const float* obs_formal,
                          const float* noise_formal, const double* probs, evo_search_result* result,
                          int32_t* best_out, int32_t* pop_history, double* fit_history, void* hip_stream) {
  return guarded([&]() -> int {
    clear_error();
    if (!p || !opt || !result || !best_out) return fail(EVO_E_INVALID, "NULL pointer");
    const Shape& s = policy_shape(p);
    if (opt->granularity != EVO_GRAN_UNIT && opt->granularity != EVO_GRAN_LAYER)
      return fail(EVO_E_INVALID, "bad granularity");
    const int rows = opt->granularity == EVO_GRAN_UNIT ? s.U() : s.L;
    int rc = ga_check(cfg, rows, s.T, probs, true);
    if (rc) return rc;
    const int P = cfg->pop_size, K = cfg->K, nq = opt->n_quick, nf = opt->n_formal;
    if (nq < 1 || (long long)P * nq > s.max_batch)
      return fail(EVO_E_INVALID, "pop_size x n_quick = %lld outside [1, max_batch %d]", (long long)P * nq, s.max_batch);
    if (nf < 0 || nf > s.max_batch) return fail(EVO_E_INVALID, "n_formal %d outside [0, %d]", nf, s.max_batch);
    if (P > s.max_sched) return fail(EVO_E_INVALID, "pop_size %d > max_schedules %d", P, s.max_sched);
    if (!(opt->tau >= 0.0f)) return fail(EVO_E_INVALID, "tau must be >= 0");
    if (std::isnan(opt->q_base) || !(opt->delta_acc >= 0.0)) return fail(EVO_E_INVALID, "bad q_base / delta_acc");
    if (!obs_quick || !noise_quick) return fail(EVO_E_INVALID, "NULL quick episodes");
    if (nf > 0 && (!obs_formal || !noise_formal)) return fail(EVO_E_INVALID, "NULL formal episodes");

    DeviceGuard guard(policy_device(p));
    hipStream_t stream = (hipStream_t)hip_stream;
    const int HA = s.H * s.A, OB = s.n_obs * s.obs_dim, T = s.T;
    const int bq = P * nq, bmax = std::max(bq, nf);
    Workspace w;
#define WS_ALLOC(ptr, n)                                                                                  \
    do {                                                                                                    \
      if ((n) > 0 && hipMalloc(&(ptr), sizeof(float) * (size_t)(n)) != hipSuccess)                         \
        return fail(EVO_E_NOMEM, "search workspace allocation of %zu bytes failed", sizeof(float) * (size_t)(n)); \
    } while (0)
    WS_ALLOC(w.ref_q, (size_t)nq * HA);
    WS_ALLOC(w.ref_f, (size_t)nf * HA);
    WS_ALLOC(w.out, (size_t)bmax * HA);
    WS_ALLOC(w.obs, (size_t)bq * OB);
    WS_ALLOC(w.noise, (size_t)T * bq * HA);
    WS_ALLOC(w.dev, (size_t)bmax);
#undef WS_ALLOC

    // uncached chunks of the quick and formal episodes (schedule id 0, all refresh)
    std::vector<uint8_t> all((size_t)rows * T, 1);
    rc = evo_set_schedule(p, 0, all.data(), rows, T, opt->granularity);
    if (rc) return rc;
    std::vector<int32_t> ids((size_t)bmax, 0);
    rc = denoise_one_workgroup_per_tile(p, nq, obs_quick, noise_quick, ids.data(), w.ref_q, stream);
    if (rc) return rc;
    if (nf > 0) {
      rc = denoise_one_workgroup_per_tile(p, nf, obs_formal, noise_formal, ids.data(), w.ref_f, stream);
      if (rc) return rc;
    }
    std::vector<float> dev((size_t)bmax);
    std::vector<int32_t> pairs(2 * (size_t)K);
    auto set_pairs = [&](int slot, const int32_t* sch) {
      for (int k = 0; k < K; ++k) {
        pairs[2 * k] = sch[k] / T;
        pairs[2 * k + 1] = sch[k] % T;
      }
      return evo_set_schedule_pairs(p, slot, pairs.data(), K, opt->granularity);
    };
    // deviations of `batch` episodes against `ref` (episode i against i % n_ref), back to the host
    auto deviations = [&](int batch, const float* ref, int n_ref) -> int {
      hipLaunchKernelGGL(deviation_kernel, dim3(batch), dim3(64), 0, stream, w.out, ref, w.dev, batch, n_ref, HA);
      if (hipGetLastError() != hipSuccess) return fail(EVO_E_HIP, "deviation kernel launch failed");
      if (hipMemcpyAsync(dev.data(), w.dev, sizeof(float) * batch, hipMemcpyDeviceToHost, stream) != hipSuccess)
        return fail(EVO_E_HIP, "deviation copy failed");
      if (hipStreamSynchronize(stream) != hipSuccess) return fail(EVO_E_HIP, "stream synchronize failed");
      return evo_synchronize(p);
    };
    int built_for = -1;  // candidates the replicated episode buffers currently hold
    SearchEval ev;
    ev.quick = [&](int n, const int32_t* sch, double* fit) -> int {
      if (n > P) return fail(EVO_E_STATE, "more new schedules than the population");
      for (int j = 0; j < n; ++j) {
        const int r = set_pairs(j, sch + (size_t)j * K);
        if (r) return r;
      }
      const int batch = n * nq;
      if (built_for != n) {
        if (replicate(obs_quick, w.obs, 1, nq, batch, OB, stream) != hipSuccess ||
            replicate(noise_quick, w.noise, T, nq, batch, HA, stream) != hipSuccess)
          return fail(EVO_E_HIP, "episode replication failed");
        built_for = n;
      }
      for (int i = 0; i < batch; ++i) ids[i] = i / nq;
      int r = denoise_one_workgroup_per_tile(p, batch, w.obs, w.noise, ids.data(), w.out, stream);
      if (r) return r;
      r = deviations(batch, w.ref_q, nq);
      if (r) return r;
      for (int j = 0; j < n; ++j) {
        int ok = 0;
        for (int e = 0; e < nq; ++e) ok += dev[(size_t)j * nq + e] <= opt->tau;
        fit[j] = (double)ok / nq;
      }
      return EVO_OK;
    };
    if (nf > 0)
      ev.formal = [&](const int32_t* sch, double* score) -> int {
        int r = set_pairs(0, sch);
        if (r) return r;
        std::fill(ids.begin(), ids.begin() + nf, 0);
        r = denoise_one_workgroup_per_tile(p, nf, obs_formal, noise_formal, ids.data(), w.out, stream);
        if (r) return r;
        r = deviations(nf, w.ref_f, nf);
        if (r) return r;
        int ok = 0;
        for (int e = 0; e < nf; ++e) ok += dev[e] <= opt->tau;
        *score = (double)ok / nf;
        return EVO_OK;
      };
    rc = ga_search(*cfg, rows, T, probs, ev, opt->q_base, opt->delta_acc, result, best_out, pop_history, fit_history);
    (void)hipStreamSynchronize(stream);
    return rc;
  });
}
