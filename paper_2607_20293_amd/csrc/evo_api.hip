// C ABI of the cached denoising library (see include/evo.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "evo_host.hpp"
#include "evo_kernels.hpp"

namespace evo {
const char* last_error();
}

using namespace evo;

namespace {

// cached values read back to the host: IEEE binary16 to fp32
float half_to_float(uint16_t h) {
  const uint32_t sign = (uint32_t)(h & 0x8000u) << 16, e = (h >> 10) & 0x1Fu, m = h & 0x3FFu;
  uint32_t u;
  if (e == 0) {  // zero or subnormal: m * 2^-24
    const float f = std::ldexp((float)m, -24);
    std::memcpy(&u, &f, 4);
    u |= sign;
  } else if (e == 31) {
    u = sign | 0x7F800000u | (m << 13);
  } else {
    u = sign | ((e + 112u) << 23) | (m << 13);
  }
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

#define HIP_TRY(expr)                                                                        \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(EVO_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

int spt_options(int horizon, int out[2]) {
  // samples per tile: tiles are whole samples and multiples of 16 rows
  if (horizon == 8) { out[0] = 2; return 1; }
  if (horizon == 16) { out[0] = 1; out[1] = 2; return 2; }
  if (horizon == 32) { out[0] = 1; return 1; }
  return 0;
}

int check_supported(const Shape& s) {
  // the kernels index one workgroup's observation keys/values with 32-bit offsets
  if ((long long)s.max_batch * s.L * s.n_obs * 2 * s.d >= (1ll << 31))
    return fail(EVO_E_UNSUPPORTED, "max_batch x n_layers x n_obs_tokens x 2 d_model must stay below 2^31");
  int opts[2];
  const int n = spt_options(s.H, opts);
  bool any = false;
  for (int i = 0; i < n; ++i) {
    KernelKey k{s.d, s.dh(), s.H, s.dff, s.dtype, opts[i], 1};
    int th;
    if (!kernel_available(k, &th)) continue;
    if (s.A > kernel_max_action_dim()) return fail(EVO_E_UNSUPPORTED, "action_dim %d > %d", s.A, kernel_max_action_dim());
    if (s.T * opts[i] > kernel_max_steps_x_spt())
      return fail(EVO_E_UNSUPPORTED, "n_steps %d too large for %d samples per tile (max %d)", s.T, opts[i],
                  kernel_max_steps_x_spt() / opts[i]);
    if (s.n_obs > kernel_max_obs_tokens_for(k))
      return fail(EVO_E_UNSUPPORTED, "n_obs_tokens %d > %d for this shape", s.n_obs, kernel_max_obs_tokens_for(k));
    any = true;
  }
  if (!any)
    return fail(EVO_E_UNSUPPORTED,
                "no kernel compiled for d_model=%d head_dim=%d horizon=%d d_ff=%d dtype=%d "
                "(compiled: d 64/hd 32/H 8/ff 256, d 256/hd 64/H 16/ff 1024, d 768/hd 64/H 32/ff 3072 bf16)",
                s.d, s.dh(), s.H, s.dff, s.dtype);
  return EVO_OK;
}

}  // namespace

// Device scratch of evo_denoise_noalloc: one fixed array per device (each
// device that loads the library holds its own copy until the process ends),
// addressed through the pointer hipGetSymbolAddress returns for that device.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};
static bool g_scratch_tried[kMaxDevices] = {};

// Looks up this device's copy of the scratch array once (the device is current).
static void* scratch_for(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_tried[device]) {
    g_scratch_tried[device] = true;
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) == hipSuccess) g_scratch_ptr[device] = ptr;
    else (void)hipGetLastError();
  }
  return g_scratch_ptr[device];
}

struct evo_policy {
  Shape s;
  int device = 0;
  int n_cu = 256;
  WeightOffsets wo;
  std::vector<LayerOff> loff_h;
  std::vector<PackOff> poff_h;
  uint64_t pk_obs = 0, pk_win = 0, pk_wout = 0;
  int obs_pad = 0;
  float* d_raw = nullptr;
  uint4* d_pk = nullptr;
  LayerOff* d_loff = nullptr;
  PackOff* d_poff = nullptr;
  float* d_tkv = nullptr;
  float* d_tfold = nullptr;  // time-token fold records (folded cross-attention)
  float* d_ddpm = nullptr;
  float* d_cache = nullptr;
  size_t cache_floats = 0;
  float* d_okv = nullptr;
  float* d_rpart = nullptr;  // per-query Eq. 6 terms [max_batch][3L][T]
  // small-batch team variants: workgroups per one-sample tile, the largest
  // batch each serves and its per-member observation K/V stride, in the
  // order they are tried (smallest max_batch first); partial-residual
  // exchange, barrier counters and the device error flag are shared
  struct TeamCfg {
    int team = 1, max_batch = 0;
    size_t okv_stride = 0;
  };
  std::vector<TeamCfg> teams;
  unsigned team_spin_limit = 1u << 20;  // EVO_TEAM_SPIN_LIMIT
  int team_withhold = 0;                // evo_debug_team_withhold (test hook)
  float* d_xchg = nullptr;
  unsigned* d_tctr = nullptr;
  unsigned* d_derr = nullptr;
  uint8_t* d_plan = nullptr;
  size_t plan_bytes = 0, tiles_cap = 0, codes_cap = 0;
  uint8_t* h_stage[2] = {nullptr, nullptr};
  hipEvent_t ev[2] = {nullptr, nullptr};
  int stage = 0;
  std::vector<uint8_t> uploaded;   // plan bytes currently in d_plan
  hipEvent_t ev_done = nullptr;    // recorded after the last launch
  hipStream_t last_stream = nullptr;
  bool launched = false;
  std::vector<Schedule> reg;
  evo_stats last{};
  bool has_last = false;
  Plan last_plan;
  int last_threads = 0;
  int last_team = 1;
  unsigned* last_derr = nullptr;  // error flag of the last call's team barriers (NULL: no team)
  bool last_noalloc = false;      // the last call ran in the device scratch array
  PlanSpace plan_ws;              // plan arrays, sized at creation
  void* scratch = nullptr;        // this device's scratch array (evo_denoise_noalloc)
  // optional timing of the denoising kernel alone: a ring of event pairs
  // recorded around its launch, harvested into t_ms / t_n
  static constexpr int kTimingPairs = 64;
  std::vector<hipEvent_t> tev;  // [2 * kTimingPairs] start, end
  std::vector<char> tev_busy;
  int tev_next = 0;
  double t_ms = 0.0;
  int64_t t_n = 0;
};

namespace evo {
const Shape& policy_shape(const evo_policy* p) { return p->s; }
int policy_device(const evo_policy* p) { return p->device; }
}  // namespace evo

static void release(evo_policy* p) {
  if (!p) return;
  // the policy's own launches end before its buffers are freed (ev_done is
  // recorded after every launch; no device-wide wait)
  if (p->launched && p->ev_done) (void)hipEventSynchronize(p->ev_done);
  (void)hipFree(p->d_raw);
  (void)hipFree(p->d_pk);
  (void)hipFree(p->d_loff);
  (void)hipFree(p->d_poff);
  (void)hipFree(p->d_tkv);
  (void)hipFree(p->d_tfold);
  (void)hipFree(p->d_ddpm);
  (void)hipFree(p->d_cache);
  (void)hipFree(p->d_okv);
  (void)hipFree(p->d_rpart);
  (void)hipFree(p->d_xchg);
  (void)hipFree(p->d_tctr);
  (void)hipFree(p->d_derr);
  (void)hipFree(p->d_plan);
  for (int i = 0; i < 2; ++i) {
    if (p->h_stage[i]) (void)hipHostFree(p->h_stage[i]);
    if (p->ev[i]) (void)hipEventDestroy(p->ev[i]);
  }
  if (p->ev_done) (void)hipEventDestroy(p->ev_done);
  for (hipEvent_t e : p->tev)
    if (e) (void)hipEventDestroy(e);
  delete p;
}

// Adds the duration of timing pair i (which must be recorded) to the sums.
static hipError_t harvest_pair(evo_policy* p, int i) {
  hipError_t e = hipEventSynchronize(p->tev[2 * i + 1]);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, p->tev[2 * i], p->tev[2 * i + 1]);
  p->tev_busy[i] = 0;
  if (e == hipSuccess) {
    p->t_ms += ms;
    p->t_n += 1;
  }
  return e;
}

static void drop_timing_events(evo_policy* p) {
  for (hipEvent_t e : p->tev)
    if (e) (void)hipEventDestroy(e);
  p->tev.clear();
  p->tev_busy.clear();
  p->tev_next = 0;
}

extern "C" {

const char* evo_last_error(void) { return evo::last_error(); }

int64_t evo_weight_count(const evo_policy_desc* desc) {
  Shape s;
  const int rc = shape_from_desc(desc, &s);
  if (rc) return rc;
  return (int64_t)weight_offsets(s).total;
}

int evo_check_desc(const evo_policy_desc* desc) {
  Shape s;
  int rc = shape_from_desc(desc, &s);
  if (rc) return rc;
  return check_supported(s);
}

int evo_create_policy(const evo_policy_desc* desc, const float* host_weights, size_t n_floats, evo_policy** out) {
  clear_error();
  Shape s;
  int rc = shape_from_desc(desc, &s);
  if (rc) return rc;
  if ((rc = check_supported(s))) return rc;
  if (!host_weights) return fail(EVO_E_INVALID, "host_weights is NULL");
  if (!out) return fail(EVO_E_INVALID, "out is NULL");
  const WeightOffsets wo = weight_offsets(s);
  if (n_floats != wo.total)
    return fail(EVO_E_INVALID, "n_floats is %zu, this shape needs %zu", n_floats, wo.total);
  if (wo.total >= (1ull << 32)) return fail(EVO_E_UNSUPPORTED, "more than 2^32 parameters");

  evo_policy* p = new (std::nothrow) evo_policy();
  if (!p) return fail(EVO_E_NOMEM, "host allocation failed");
  p->s = s;
  p->wo = wo;
  if (hipGetDevice(&p->device) != hipSuccess) {
    delete p;
    return fail(EVO_E_HIP, "no current HIP device");
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, p->device) == hipSuccess) p->n_cu = prop.multiProcessorCount;

  // the rest releases the policy itself on a failed HIP call; an exception
  // (a host allocation) is caught below and releases it too
  const auto body = [&]() -> int {
#define CREATE_TRY(expr)                                                                        \
    do {                                                                                        \
      hipError_t e_ = (expr);                                                                   \
      if (e_ != hipSuccess) {                                                                   \
        int code_ = (e_ == hipErrorOutOfMemory) ? EVO_E_NOMEM : EVO_E_HIP;                      \
        fail(code_, "%s failed: %s", #expr, hipGetErrorString(e_));                             \
        release(p);                                                                             \
        return code_;                                                                           \
      }                                                                                         \
    } while (0)

    const int L = s.L, d = s.d, T = s.T, U = s.U();
    const int KF = s.dtype == EVO_BF16 ? 32 : 16;
    // fp32 parameter copy (biases, norms, embeddings, head, and the source of the packed matrices)
    // (folded cross-attention: followed by the transpose of every layer's W_o2)
    const bool fold = s.folds_ca();
    const size_t tr_off = (wo.total + 63) / 64 * 64;  // 256-byte aligned
    const size_t raw_floats = fold ? tr_off + (size_t)L * d * d : wo.total;
    CREATE_TRY(hipMalloc(&p->d_raw, raw_floats * sizeof(float)));
    CREATE_TRY(hipMemcpy(p->d_raw, host_weights, wo.total * sizeof(float), hipMemcpyHostToDevice));
    if (fold) {
      std::vector<float> tr((size_t)L * d * d);
      for (int l = 0; l < L; ++l) {
        const float* W = static_cast<const float*>(host_weights) + wo.layer[l].W_o2;
        float* o = tr.data() + (size_t)l * d * d;
        for (int c = 0; c < d; ++c)
          for (int e = 0; e < d; ++e) o[(size_t)e * d + c] = W[(size_t)c * d + e];
      }
      CREATE_TRY(hipMemcpy(p->d_raw + tr_off, tr.data(), tr.size() * sizeof(float), hipMemcpyHostToDevice));
    }

    // packed projection matrices
    auto frag16 = [&](int N, int Kpad) { return (uint64_t)(N / 16) * (Kpad / KF) * 64; };
    p->obs_pad = (s.obs_dim + 63) / 64 * 64;
    uint64_t off = 0;
    p->pk_obs = off;
    off += frag16(d, p->obs_pad);
    // embedding and head matrices stay fp32 (16 k per fragment)
    p->pk_win = off;
    off += (uint64_t)(d / 16) * 1 * 64;
    p->pk_wout = off;
    off += (uint64_t)1 * (d / 16) * 64;
    p->poff_h.resize(L);
    for (int l = 0; l < L; ++l) {
      PackOff& po = p->poff_h[l];
      po.qkv = off; off += frag16(3 * d, d);
      po.o = off; off += frag16(d, d);
      po.q = off; off += frag16(d, d);
      po.kv = off; off += frag16(2 * d, d);
      po.o2 = off; off += frag16(d, d);
      po.w1 = off; off += frag16(s.dff, d);
      po.w2 = off; off += frag16(d, s.dff);
      po.pad_ = 0;
    }
    CREATE_TRY(hipMalloc(&p->d_pk, off * sizeof(uint4)));
    CREATE_TRY(launch_pack(p->d_raw, wo.W_obs, d, d, s.obs_dim, p->obs_pad, s.dtype, p->d_pk + p->pk_obs, 0));
    CREATE_TRY(launch_pack(p->d_raw, wo.W_in, d, d, s.A, 16, EVO_FP32, p->d_pk + p->pk_win, 0));
    CREATE_TRY(launch_pack(p->d_raw, wo.W_out, 16, s.A, d, d, EVO_FP32, p->d_pk + p->pk_wout, 0));
    for (int l = 0; l < L; ++l) {
      const auto& y = wo.layer[l];
      const PackOff& po = p->poff_h[l];
      CREATE_TRY(launch_pack(p->d_raw, y.W_qkv, 3 * d, 3 * d, d, d, s.dtype, p->d_pk + po.qkv, 0));
      CREATE_TRY(launch_pack(p->d_raw, y.W_o, d, d, d, d, s.dtype, p->d_pk + po.o, 0));
      CREATE_TRY(launch_pack(p->d_raw, y.W_q, d, d, d, d, s.dtype, p->d_pk + po.q, 0));
      CREATE_TRY(launch_pack(p->d_raw, y.W_kv, 2 * d, 2 * d, d, d, s.dtype, p->d_pk + po.kv, 0));
      CREATE_TRY(launch_pack(p->d_raw, y.W_o2, d, d, d, d, s.dtype, p->d_pk + po.o2, 0));
      CREATE_TRY(launch_pack(p->d_raw, y.W_1, s.dff, s.dff, d, d, s.dtype, p->d_pk + po.w1, 0));
      CREATE_TRY(launch_pack(p->d_raw, y.W_2, d, d, s.dff, s.dff, s.dtype, p->d_pk + po.w2, 0));
    }
    // per-layer offsets of the small tensors
    p->loff_h.resize(L);
    std::vector<uint32_t> wkv(L), bkv(L);
    for (int l = 0; l < L; ++l) {
      const auto& y = wo.layer[l];
      LayerOff& lo = p->loff_h[l];
      lo.ln1_g = (uint32_t)y.ln1_g; lo.ln1_b = (uint32_t)y.ln1_b; lo.b_qkv = (uint32_t)y.b_qkv;
      lo.b_o = (uint32_t)y.b_o; lo.ln2_g = (uint32_t)y.ln2_g; lo.ln2_b = (uint32_t)y.ln2_b;
      lo.b_q = (uint32_t)y.b_q; lo.b_kv = (uint32_t)y.b_kv; lo.b_o2 = (uint32_t)y.b_o2;
      lo.ln3_g = (uint32_t)y.ln3_g; lo.ln3_b = (uint32_t)y.ln3_b; lo.b_1 = (uint32_t)y.b_1;
      lo.b_2 = (uint32_t)y.b_2;
      lo.w_q = (uint32_t)y.W_q;
      lo.w_o2t = fold ? (uint32_t)(tr_off + (size_t)l * d * d) : 0u;
      lo.pad_ = 0;
      wkv[l] = (uint32_t)y.W_kv;
      bkv[l] = (uint32_t)y.b_kv;
    }
    CREATE_TRY(hipMalloc(&p->d_loff, L * sizeof(LayerOff)));
    CREATE_TRY(hipMemcpy(p->d_loff, p->loff_h.data(), L * sizeof(LayerOff), hipMemcpyHostToDevice));
    CREATE_TRY(hipMalloc(&p->d_poff, L * sizeof(PackOff)));
    CREATE_TRY(hipMemcpy(p->d_poff, p->poff_h.data(), L * sizeof(PackOff), hipMemcpyHostToDevice));

    // time-token keys/values for every timestep and layer; sampler constants
    {
      uint32_t *d_wkv = nullptr, *d_bkv = nullptr;
      float* rows = nullptr;
      CREATE_TRY(hipMalloc(&p->d_tkv, (size_t)T * L * 2 * d * sizeof(float)));
      CREATE_TRY(hipMalloc(&d_wkv, L * sizeof(uint32_t)));
      hipError_t e = hipMalloc(&d_bkv, L * sizeof(uint32_t));
      if (e == hipSuccess) e = hipMalloc(&rows, (size_t)T * d * sizeof(float));
      if (e == hipSuccess) e = hipMemcpy(d_wkv, wkv.data(), L * sizeof(uint32_t), hipMemcpyHostToDevice);
      if (e == hipSuccess) e = hipMemcpy(d_bkv, bkv.data(), L * sizeof(uint32_t), hipMemcpyHostToDevice);
      if (e == hipSuccess)
        e = launch_time_kv(p->d_raw, (uint32_t)wo.P_mem, d_wkv, d_bkv, T, L, d, s.dtype, rows, p->d_tkv, 0);
      if (e == hipSuccess && fold) e = hipMalloc(&p->d_tfold, (size_t)T * L * s.fold_rec() * sizeof(float));
      if (e == hipSuccess && fold)
        e = launch_time_fold(p->d_raw, p->d_loff, p->d_tkv, T, L, d, s.dh(), s.dtype, p->d_tfold, 0);
      if (e == hipSuccess) e = hipDeviceSynchronize();
      (void)hipFree(d_wkv);
      (void)hipFree(d_bkv);
      (void)hipFree(rows);
      CREATE_TRY(e);
    }
    CREATE_TRY(hipMalloc(&p->d_ddpm, (size_t)T * 8 * sizeof(float)));
    CREATE_TRY(launch_ddpm_table(T, p->d_ddpm, 0));

    // caches, observation keys/values, per-call plan buffers
    {
      int opts[2];
      const int n = spt_options(s.H, opts);
      size_t rows = 0, tiles = 0;
      int spt_max = 1;
      for (int i = 0; i < n; ++i) {
        const size_t t = (size_t)(s.max_batch + opts[i] - 1) / opts[i];
        rows = std::max(rows, t * opts[i] * s.H);
        tiles = std::max(tiles, t);
        spt_max = std::max(spt_max, opts[i]);
      }
      // team variants (one sample per tile, `team` workgroups per tile) for
      // batches that fill at most n_cu workgroups; they need cooperative
      // launch.  A team size t serves batches up to n_cu / t, the largest
      // compiled size that fits being chosen.  With bf16 operands the
      // automatic choice keeps only the smallest size: teams of 2 measured
      // faster than teams of 4 at every batch (Push-T shape, 25% density:
      // 3.57 and 3.63 ms at batch 1 and 64 against 3.65 and 4.06 ms), while
      // with fp32 operands teams of 4 are far ahead wherever they fit
      // (6.7-6.8 ms against 9.3-9.5 ms up to batch 64).
      // EVO_TEAM=0 switches teams off, EVO_TEAM=<size> keeps only that size.
      const char* env = std::getenv("EVO_TEAM");
      const int team_only = env ? std::atoi(env) : -1;
      if (const char* e = std::getenv("EVO_TEAM_SPIN_LIMIT"))
        p->team_spin_limit = (unsigned)std::min(std::strtoul(e, nullptr, 10), 1ul << 28);
      int sizes[4];
      int nsz = kernel_team_sizes(KernelKey{s.d, s.dh(), s.H, s.dff, s.dtype, 1, 0}, sizes);
      if (team_only >= 0) {
        int k = 0;
        for (int i = 0; i < nsz; ++i)
          if (sizes[i] == team_only) sizes[k++] = sizes[i];
        nsz = k;
      } else if (s.dtype == EVO_BF16 && nsz > 1) {
        sizes[0] = sizes[nsz - 1];  // sizes are sorted descending
        nsz = 1;
      }
      int coop = 0;
      (void)hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, p->device);
      // observation keys/values, or their fold records
      const size_t okv_per = (size_t)L * s.n_obs * (fold ? s.fold_rec() : 2 * d);
      size_t okv_floats = (size_t)s.max_batch * okv_per, xchg_rows = 0, ctr_tiles = 0;
      if (coop) {
        for (int i = nsz - 1; i >= 0; --i) {  // smallest team (largest batches) last in `teams`
          const int t = sizes[i];
          if (p->n_cu < t) continue;
          const int cap = p->n_cu / t;
          evo_policy::TeamCfg tc;
          tc.team = t;
          tc.max_batch = std::min(s.max_batch, std::max(cap, 1));
          tc.okv_stride = (size_t)tc.max_batch * okv_per;
          p->teams.insert(p->teams.begin(), tc);
          rows = std::max(rows, (size_t)tc.max_batch * t * s.H);
          if (!fold) okv_floats = std::max(okv_floats, tc.okv_stride * t);  // fold records: one shared copy
          xchg_rows = std::max(xchg_rows, (size_t)tc.max_batch * t * s.H);
          ctr_tiles = std::max(ctr_tiles, (size_t)tc.max_batch);
        }
      }
      p->cache_floats = (size_t)U * rows * d;  // values (bytes per value: cache_elt)
      CREATE_TRY(hipMalloc(&p->d_cache, p->cache_floats * s.cache_elt()));
      CREATE_TRY(hipMalloc(&p->d_okv, okv_floats * sizeof(float)));
      CREATE_TRY(hipMalloc(&p->d_rpart, (size_t)s.max_batch * U * T * sizeof(float)));
      if (!p->teams.empty()) {
        CREATE_TRY(hipMalloc(&p->d_xchg, xchg_rows * 3 * d * sizeof(float)));
        CREATE_TRY(hipMalloc(&p->d_tctr, ctr_tiles * 16 * sizeof(unsigned)));
        CREATE_TRY(hipMalloc(&p->d_derr, sizeof(unsigned)));
        CREATE_TRY(hipMemset(p->d_derr, 0, sizeof(unsigned)));
      }
      p->tiles_cap = tiles * spt_max;
      p->codes_cap = (size_t)std::min(s.max_sched, s.max_batch) * T * 3 * sizeof(uint64_t);
      // (room for both tile arrays, each rounded up to 256 bytes)
      p->plan_bytes = 2 * ((p->tiles_cap * sizeof(int32_t) + 255) / 256 * 256) + p->codes_cap;
      CREATE_TRY(hipMalloc(&p->d_plan, p->plan_bytes));
      for (int i = 0; i < 2; ++i) {
        CREATE_TRY(hipHostMalloc((void**)&p->h_stage[i], p->plan_bytes, hipHostMallocDefault));
        CREATE_TRY(hipEventCreateWithFlags(&p->ev[i], hipEventDisableTiming));
      }
      CREATE_TRY(hipEventCreateWithFlags(&p->ev_done, hipEventDisableTiming));
    }
    CREATE_TRY(hipDeviceSynchronize());
#undef CREATE_TRY
    p->reg.assign(s.max_sched, Schedule());
    p->plan_ws.reserve(s.max_batch, s.max_sched);
    p->scratch = scratch_for(p->device);
    *out = p;
    return EVO_OK;
  };
  try {
    return body();
  } catch (const std::bad_alloc&) {
    release(p);
    return fail(EVO_E_NOMEM, "host allocation failed");
  } catch (...) {
    release(p);
    return fail(EVO_E_STATE, "internal error");
  }
}

int evo_set_schedule(evo_policy* p, int32_t schedule_id, const uint8_t* lattice, int32_t rows, int32_t n_steps,
                     int32_t granularity) {
  return guarded([&]() -> int {
    clear_error();
    if (!p) return fail(EVO_E_INVALID, "policy is NULL");
    if (schedule_id < 0 || schedule_id >= p->s.max_sched)
      return fail(EVO_E_INVALID, "schedule_id %d outside [0, %d)", schedule_id, p->s.max_sched);
    if (n_steps != p->s.T) return fail(EVO_E_INVALID, "n_steps is %d, the policy has %d", n_steps, p->s.T);
    Schedule sc;
    const int rc = build_schedule(p->s, lattice, rows, granularity, &sc);
    if (rc) return rc;
    p->reg[schedule_id] = std::move(sc);
    return EVO_OK;
  });
}

int evo_set_schedule_pairs(evo_policy* p, int32_t schedule_id, const int32_t* pairs, int32_t K,
                           int32_t granularity) {
  return guarded([&]() -> int {
    clear_error();
    if (!p) return fail(EVO_E_INVALID, "policy is NULL");
    if (K < 0 || (K > 0 && !pairs)) return fail(EVO_E_INVALID, "bad pairs / K");
    if (granularity != EVO_GRAN_LAYER && granularity != EVO_GRAN_UNIT)
      return fail(EVO_E_INVALID, "bad granularity");
    const int rows = granularity == EVO_GRAN_LAYER ? p->s.L : p->s.U();
    const int T = p->s.T;
    std::vector<uint8_t> lat((size_t)rows * T, 0);
    for (int i = 0; i < K; ++i) {
      const int b = pairs[2 * i], t = pairs[2 * i + 1];
      if (b < 0 || b >= rows || t < 0 || t >= T) return fail(EVO_E_INVALID, "pair %d = (%d, %d) out of range", i, b, t);
      if (lat[(size_t)b * T + t]) return fail(EVO_E_INVALID, "pair %d = (%d, %d) is a duplicate", i, b, t);
      lat[(size_t)b * T + t] = 1;
    }
    return evo_set_schedule(p, schedule_id, lat.data(), rows, T, granularity);
  });
}

namespace {
// Where a call's kernels keep their working data.
struct CallBuffers {
  float* cache = nullptr;
  float* okv = nullptr;
  float* xchg = nullptr;
  unsigned* tctr = nullptr;
  unsigned* derr = nullptr;
  uint8_t* plan = nullptr;  // tile samples, tile slots, schedule masks
  size_t plan_tiles = 0;    // entries reserved for each tile array in `plan`
  size_t okv_stride = 0;    // floats between team members' observation keys/values
};
}  // namespace

// noalloc: the call's buffers are carved from the device scratch array, the
// plan is written straight into pinned staging memory and always uploaded,
// and nothing is allocated (device, pinned or host heap).
// allow_team = false: one workgroup per tile whatever the batch (the
// single- and two-sample-tile variants sum in the same order, so results do
// not depend on the batch size; the small-batch teams sum their partial
// residuals in another order).
static int denoise_impl(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                        const int32_t* schedule_ids, float* actions_out, float* acts_out, void* hip_stream,
                        bool noalloc = false, bool allow_team = true) {
  return guarded([&]() -> int {
    clear_error();
    if (!p) return fail(EVO_E_INVALID, "policy is NULL");
    const Shape& s = p->s;
    if (batch < 1 || batch > s.max_batch) return fail(EVO_E_INVALID, "batch %d outside [1, %d]", batch, s.max_batch);
    if (!obs_cond || !noise || !actions_out) return fail(EVO_E_INVALID, "NULL device pointer");
    for (int n = 0; n < batch; ++n) {
      const int id = schedule_ids ? schedule_ids[n] : 0;
      if (id < 0 || id >= s.max_sched) return fail(EVO_E_INVALID, "schedule id %d of sample %d out of range", id, n);
      if (!p->reg[id].valid) return fail(EVO_E_STATE, "schedule id %d of sample %d is not registered", id, n);
    }
    DeviceGuard guard(p->device);
    hipStream_t stream = (hipStream_t)hip_stream;
    // samples per tile: two when a single-sample tiling would oversubscribe the CUs
    int opts[2];
    const int nopt = spt_options(s.H, opts);
    int spt = 0, threads = 0, team = 1;
    for (int i = 0; i < nopt; ++i) {
      KernelKey k{s.d, s.dh(), s.H, s.dff, s.dtype, opts[i], 1};
      int th;
      if (!kernel_available(k, &th)) continue;
      if (spt == 0 || (opts[i] > spt && batch > p->n_cu)) {
        spt = opts[i];
        threads = th;
      }
    }
    if (!spt) return fail(EVO_E_UNSUPPORTED, "no kernel for this shape");
    // small batches: several workgroups per one-sample tile
    const evo_policy::TeamCfg* tc = nullptr;
    for (const auto& c : p->teams) {
      if (!allow_team || batch > c.max_batch) continue;
      KernelKey k{s.d, s.dh(), s.H, s.dff, s.dtype, 1, c.team};
      int th;
      if (kernel_available(k, &th)) {
        spt = 1;
        threads = th;
        team = c.team;
        tc = &c;
        break;
      }
    }
    PlanSpace& ps = p->plan_ws;
    int rc = plan_into(p->reg, schedule_ids, batch, spt, 8, &ps);
    if (rc) return rc;
    const size_t ntile_ent = (size_t)ps.n_tiles * spt;
    const size_t ucodes = (size_t)s.T * 3 * sizeof(uint64_t);
    if (ntile_ent > p->tiles_cap || (size_t)ps.n_used * ucodes > p->codes_cap)
      return fail(EVO_E_STATE, "plan exceeds the policy's buffers");
    if (team > 1 && ps.n_tiles > tc->max_batch) return fail(EVO_E_STATE, "team plan exceeds the buffers");
    const bool fold = s.folds_ca();
    const size_t R = (size_t)spt * s.H, D = s.d;
    CallBuffers cb;
    if (!noalloc) {
      cb.cache = p->d_cache;
      cb.okv = p->d_okv;
      cb.xchg = p->d_xchg;
      cb.tctr = p->d_tctr;
      cb.derr = p->d_derr;
      cb.plan = p->d_plan;
      cb.plan_tiles = p->tiles_cap;
      cb.okv_stride = team > 1 ? tc->okv_stride : 0;
    } else {
      // carve the scratch array: plan, caches, observation keys/values (or
      // fold records), team exchange slots, team counters and error flag
      uint8_t* base = static_cast<uint8_t*>(p->scratch);
      if (!base) return fail(EVO_E_HIP, "the device scratch array has no address on device %d", p->device);
      const auto al = [](size_t v) { return (v + 255) / 256 * 256; };
      const size_t okv_per = (size_t)s.L * s.n_obs * (fold ? s.fold_rec() : 2 * s.d);
      const size_t okv_copies = (fold || team == 1) ? 1 : (size_t)team;
      size_t off = 0;
      const size_t o_plan = off;
      off += al(2 * al(ntile_ent * sizeof(int32_t)) + (size_t)ps.n_used * ucodes);
      const size_t o_cache = off;
      off += al((size_t)ps.n_tiles * team * s.U() * R * D * s.cache_elt());
      const size_t o_okv = off;
      off += al(okv_copies * batch * okv_per * sizeof(float));
      const size_t o_xchg = off;
      if (team > 1) off += al((size_t)ps.n_tiles * 3 * team * R * D * sizeof(float));
      const size_t o_ctr = off;
      off += al(((size_t)ps.n_tiles * 16 + 1) * sizeof(unsigned));
      if (off > kScratchBytes)
        return fail(EVO_E_UNSUPPORTED,
                    "evo_denoise_noalloc: batch %d needs %zu bytes of device scratch, the array holds %zu "
                    "(use evo_denoise, or a smaller batch)",
                    batch, off, kScratchBytes);
      cb.plan = base + o_plan;
      cb.plan_tiles = al(ntile_ent * sizeof(int32_t)) / sizeof(int32_t);
      cb.cache = reinterpret_cast<float*>(base + o_cache);
      cb.okv = reinterpret_cast<float*>(base + o_okv);
      cb.xchg = team > 1 ? reinterpret_cast<float*>(base + o_xchg) : nullptr;
      cb.tctr = reinterpret_cast<unsigned*>(base + o_ctr);
      cb.derr = cb.tctr + (size_t)ps.n_tiles * 16;
      cb.okv_stride = (fold || team == 1) ? 0 : batch * okv_per;
    }
    // Calls on a different stream than the previous one wait for it: the
    // plan, caches and observation keys/values are per-policy buffers (or
    // the device's scratch array).
    if (p->launched && stream != p->last_stream) HIP_TRY(hipStreamWaitEvent(stream, p->ev_done, 0));
    // Plan bytes: tile samples, tile slots (each array cb.plan_tiles
    // entries), then the used schedules' step masks.  Staged in pinned
    // memory and uploaded; the policy's own plan buffer is not re-uploaded
    // when it already holds exactly these bytes (repeated calls).
    const size_t codes_off = (2 * cb.plan_tiles * sizeof(int32_t) + 255) / 256 * 256;
    const size_t nbytes = codes_off + (size_t)ps.n_used * ucodes;
    if (nbytes > p->plan_bytes) return fail(EVO_E_STATE, "plan exceeds the staging buffer");
    const auto fill = [&](uint8_t* dst) {
      std::memset(dst, 0, codes_off);
      std::memcpy(dst, ps.tile_sample.data(), ntile_ent * sizeof(int32_t));
      std::memcpy(dst + cb.plan_tiles * sizeof(int32_t), ps.tile_slot.data(), ntile_ent * sizeof(int32_t));
      for (int i = 0; i < ps.n_used; ++i)
        std::memcpy(dst + codes_off + i * ucodes, p->reg[ps.used[i]].masks.data(), ucodes);
    };
    const auto upload = [&](const uint8_t* src) -> int {
      const int st = p->stage;
      if (hipEventSynchronize(p->ev[st]) != hipSuccess) return fail(EVO_E_HIP, "event synchronize failed");
      if (src) std::memcpy(p->h_stage[st], src, nbytes);
      else fill(p->h_stage[st]);
      HIP_TRY(hipMemcpyAsync(cb.plan, p->h_stage[st], nbytes, hipMemcpyHostToDevice, stream));
      HIP_TRY(hipEventRecord(p->ev[st], stream));
      p->stage ^= 1;
      return EVO_OK;
    };
    if (noalloc) {
      if ((rc = upload(nullptr))) return rc;
    } else {
      std::vector<uint8_t> bytes(nbytes, 0);
      fill(bytes.data());
      if (bytes != p->uploaded) {
        if ((rc = upload(bytes.data()))) return rc;
        p->uploaded.swap(bytes);
      }
    }

    KParams kp;
    std::memset(&kp, 0, sizeof(kp));
    kp.L = s.L; kp.A = s.A; kp.n_obs = s.n_obs; kp.obs_dim = s.obs_dim; kp.obs_pad = p->obs_pad;
    kp.T = s.T; kp.clip = s.clip; kp.n_tiles = ps.n_tiles;
    kp.raw = p->d_raw; kp.pk = p->d_pk; kp.loff = p->d_loff; kp.poff = p->d_poff; kp.pk_obs = p->pk_obs;
    const WeightOffsets& wo = p->wo;
    kp.W_in = (uint32_t)wo.W_in; kp.b_in = (uint32_t)wo.b_in; kp.P_act = (uint32_t)wo.P_act;
    kp.b_obs = (uint32_t)wo.b_obs; kp.P_mem = (uint32_t)wo.P_mem; kp.lnf_g = (uint32_t)wo.lnf_g;
    kp.lnf_b = (uint32_t)wo.lnf_b; kp.W_out = (uint32_t)wo.W_out; kp.b_out = (uint32_t)wo.b_out;
    kp.tkv = p->d_tkv; kp.ddpm = p->d_ddpm;
    kp.fold = fold ? 1 : 0;
    kp.tfold = p->d_tfold;
    kp.tile_sample = reinterpret_cast<const int32_t*>(cb.plan);
    kp.tile_slot = reinterpret_cast<const int32_t*>(cb.plan) + cb.plan_tiles;
    kp.masks = reinterpret_cast<const uint64_t*>(cb.plan + codes_off);
    kp.pk_win = p->pk_win;
    kp.pk_wout = p->pk_wout;
    kp.obs = obs_cond; kp.noise = noise; kp.out = actions_out; kp.okv = cb.okv; kp.cache = cb.cache;
    kp.acts = acts_out;
    kp.batch = batch;
    kp.team = team;
    kp.okv_member_stride = fold ? 0 : cb.okv_stride;  // fold records: one copy read by every team member
    if (team > 1) {
      kp.xchg = cb.xchg;
      kp.tctr = cb.tctr;
      kp.derr = cb.derr;
      kp.spin_limit = p->team_spin_limit;
      kp.withhold = p->team_withhold;
    }
    // team counters (and, in the scratch, the error flag after them) start
    // at zero: a fill kernel, not a memset node
    if (team > 1 || noalloc)
      HIP_TRY(launch_zero_u32(cb.tctr, ps.n_tiles * 16 + (noalloc ? 1 : 0), stream));
    KernelKey key{s.d, s.dh(), s.H, s.dff, s.dtype, spt, team};
    if (kp.fold) HIP_TRY(launch_obs_fold(kp, s.dtype, stream));
    const int tslot = p->tev.empty() ? -1 : p->tev_next;
    if (tslot >= 0) {
      if (p->tev_busy[tslot]) HIP_TRY(harvest_pair(p, tslot));
      HIP_TRY(hipEventRecord(p->tev[2 * tslot], stream));
    }
    HIP_TRY(launch_denoise(key, kp, stream));
    if (tslot >= 0) {
      HIP_TRY(hipEventRecord(p->tev[2 * tslot + 1], stream));
      p->tev_busy[tslot] = 1;
      p->tev_next = (tslot + 1) % evo_policy::kTimingPairs;
    }
    HIP_TRY(hipEventRecord(p->ev_done, stream));
    p->last_stream = stream;
    p->launched = true;
    p->last_derr = team > 1 ? cb.derr : nullptr;

    call_stats(s, p->reg, schedule_ids, batch, ps.tile_sample.data(), ps.n_tiles, spt, team, &p->last);
    p->has_last = true;
    p->last_noalloc = noalloc;
    if (!noalloc) {
      Plan& lp = p->last_plan;
      lp.spt = spt;
      lp.n_tiles = ps.n_tiles;
      lp.tile_sample.assign(ps.tile_sample.begin(), ps.tile_sample.begin() + ntile_ent);
      lp.tile_slot.assign(ps.tile_slot.begin(), ps.tile_slot.begin() + ntile_ent);
      lp.used.assign(ps.used.begin(), ps.used.begin() + ps.n_used);
    }
    p->last_threads = threads;
    p->last_team = team;
    return EVO_OK;
  });
}

}  // extern "C"

namespace evo {
int denoise_one_workgroup_per_tile(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                                   const int32_t* schedule_ids, float* actions_out, void* hip_stream) {
  return denoise_impl(p, batch, obs_cond, noise, schedule_ids, actions_out, nullptr, hip_stream, false, false);
}
}  // namespace evo

extern "C" {

int evo_synchronize(evo_policy* p) {
  clear_error();
  if (!p) return fail(EVO_E_INVALID, "policy is NULL");
  DeviceGuard guard(p->device);
  if (p->launched) HIP_TRY(hipEventSynchronize(p->ev_done));
  if (p->last_derr) {
    unsigned flag = 0;
    HIP_TRY(hipMemcpy(&flag, p->last_derr, sizeof(unsigned), hipMemcpyDeviceToHost));
    if (flag) {
      HIP_TRY(hipMemset(p->last_derr, 0, sizeof(unsigned)));
      return fail(EVO_E_HIP, "a team barrier timed out on the device; outputs of that call are invalid");
    }
  }
  return EVO_OK;
}

int evo_denoise(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise, const int32_t* schedule_ids,
                float* actions_out, void* hip_stream) {
  return denoise_impl(p, batch, obs_cond, noise, schedule_ids, actions_out, nullptr, hip_stream);
}

int evo_denoise_noalloc(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                        const int32_t* schedule_ids, float* actions_out, void* hip_stream) {
  return denoise_impl(p, batch, obs_cond, noise, schedule_ids, actions_out, nullptr, hip_stream, true);
}

size_t evo_noalloc_scratch_bytes(void) { return kScratchBytes; }

int evo_collect_activations(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                            const int32_t* schedule_ids, float* actions_out, float* acts_out, void* hip_stream) {
  clear_error();
  if (!acts_out) return fail(EVO_E_INVALID, "acts_out is NULL");
  return denoise_impl(p, batch, obs_cond, noise, schedule_ids, actions_out, acts_out, hip_stream);
}

int evo_redundancy_scores(evo_policy* p, int32_t rollouts, const float* acts, float* scores_out, void* hip_stream) {
  return guarded([&]() -> int {
    clear_error();
    if (!p) return fail(EVO_E_INVALID, "policy is NULL");
    const Shape& s = p->s;
    if (!acts || !scores_out) return fail(EVO_E_INVALID, "NULL device pointer");
    if (rollouts < 1 || rollouts > s.max_batch)
      return fail(EVO_E_INVALID, "rollouts %d outside [1, %d]", rollouts, s.max_batch);
    if (s.T < 2 || s.T > kGramMaxSteps)
      return fail(EVO_E_UNSUPPORTED, "redundancy scores need 2 <= n_steps <= %d", kGramMaxSteps);
    DeviceGuard guard(p->device);
    hipStream_t stream = (hipStream_t)hip_stream;
    if (p->launched && stream != p->last_stream) HIP_TRY(hipStreamWaitEvent(stream, p->ev_done, 0));
    HIP_TRY(launch_redundancy(acts, rollouts, s.U(), s.T, (long long)s.H * s.d, p->d_rpart, scores_out, stream));
    HIP_TRY(hipEventRecord(p->ev_done, stream));
    p->last_stream = stream;
    p->launched = true;
    return EVO_OK;
  });
}

int evo_guided_probabilities(const float* scores, int32_t rows, int32_t n_steps, double eps, double gamma,
                             double* probs_out) {
  return guarded([&]() -> int {
    clear_error();
    if (!scores || !probs_out || rows < 1 || n_steps < 1) return fail(EVO_E_INVALID, "bad arguments");
    if (!(eps >= 0.0) || !(gamma >= 0.0)) return fail(EVO_E_INVALID, "eps and gamma must be >= 0");
    return guided_probabilities(scores, (size_t)rows * n_steps, eps, gamma, probs_out);
  });
}

int evo_guided_sample(const double* probs, int32_t rows, int32_t n_steps, int32_t K, const double* uniforms,
                      int32_t* pairs_out) {
  return guarded([&]() -> int {
    clear_error();
    if (!probs || !uniforms || !pairs_out || rows < 1 || n_steps < 1) return fail(EVO_E_INVALID, "bad arguments");
    return guided_sample(probs, rows, n_steps, K, uniforms, pairs_out);
  });
}

int evo_set_kernel_timing(evo_policy* p, int32_t enable) {
  clear_error();
  if (!p) return fail(EVO_E_INVALID, "policy is NULL");
  DeviceGuard guard(p->device);
  if (!enable) {
    drop_timing_events(p);
    return EVO_OK;
  }
  if (!p->tev.empty()) return EVO_OK;
  return guarded([&]() -> int {
    p->tev.assign(2 * evo_policy::kTimingPairs, nullptr);
    p->tev_busy.assign(evo_policy::kTimingPairs, 0);
    for (auto& e : p->tev) {
      const hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) {
        drop_timing_events(p);
        return fail(EVO_E_HIP, "hipEventCreate failed: %s", hipGetErrorString(r));
      }
    }
    p->t_ms = 0.0;
    p->t_n = 0;
    return EVO_OK;
  });
}

int evo_kernel_time(evo_policy* p, double* ms_total, int64_t* launches) {
  clear_error();
  if (!p) return fail(EVO_E_INVALID, "policy is NULL");
  DeviceGuard guard(p->device);
  for (int i = 0; i < (int)p->tev_busy.size(); ++i)
    if (p->tev_busy[i]) HIP_TRY(harvest_pair(p, i));
  if (ms_total) *ms_total = p->t_ms;
  if (launches) *launches = p->t_n;
  p->t_ms = 0.0;
  p->t_n = 0;
  return EVO_OK;
}

int evo_get_stats(const evo_policy* p, evo_stats* out) {
  clear_error();
  if (!p || !out) return fail(EVO_E_INVALID, "NULL argument");
  if (!p->has_last) return fail(EVO_E_STATE, "no evo_denoise call yet");
  *out = p->last;
  return EVO_OK;
}

int evo_schedule_stats(const evo_policy_desc* desc, const uint8_t* lattices, int32_t n_lat, int32_t rows,
                       int32_t granularity, const int32_t* ids, int32_t batch, evo_stats* out) {
  return guarded([&]() -> int {
    clear_error();
    Shape s;
    int rc = shape_from_desc(desc, &s);
    if (rc) return rc;
    if (!lattices || !out || n_lat < 1 || batch < 1) return fail(EVO_E_INVALID, "bad arguments");
    std::vector<Schedule> reg(n_lat);
    for (int i = 0; i < n_lat; ++i) {
      rc = build_schedule(s, lattices + (size_t)i * rows * s.T, rows, granularity, &reg[i]);
      if (rc) return rc;
    }
    for (int n = 0; n < batch; ++n) {
      const int id = ids ? ids[n] : 0;
      if (id < 0 || id >= n_lat) return fail(EVO_E_INVALID, "id %d of sample %d out of range", id, n);
    }
    call_stats(s, reg, ids, batch, nullptr, 0, 1, 1, out);
    return EVO_OK;
  });
}

int evo_schedule_codes(const evo_policy_desc* desc, const uint8_t* lattice, int32_t rows, int32_t granularity,
                       uint8_t* out) {
  return guarded([&]() -> int {
    clear_error();
    Shape s;
    int rc = shape_from_desc(desc, &s);
    if (rc) return rc;
    if (!out) return fail(EVO_E_INVALID, "out is NULL");
    Schedule sc;
    rc = build_schedule(s, lattice, rows, granularity, &sc);
    if (rc) return rc;
    std::memcpy(out, sc.codes.data(), sc.codes.size());
    return EVO_OK;
  });
}

int evo_debug_team_withhold(evo_policy* p, int32_t enable) {
  clear_error();
  if (!p) return fail(EVO_E_INVALID, "policy is NULL");
  p->team_withhold = enable != 0;
  return (int)EVO_OK;
}

int evo_debug_read_cache(evo_policy* p, int32_t unit, int32_t sample, float* host_dst) {
  return guarded([&]() -> int {
    clear_error();
    if (!p || !host_dst) return fail(EVO_E_INVALID, "NULL argument");
    if (!p->has_last) return fail(EVO_E_STATE, "no evo_denoise call yet");
    if (p->last_noalloc) return fail(EVO_E_STATE, "the last call ran in the device scratch array");
    const Shape& s = p->s;
    if (unit < 0 || unit >= s.U()) return fail(EVO_E_INVALID, "unit out of range");
    const Plan& pl = p->last_plan;
    int tile = -1, slot = -1;
    for (int q = 0; q < pl.n_tiles && tile < 0; ++q)
      for (int j = 0; j < pl.spt; ++j)
        if (pl.tile_sample[(size_t)q * pl.spt + j] == sample) { tile = q; slot = j; }
    if (tile < 0) return fail(EVO_E_INVALID, "sample %d not in the last call", sample);
    DeviceGuard guard(p->device);
    HIP_TRY(hipDeviceSynchronize());
    const int R = pl.spt * s.H, d = s.d, NW = p->last_threads / 64, RB = R / 16, CBW = d / 16 / NW;
    const size_t elt = s.cache_elt();
    std::vector<uint8_t> raw((size_t)R * d * elt);
    HIP_TRY(hipMemcpy(raw.data(),
                      reinterpret_cast<const uint8_t*>(p->d_cache) +
                          ((size_t)tile * p->last_team * s.U() + unit) * R * d * elt,
                      raw.size(), hipMemcpyDeviceToHost));
    std::vector<float> buf((size_t)R * d);
    for (size_t i = 0; i < buf.size(); ++i) {
      if (elt == 2) {
        uint16_t h;
        std::memcpy(&h, raw.data() + 2 * i, 2);
        buf[i] = half_to_float(h);
      } else {
        std::memcpy(&buf[i], raw.data() + 4 * i, 4);
      }
    }
    for (int i = 0; i < s.H; ++i) {
      const int row = slot * s.H + i, rb = row / 16, rr = row % 16;
      for (int col = 0; col < d; ++col) {
        const int cbk = col / 16, w = cbk / CBW, c = cbk % CBW;
        const int lane = (col % 16) + 16 * (rr / 4);
        host_dst[(size_t)i * d + col] = buf[((size_t)((w * RB + rb) * CBW + c) * 64 + lane) * 4 + rr % 4];
      }
    }
    return EVO_OK;
  });
}

void evo_destroy_policy(evo_policy* p) {
  if (!p) return;
  DeviceGuard guard(p->device);
  release(p);
}

}  // extern "C"
