// Device-side interface shared by the kernels and the ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace evo {

// Makes a device current for the duration of a scope.
struct DeviceGuard {
  int prev = -1, want = -1;
  explicit DeviceGuard(int dev) : want(dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != want) (void)hipSetDevice(want);
  }
  ~DeviceGuard() {
    if (prev >= 0 && prev != want) (void)hipSetDevice(prev);
  }
};

// Float offsets (into the fp32 parameter copy) of one layer's small tensors.
struct LayerOff {
  uint32_t ln1_g, ln1_b, b_qkv, b_o, ln2_g, ln2_b, b_q, b_kv, b_o2, ln3_g, ln3_b, b_1, b_2;
  uint32_t w_q;    // W_q [d][d] (fp32 parameters), folded cross-attention only
  uint32_t w_o2t;  // W_o2 transposed [d][d] (appended to the fp32 parameters), folded only
  uint32_t pad_;
};

// Offsets (in 16-byte units) of one layer's packed matrices.
struct PackOff {
  uint64_t qkv, o, q, kv, o2, w1, w2, pad_;
};

struct KParams {
  int L, A, n_obs, obs_dim, obs_pad, T, clip, n_tiles;
  const float* raw;          // fp32 parameters (flat order of evo.h)
  const uint4* pk;           // packed projection matrices
  const LayerOff* loff;      // [L]
  const PackOff* poff;       // [L]
  uint64_t pk_obs;           // fragment offset of W_obs (K padded to obs_pad)
  uint64_t pk_win;           // fp32 fragments of W_in (K = action_dim padded to 16)
  uint64_t pk_wout;          // fp32 fragments of W_out (rows padded to 16)
  uint32_t W_in, b_in, P_act, b_obs, P_mem, lnf_g, lnf_b, W_out, b_out, pad_;
  const float* tkv;          // [T][L][2d] time-token keys/values, indexed by timestep k
  const float* ddpm;         // [T][8] sampler constants by timestep k: sqrt(1-abar), 1/sqrt(abar), c0, ct, sigma
  const int32_t* tile_sample;  // [n_tiles][spt] sample index or -1
  const int32_t* tile_slot;    // [n_tiles][spt] schedule slot
  const uint64_t* masks;       // [slots][T][3] unit bitmasks {evaluate(+merged bit 63), reuse, store}
  const float* obs;          // [batch][n_obs][obs_dim]
  const float* noise;        // [T][batch][H][A]
  float* out;                // [batch][H][A]
  float* okv;                // [batch][L][n_obs][2d] observation-token keys/values
  float* cache;              // [n_tiles * team][3L][rows*d] per-workgroup residual caches
  float* acts;               // optional [batch][3L][T][H][d] record of evaluated residuals (else null)
  float* xchg;               // [n_tiles][3][team][rows*d] partial residuals of team members
  unsigned* tctr;            // [n_tiles][16] team barrier counters (zeroed before each launch)
  unsigned* derr;            // device error flag (team barrier timed out)
  size_t okv_member_stride;  // floats between team members' observation key/value copies
  int batch, team;
  unsigned spin_limit;       // polls before a team wait gives up (sets *derr)
  int withhold;              // test hook: team member 0 never publishes its partials
  int fold;                  // cross-attention folded: okv holds fold records [batch][L][n_obs][2 NH d + 16]
  const float* tfold;        // [T][L][2 NH d + 16] fold records of the time token (folded only)
};

// Shape key of a compiled kernel instantiation.
struct KernelKey {
  int d, dh, horizon, d_ff, dtype, spt, team;
};

// Returns true and the workgroup size if `key` is compiled.
bool kernel_available(const KernelKey& key, int* threads);
// Largest supported action_dim (all shapes) and n_obs_tokens (per shape).
int kernel_max_action_dim();
int kernel_max_obs_tokens_for(const KernelKey& key);
// Launch the denoising kernel: one workgroup per tile.
hipError_t launch_denoise(const KernelKey& key, const KParams& p, hipStream_t stream);

// Creation-time kernels.
// Pack rows [0, N) of the [Nvalid][K] matrix at raw + off into MFMA
// fragments (rows >= Nvalid and columns >= K are zero); dtype 1 = bf16.
hipError_t launch_pack(const float* raw, size_t off, int N, int Nvalid, int K, int Kpad, int dtype,
                       uint4* dst, hipStream_t stream);
// Largest T * samples-per-tile the kernels accept (schedule masks live in LDS).
int kernel_max_steps_x_spt();
// Time-token keys/values tkv[T][L][2d]; wkv/bkv: device arrays of the
// layers' W_kv / b_kv float offsets; rows_scratch: device float[T][d].
hipError_t launch_time_kv(const float* raw, uint32_t pmem0, const uint32_t* wkv, const uint32_t* bkv,
                          int T, int L, int D, int dtype, float* rows_scratch, float* tkv,
                          hipStream_t stream);
hipError_t launch_ddpm_table(int T, float* table, hipStream_t stream);
// Folded cross-attention: observation tokens, keys/values and fold records
// of every (sample, token, layer) into p.okv, before the denoising launch
// (d = 256; fields used: L, n_obs, obs_dim, obs_pad, raw, pk, loff, poff,
// pk_obs, b_obs, P_mem, obs, okv, batch).
hipError_t launch_obs_fold(const KParams& p, int dtype, hipStream_t stream);
// Fold records of the time token for every (timestep, layer) from its
// keys/values tkv [T][L][2d] (folded cross-attention, d = 256 only).
hipError_t launch_time_fold(const float* raw, const LayerOff* loff, const float* tkv, int T, int L, int d, int dh,
                            int dtype, float* tfold, hipStream_t stream);

// team barrier counters must start at zero on every launch (a fill kernel,
// not a memset node, so that the call may be captured into a graph)
hipError_t launch_zero_u32(unsigned* dst, int n, hipStream_t stream);

// team size of the small-batch variant for a shape (1: none compiled)
// team sizes (> 1) compiled for a shape, largest first; returns their number
int kernel_team_sizes(const KernelKey& key, int out[4]);

// Eq. 6 dissimilarity scores from recorded activations acts [R][U][T][V]:
// part [R][U][T] receives each query's term, d [U][T] their mean over R
// (in query order).  T <= kGramMaxSteps.
constexpr int kGramMaxSteps = 128;
hipError_t launch_redundancy(const float* acts, int R, int U, int T, long long V, float* part, float* d,
                             hipStream_t stream);

}  // namespace evo
