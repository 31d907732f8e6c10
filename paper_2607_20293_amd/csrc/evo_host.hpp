// Host-side runtime of the cached denoising library: descriptor checks,
// weight offsets, schedule execution codes, batch plans and integer
// bookkeeping.  Pure C++ (no HIP), so every decision made here can be tested
// on a machine without a GPU.
#pragma once

#include <cstdint>
#include <string>
#include <exception>
#include <functional>
#include <new>
#include <vector>

#include "evo.h"

namespace evo {

// thread-local error message of the last failed ABI call
int fail(int code, const char* fmt, ...);
void clear_error();

// Execution code of one (unit, step) position for one schedule.
enum : uint8_t {
  CODE_EVAL = 1,    // evaluate the residual branch (Eq. 1, (b,t) in S')
  CODE_STORE = 2,   // store the cache after evaluating (it is read later)
  CODE_REUSE = 4,   // add the cached residual (Eq. 1, (b,t) not in S')
  CODE_MERGED = 8,  // layer-merged caches: SA+CA+FFN residuals cached as one sum
};

enum { UNIT_SA = 0, UNIT_CA = 1, UNIT_FFN = 2 };

struct Shape {
  int L = 0, d = 0, nh = 0, dff = 0, H = 0, A = 0, n_obs = 0, obs_dim = 0, T = 0;
  int dtype = EVO_BF16, cold = EVO_COLD_COMPUTE, clip = 1;
  int max_batch = 0, max_sched = 0;
  int U() const { return 3 * L; }
  int dh() const { return d / nh; }
  int S() const { return 1 + n_obs; }
  int elt() const { return dtype == EVO_BF16 ? 2 : 4; }
  // bytes per cached residual value (the kernels' cache layout): fp16 with
  // bf16 operands, fp32 otherwise, at every tile size
  int cache_elt() const { return dtype == EVO_BF16 ? 2 : 4; }
  // Cross-attention folded into per-token fold records (the kernels of
  // width 256 compile the folded unit; its n_heads x S score columns must
  // fit one 16-wide tile).
  bool folds_ca() const { return d == 256 && dh() == 64 && H >= 16 && nh * S() <= 16; }
  int fold_rec() const { return 2 * nh * d + 16; }  // floats per fold record
};

// Validates field ranges; does not check compiled-shape support.
int shape_from_desc(const evo_policy_desc* desc, Shape* out);

// Offsets (in floats) of every tensor of the flat weight vector.
struct WeightOffsets {
  size_t W_in, b_in, P_act, W_obs, b_obs, P_mem;
  struct Layer {
    size_t ln1_g, ln1_b, W_qkv, b_qkv, W_o, b_o;
    size_t ln2_g, ln2_b, W_q, b_q, W_kv, b_kv, W_o2, b_o2;
    size_t ln3_g, ln3_b, W_1, b_1, W_2, b_2;
  };
  std::vector<Layer> layer;
  size_t lnf_g, lnf_b, W_out, b_out;
  size_t total;
};
WeightOffsets weight_offsets(const Shape& s);

// Integer FLOP constants (2 per multiply-add) per sample.
struct Flops {
  uint64_t unit[3];          // convention of Tables 1-3 (CA includes memory K/V)
  uint64_t unit_kernel[3];   // this implementation (CA memory K/V hoisted)
  uint64_t always_step;      // embedding + head
  uint64_t always_query;     // observation projection
  uint64_t query_kernel;     // observation projection + observation-token K/V, all layers
};
Flops flops_of(const Shape& s);

// Weight bytes an evaluation of each unit type streams (bf16 or fp32).
void unit_weight_bytes(const Shape& s, uint64_t out[3]);

struct Schedule {
  bool valid = false;
  bool merged = false;
  std::vector<uint8_t> codes;   // [U][T]
  uint64_t requested = 0;       // unit positions in S
  uint64_t effective = 0;       // unit positions in S'
  uint64_t flops = 0;           // Tables 1-3 convention, per sample
  uint64_t flops_kernel = 0;    // this implementation, per sample (without per-query work)
  uint64_t reuse_count = 0;     // positions with CODE_REUSE
  uint64_t store_count = 0;     // positions with CODE_STORE
  std::vector<uint64_t> eval_mask;  // [T] bitmask of evaluated units (U <= 63)
  // Device form of the codes: per step t, three unit bitmasks
  // {evaluate, reuse, store} (bit 63 of the evaluate mask = layer-merged).
  std::vector<uint64_t> masks;      // [T][3]
};

constexpr uint64_t MASK_MERGED_BIT = 1ull << 63;

// Build execution codes from a lattice (rows = L or 3L, row-major [rows][T]).
int build_schedule(const Shape& s, const uint8_t* lattice, int rows, int granularity,
                   Schedule* out);

// Per-call plan: samples grouped into tiles of `spt` samples sharing a
// schedule where possible, tiles ordered so that consecutive tiles of the
// sorted order land on the same XCD (workgroup i runs on XCD i % 8).
struct Plan {
  int spt = 1;
  int n_tiles = 0;
  std::vector<int32_t> tile_sample;   // [n_tiles][spt], -1 = empty slot
  std::vector<int32_t> tile_slot;     // [n_tiles][spt], index into `used`
  std::vector<int32_t> used;          // schedule ids referenced by the call
};
int build_plan(const Shape& s, const std::vector<Schedule>& reg, const int32_t* ids, int batch,
               int spt, int n_xcd, Plan* out);

// The same plan built without allocating: every array is sized once by
// reserve() (a batch of up to max_batch samples, schedule ids below
// max_sched, up to 8 samples per tile); plan_into only writes into them.
struct PlanSpace {
  std::vector<int32_t> order, count, slot_of, merged;  // work arrays
  std::vector<int32_t> tile_sample, tile_slot, used;   // the plan (first n_tiles*spt / n_used entries)
  int spt = 1, n_tiles = 0, n_used = 0;
  void reserve(int max_batch, int max_sched);
};
int plan_into(const std::vector<Schedule>& reg, const int32_t* ids, int batch, int spt, int n_xcd, PlanSpace* ps);

// Eq. 7 (Sec. 3.3): min-max normalise n scores into w and return
// p_i = (eps + w_i)^gamma / sum_j (eps + w_j)^gamma in fp64.
int guided_probabilities(const float* scores, size_t n, double eps, double gamma, double* p_out);
// K distinct positions of the [rows][T] lattice drawn one after another
// without replacement from p, by the Gumbel-top-K construction with one
// given uniform per position in (0, 1) (ties to the lower flat index);
// pairs_out [K][2] = (row, step) in flat order.
int guided_sample(const double* p, int rows, int T, int K, const double* u, int32_t* pairs_out);

// Bookkeeping of a call (refreshes, FLOPs, algorithmic bytes).  With
// `team` workgroups per tile, every member keeps its own caches and
// observation keys/values, while the per-unit weights are split among them.
// shape and device of a policy (evo_api.hip)
const Shape& policy_shape(const evo_policy* p);
int policy_device(const evo_policy* p);
// evo_denoise with one workgroup per tile at every batch size: results do
// not depend on the batch (evo_api.hip)
int denoise_one_workgroup_per_tile(evo_policy* p, int32_t batch, const float* obs_cond, const float* noise,
                                   const int32_t* schedule_ids, float* actions_out, void* hip_stream);

// Runs an ABI call's body and turns C++ exceptions (host allocation
// failures of vectors sized by the caller's arguments) into error codes, so
// none crosses the C boundary.
template <class F>
int guarded(F&& f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return fail(EVO_E_NOMEM, "host allocation failed");
  } catch (const std::exception& e) {
    return fail(EVO_E_STATE, "internal error: %s", e.what());
  } catch (...) {
    return fail(EVO_E_STATE, "internal error");
  }
}

// schedule search (evo_ga.cpp)
struct SearchEval {
  std::function<int(int, const int32_t*, double*)> quick;  // n schedules [n][K] -> fitness [n]
  std::function<int(const int32_t*, double*)> formal;      // one schedule -> formal score (empty: none)
};
int ga_check(const evo_ga_config* c, int rows, int T, const double* probs, bool initial);
int ga_check_population(const int32_t* pop, int P, int K, int N);
int ga_initial(const evo_ga_config& c, int rows, int T, const double* probs, int32_t* pop);
int ga_next(const evo_ga_config& c, int rows, int T, int gen, const int32_t* pop, const double* fit, int32_t* next);
int ga_search(const evo_ga_config& c, int rows, int T, const double* probs, const SearchEval& ev, double q_base,
              double delta_acc, evo_search_result* res, int32_t* best_out, int32_t* pop_hist, double* fit_hist);

// tile_sample: the call's plan ([n_tiles][spt], -1 = empty), or NULL for
// the counts that do not depend on it.  Allocates nothing.
void call_stats(const Shape& s, const std::vector<Schedule>& reg, const int32_t* ids, int batch,
                const int32_t* tile_sample, int n_tiles, int spt, int team, evo_stats* out);

}  // namespace evo
