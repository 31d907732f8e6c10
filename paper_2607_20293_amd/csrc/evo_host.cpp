// Host-side runtime: see evo_host.hpp.
#include "evo_host.hpp"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <vector>

namespace evo {

static thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

void clear_error() { g_err.clear(); }

const char* last_error() { return g_err.c_str(); }

int shape_from_desc(const evo_policy_desc* desc, Shape* out) {
  if (!desc) return fail(EVO_E_INVALID, "desc is NULL");
  Shape s;
  s.L = desc->n_layers; s.d = desc->d_model; s.nh = desc->n_heads; s.dff = desc->d_ff;
  s.H = desc->horizon; s.A = desc->action_dim; s.n_obs = desc->n_obs_tokens;
  s.obs_dim = desc->obs_dim; s.T = desc->n_steps; s.dtype = desc->dtype;
  s.cold = desc->cold_policy; s.clip = desc->clip_sample != 0;
  s.max_batch = desc->max_batch; s.max_sched = desc->max_schedules;
  if (s.L < 1 || s.L > 21) return fail(EVO_E_INVALID, "n_layers must be in [1, 21] (3L <= 63 units)");
  if (s.d < 16 || s.nh < 1 || s.d % s.nh) return fail(EVO_E_INVALID, "d_model must be >= 16 and divisible by n_heads");
  if (s.d % 2) return fail(EVO_E_INVALID, "d_model must be even (sinusoidal time embedding)");
  if (s.d / 2 < 2) return fail(EVO_E_INVALID, "d_model too small for the time embedding");
  if (s.dff < 1) return fail(EVO_E_INVALID, "d_ff must be positive");
  if (s.H < 1 || s.A < 1) return fail(EVO_E_INVALID, "horizon and action_dim must be positive");
  if (s.n_obs < 1 || s.obs_dim < 1) return fail(EVO_E_INVALID, "n_obs_tokens and obs_dim must be positive");
  if (s.T < 1 || s.T > 1000) return fail(EVO_E_INVALID, "n_steps must be in [1, 1000]");
  if (s.dtype != EVO_FP32 && s.dtype != EVO_BF16) return fail(EVO_E_INVALID, "dtype must be EVO_FP32 or EVO_BF16");
  if (s.cold != EVO_COLD_COMPUTE && s.cold != EVO_COLD_ZERO) return fail(EVO_E_INVALID, "bad cold_policy");
  if (s.max_batch < 1 || s.max_batch > (1 << 20)) return fail(EVO_E_INVALID, "max_batch must be in [1, 2^20]");
  if (s.max_sched < 1 || s.max_sched > 4096) return fail(EVO_E_INVALID, "max_schedules must be in [1, 4096]");
  *out = s;
  return EVO_OK;
}

WeightOffsets weight_offsets(const Shape& s) {
  WeightOffsets o;
  size_t off = 0;
  auto take = [&](size_t n) { size_t r = off; off += n; return r; };
  const size_t d = s.d;
  o.W_in = take(d * s.A); o.b_in = take(d); o.P_act = take((size_t)s.H * d);
  o.W_obs = take(d * s.obs_dim); o.b_obs = take(d); o.P_mem = take((size_t)s.S() * d);
  o.layer.resize(s.L);
  for (int l = 0; l < s.L; ++l) {
    auto& y = o.layer[l];
    y.ln1_g = take(d); y.ln1_b = take(d); y.W_qkv = take(3 * d * d); y.b_qkv = take(3 * d);
    y.W_o = take(d * d); y.b_o = take(d);
    y.ln2_g = take(d); y.ln2_b = take(d); y.W_q = take(d * d); y.b_q = take(d);
    y.W_kv = take(2 * d * d); y.b_kv = take(2 * d); y.W_o2 = take(d * d); y.b_o2 = take(d);
    y.ln3_g = take(d); y.ln3_b = take(d); y.W_1 = take((size_t)s.dff * d); y.b_1 = take(s.dff);
    y.W_2 = take(d * (size_t)s.dff); y.b_2 = take(d);
  }
  o.lnf_g = take(d); o.lnf_b = take(d); o.W_out = take((size_t)s.A * d); o.b_out = take(s.A);
  o.total = off;
  return o;
}

Flops flops_of(const Shape& s) {
  Flops f;
  const uint64_t H = s.H, d = s.d, S = s.S(), dff = s.dff, A = s.A;
  f.unit[UNIT_SA] = 2 * (4 * H * d * d + 2 * H * H * d);
  f.unit[UNIT_CA] = 2 * (2 * H * d * d + 2 * S * d * d + 2 * H * S * d);
  f.unit[UNIT_FFN] = 2 * (2 * H * d * dff);
  f.unit_kernel[UNIT_SA] = f.unit[UNIT_SA];
  f.unit_kernel[UNIT_CA] = 2 * (2 * H * d * d + 2 * H * S * d);
  f.unit_kernel[UNIT_FFN] = f.unit[UNIT_FFN];
  f.always_step = 4 * H * A * d;
  f.always_query = 2 * (uint64_t)s.n_obs * s.obs_dim * d;
  f.query_kernel = f.always_query + 2 * (uint64_t)s.n_obs * (2 * d) * d * s.L;
  if (s.folds_ca()) {
    // folded: scores and output against n_heads x S columns; the fold of the
    // observation tokens (u and w, a d x d product each) once per query
    const uint64_t nh = s.nh;
    f.unit_kernel[UNIT_CA] = 2 * (2 * H * S * nh * d);
    f.query_kernel += 2 * (uint64_t)s.n_obs * (2 * d) * d * s.L;
  }
  return f;
}

void unit_weight_bytes(const Shape& s, uint64_t out[3]) {
  const uint64_t d = s.d, e = s.elt();
  out[UNIT_SA] = 4 * d * d * e;
  out[UNIT_CA] = 2 * d * d * e;
  out[UNIT_FFN] = 2 * d * (uint64_t)s.dff * e;
}

int build_schedule(const Shape& s, const uint8_t* lattice, int rows, int granularity, Schedule* out) {
  if (!lattice) return fail(EVO_E_INVALID, "lattice is NULL");
  if (granularity != EVO_GRAN_LAYER && granularity != EVO_GRAN_UNIT)
    return fail(EVO_E_INVALID, "granularity must be EVO_GRAN_LAYER or EVO_GRAN_UNIT");
  const int L = s.L, U = s.U(), T = s.T;
  const int want = granularity == EVO_GRAN_LAYER ? L : U;
  if (rows != want)
    return fail(EVO_E_INVALID, "lattice has %d rows, expected %d for this granularity", rows, want);
  for (size_t i = 0; i < (size_t)rows * T; ++i)
    if (lattice[i] > 1) return fail(EVO_E_INVALID, "lattice entry %zu is %d (must be 0 or 1)", i, (int)lattice[i]);
  // unit lattice (requested) and effective lattice (cold-cache reading)
  std::vector<uint8_t> req((size_t)U * T), eff;
  for (int b = 0; b < U; ++b) {
    const int r = granularity == EVO_GRAN_LAYER ? b / 3 : b;
    for (int t = 0; t < T; ++t) req[(size_t)b * T + t] = lattice[(size_t)r * T + t];
  }
  eff = req;
  if (s.cold == EVO_COLD_COMPUTE)
    for (int b = 0; b < U; ++b) eff[(size_t)b * T] = 1;
  Schedule sc;
  sc.valid = true;
  sc.merged = granularity == EVO_GRAN_LAYER;
  sc.codes.assign((size_t)U * T, 0);
  sc.eval_mask.assign(T, 0);
  const Flops f = flops_of(s);
  for (int b = 0; b < U; ++b) {
    const int u = b % 3;
    bool seen = false;  // refreshed at an earlier step of this query
    for (int t = 0; t < T; ++t) {
      const bool e = eff[(size_t)b * T + t];
      sc.requested += req[(size_t)b * T + t];
      uint8_t c = 0;
      if (e) {
        c = CODE_EVAL;
        const bool next_reuse = (t + 1 < T) && !eff[(size_t)b * T + t + 1];
        // merged: the layer's sum is stored at its FFN position
        if (next_reuse && (!sc.merged || u == UNIT_FFN)) c |= CODE_STORE;
        sc.effective += 1;
        sc.flops += f.unit[u];
        sc.flops_kernel += f.unit_kernel[u];
        sc.eval_mask[t] |= (1ull << b);
        seen = true;
      } else if (seen && (!sc.merged || u == UNIT_FFN)) {
        c = CODE_REUSE;
      }
      if (sc.merged) c |= CODE_MERGED;
      if (c & CODE_REUSE) sc.reuse_count++;
      if (c & CODE_STORE) sc.store_count++;
      sc.codes[(size_t)b * T + t] = c;
    }
  }
  sc.masks.assign((size_t)T * 3, 0);
  for (int t = 0; t < T; ++t) {
    uint64_t ev = 0, ru = 0, st = 0;
    for (int b = 0; b < U; ++b) {
      const uint8_t c = sc.codes[(size_t)b * T + t];
      if (c & CODE_EVAL) ev |= 1ull << b;
      if (c & CODE_REUSE) ru |= 1ull << b;
      if (c & CODE_STORE) st |= 1ull << b;
    }
    sc.masks[(size_t)t * 3 + 0] = ev | (sc.merged ? MASK_MERGED_BIT : 0);
    sc.masks[(size_t)t * 3 + 1] = ru;
    sc.masks[(size_t)t * 3 + 2] = st;
  }
  *out = std::move(sc);
  return EVO_OK;
}

void PlanSpace::reserve(int max_batch, int max_sched) {
  const size_t B = (size_t)std::max(max_batch, 1), S = (size_t)std::max(max_sched, 1);
  order.assign(B, 0);
  count.assign(S + 1, 0);
  slot_of.assign(S, -1);
  merged.assign(B + 8, -1);  // tiles of up to 8 samples, the last one padded
  tile_sample.assign(B + 8, -1);
  tile_slot.assign(B + 8, 0);
  used.assign(S, 0);
}

int plan_into(const std::vector<Schedule>& reg, const int32_t* ids, int batch, int spt, int n_xcd, PlanSpace* ps) {
  if (spt < 1) spt = 1;
  if (n_xcd < 1) n_xcd = 1;
  const int S = (int)reg.size();
  if (spt > 8 || batch < 0 || (size_t)batch > ps->order.size() || ps->count.size() < (size_t)S + 1 ||
      ps->slot_of.size() < (size_t)S || ps->used.size() < (size_t)S)
    return fail(EVO_E_STATE, "plan workspace too small");
  auto id_of = [&](int n) { return ids ? ids[n] : 0; };
  // samples sorted by schedule id, stable (counting sort)
  std::fill(ps->count.begin(), ps->count.begin() + S + 1, 0);
  for (int n = 0; n < batch; ++n) ++ps->count[id_of(n) + 1];
  for (int i = 0; i < S; ++i) ps->count[i + 1] += ps->count[i];
  for (int n = 0; n < batch; ++n) ps->order[ps->count[id_of(n)]++] = n;
  // tiles in sorted order, a tile never mixing schedules; short tiles (a
  // schedule's sample count not a multiple of spt) are then merged in order
  // to avoid idle slots (correct for any mix: the kernel evaluates the
  // union and selects per sample).  Emitted tiles land in `merged`.
  int32_t cur[8];
  int ncur = 0, nt = 0;
  const auto emit = [&](const int32_t* t, int len) {
    for (int j = 0; j < spt; ++j) ps->merged[(size_t)nt * spt + j] = j < len ? t[j] : -1;
    ++nt;
  };
  for (int i = 0; i < batch;) {
    const int sid = id_of(ps->order[i]);
    const int i0 = i;
    while (i < batch && i - i0 < spt && id_of(ps->order[i]) == sid) ++i;
    if (i - i0 == spt) {
      emit(&ps->order[i0], spt);
      continue;
    }
    for (int k = i0; k < i; ++k) {
      cur[ncur++] = ps->order[k];
      if (ncur == spt) {
        emit(cur, spt);
        ncur = 0;
      }
    }
  }
  if (ncur) emit(cur, ncur);
  // schedules referenced by the call, in order of first use
  std::fill(ps->slot_of.begin(), ps->slot_of.begin() + S, -1);
  int nu = 0;
  for (int n = 0; n < batch; ++n) {
    const int sid = id_of(n);
    if (ps->slot_of[sid] < 0) {
      ps->slot_of[sid] = nu;
      ps->used[nu++] = sid;
    }
  }
  // XCD-aware placement: position q runs on XCD q % n_xcd; the tiles of
  // XCD x are a contiguous run of the sorted order
  int next = 0;
  for (int x = 0; x < n_xcd && x < nt; ++x)
    for (int q = x; q < nt; q += n_xcd, ++next)
      for (int j = 0; j < spt; ++j) {
        const int32_t smp = ps->merged[(size_t)next * spt + j];
        ps->tile_sample[(size_t)q * spt + j] = smp;
        ps->tile_slot[(size_t)q * spt + j] = smp >= 0 ? ps->slot_of[id_of(smp)] : 0;
      }
  ps->spt = spt;
  ps->n_tiles = nt;
  ps->n_used = nu;
  return EVO_OK;
}

int build_plan(const Shape& s, const std::vector<Schedule>& reg, const int32_t* ids, int batch,
               int spt, int n_xcd, Plan* out) {
  (void)s;
  PlanSpace ps;
  ps.reserve(batch, (int)reg.size());
  const int rc = plan_into(reg, ids, batch, spt, n_xcd, &ps);
  if (rc) return rc;
  Plan p;
  p.spt = ps.spt;
  p.n_tiles = ps.n_tiles;
  p.tile_sample.assign(ps.tile_sample.begin(), ps.tile_sample.begin() + (size_t)ps.n_tiles * ps.spt);
  p.tile_slot.assign(ps.tile_slot.begin(), ps.tile_slot.begin() + (size_t)ps.n_tiles * ps.spt);
  p.used.assign(ps.used.begin(), ps.used.begin() + ps.n_used);
  *out = std::move(p);
  return EVO_OK;
}

int guided_probabilities(const float* scores, size_t n, double eps, double gamma, double* p_out) {
  double lo = scores[0], hi = scores[0];
  for (size_t i = 0; i < n; ++i) {
    const double v = scores[i];
    if (!std::isfinite(v)) return fail(EVO_E_INVALID, "score %zu is not finite", i);
    lo = std::min(lo, v);
    hi = std::max(hi, v);
  }
  double tot = 0.0;
  for (size_t i = 0; i < n; ++i) {
    const double w = hi > lo ? ((double)scores[i] - lo) / (hi - lo) : 0.0;
    p_out[i] = std::pow(eps + w, gamma);
    tot += p_out[i];
  }
  if (!(tot > 0.0)) return fail(EVO_E_INVALID, "all weights are zero (eps = 0 and constant scores?)");
  for (size_t i = 0; i < n; ++i) p_out[i] /= tot;
  return EVO_OK;
}

int guided_sample(const double* p, int rows, int T, int K, const double* u, int32_t* pairs_out) {
  const size_t n = (size_t)rows * T;
  size_t positive = 0;
  for (size_t i = 0; i < n; ++i) {
    if (!(p[i] >= 0.0) || !std::isfinite(p[i])) return fail(EVO_E_INVALID, "probability %zu invalid", i);
    if (!(u[i] > 0.0 && u[i] < 1.0)) return fail(EVO_E_INVALID, "uniform %zu not in (0, 1)", i);
    positive += p[i] > 0.0;
  }
  if (K < 0 || (size_t)K > positive) return fail(EVO_E_INVALID, "K = %d exceeds the %zu positions with p > 0", K, positive);
  std::vector<std::pair<double, size_t>> key(n);
  for (size_t i = 0; i < n; ++i)
    key[i] = {p[i] > 0.0 ? std::log(p[i]) - std::log(-std::log(u[i])) : -HUGE_VAL, i};
  // K largest keys; equal keys: the lower flat index first
  std::partial_sort(key.begin(), key.begin() + K, key.end(), [](const auto& a, const auto& b) {
    return a.first != b.first ? a.first > b.first : a.second < b.second;
  });
  std::vector<size_t> chosen(K);
  for (int k = 0; k < K; ++k) chosen[k] = key[k].second;
  std::sort(chosen.begin(), chosen.end());
  for (int k = 0; k < K; ++k) {
    pairs_out[2 * k] = (int32_t)(chosen[k] / T);
    pairs_out[2 * k + 1] = (int32_t)(chosen[k] % T);
  }
  return EVO_OK;
}

void call_stats(const Shape& s, const std::vector<Schedule>& reg, const int32_t* ids, int batch,
                const int32_t* tile_sample, int n_tiles, int spt, int team, evo_stats* out) {
  evo_stats st;
  std::memset(&st, 0, sizeof(st));
  const Flops f = flops_of(s);
  uint64_t F_layer = f.unit[0] + f.unit[1] + f.unit[2];
  const uint64_t rowbytes = (uint64_t)s.H * s.d * s.cache_elt();  // cache of one sample and unit
  for (int n = 0; n < batch; ++n) {
    const Schedule& sc = reg[ids ? ids[n] : 0];
    st.refreshes_requested += sc.requested;
    st.refreshes_effective += sc.effective;
    st.flops_cacheable += sc.flops;
    st.flops_kernel += sc.flops_kernel + f.query_kernel + (uint64_t)s.T * f.always_step;
    st.cache_bytes_read += sc.reuse_count * rowbytes;
    st.cache_bytes_written += sc.store_count * rowbytes;
  }
  st.flops_always = (uint64_t)batch * ((uint64_t)s.T * f.always_step + f.always_query);
  st.flops_full = (uint64_t)batch * s.T * s.L * F_layer + st.flops_always;
  if (tile_sample) {
    uint64_t wb[3];
    unit_weight_bytes(s, wb);
    const uint64_t e = s.elt();
    const uint64_t obs_pad = (uint64_t)((s.obs_dim + 31) / 32 * 32);
    uint64_t per_query_w = obs_pad * s.d * e + (uint64_t)s.L * 2 * s.d * s.d * e;
    // folded cross-attention: the fold reads fp32 W_q and W_o2 once per
    // query; an evaluation reads the fold records (u, w, c) of its samples'
    // S tokens instead of the unit's weights
    const bool fold = s.folds_ca();
    const uint64_t rec_bytes = (uint64_t)s.S() * (2 * s.nh * s.d + s.nh) * 4;
    if (fold) per_query_w += (uint64_t)s.L * 2 * s.d * s.d * 4;
    st.n_tiles = n_tiles;
    st.n_workgroups = (uint64_t)n_tiles * team;
    st.cache_bytes_read *= team;
    st.cache_bytes_written *= team;
    for (int q = 0; q < n_tiles; ++q) {
      st.weight_bytes += per_query_w * team;
      for (int t = 0; t < s.T; ++t) {
        uint64_t mask = 0, live = 0;
        for (int j = 0; j < spt; ++j) {
          const int smp = tile_sample[(size_t)q * spt + j];
          if (smp < 0) continue;
          mask |= reg[ids ? ids[smp] : 0].eval_mask[t];
          ++live;
        }
        for (int b = 0; b < s.U(); ++b)
          if (mask >> b & 1) st.weight_bytes += (fold && b % 3 == UNIT_CA) ? live * rec_bytes * team : wb[b % 3];
      }
    }
  }
  *out = st;
}

}  // namespace evo
