// Host-runtime driver for the AddressSanitizer / UndefinedBehaviorSanitizer
// build (tests/test_host_sanitizers.py).  It links only the pure C++ host
// code of the library (schedule ingestion, batch plans, bookkeeping, Eq. 7
// helpers and the Sec. 3.2 search) and drives it over random and edge-case
// inputs: valid lattices of both granularities and cold readings, malformed
// arguments that must be refused, ragged batches with mixed schedule ids,
// and whole searches with a synthetic fitness.  Any out-of-bounds access,
// use after free, leak or undefined operation aborts the run.  On success it
// prints integer results that the Python test compares with the oracle.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "evo.h"
#include "evo_host.hpp"

using namespace evo;

namespace {

int g_fail = 0;

#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++g_fail;                                                        \
    }                                                                  \
  } while (0)

evo_policy_desc pusht_desc(int max_batch, int max_sched, int cold) {
  evo_policy_desc d{};
  d.n_layers = 8; d.d_model = 256; d.n_heads = 4; d.d_ff = 1024; d.horizon = 16; d.action_dim = 2;
  d.n_obs_tokens = 2; d.obs_dim = 20; d.n_steps = 100; d.dtype = EVO_BF16; d.cold_policy = cold;
  d.clip_sample = 1; d.max_batch = max_batch; d.max_schedules = max_sched;
  return d;
}

std::vector<uint8_t> bernoulli(std::mt19937_64& rng, int rows, int T, double p) {
  std::vector<uint8_t> lat((size_t)rows * T);
  std::bernoulli_distribution b(p);
  for (auto& v : lat) v = b(rng) ? 1 : 0;
  return lat;
}

void schedules_and_plans(std::mt19937_64& rng) {
  for (int cold : {EVO_COLD_COMPUTE, EVO_COLD_ZERO}) {
    evo_policy_desc d = pusht_desc(512, 8, cold);
    Shape s;
    EXPECT(shape_from_desc(&d, &s) == EVO_OK);
    const WeightOffsets wo = weight_offsets(s);
    EXPECT(wo.total > 0 && wo.b_out < wo.total);
    std::vector<Schedule> reg(8);
    for (int id = 0; id < 8; ++id) {
      const int gran = id % 2 ? EVO_GRAN_UNIT : EVO_GRAN_LAYER;
      const int rows = gran == EVO_GRAN_UNIT ? s.U() : s.L;
      const double p = 0.05 + 0.12 * id;
      const std::vector<uint8_t> lat = bernoulli(rng, rows, s.T, p);
      EXPECT(build_schedule(s, lat.data(), rows, gran, &reg[id]) == EVO_OK);
      EXPECT(reg[id].codes.size() == (size_t)s.U() * s.T);
      EXPECT(reg[id].masks.size() == (size_t)s.T * 3);
      EXPECT(reg[id].effective >= reg[id].requested);
    }
    // the empty lattice, the full lattice
    std::vector<uint8_t> zero((size_t)s.L * s.T, 0), full((size_t)s.U() * s.T, 1);
    Schedule z, f;
    EXPECT(build_schedule(s, zero.data(), s.L, EVO_GRAN_LAYER, &z) == EVO_OK);
    EXPECT(build_schedule(s, full.data(), s.U(), EVO_GRAN_UNIT, &f) == EVO_OK);
    EXPECT(f.effective == (uint64_t)s.U() * s.T && f.reuse_count == 0);
    // malformed arguments are refused without touching memory
    Schedule bad;
    EXPECT(build_schedule(s, nullptr, s.L, EVO_GRAN_LAYER, &bad) != EVO_OK);
    EXPECT(build_schedule(s, zero.data(), s.L + 1, EVO_GRAN_LAYER, &bad) != EVO_OK);
    EXPECT(build_schedule(s, zero.data(), s.L, 7, &bad) != EVO_OK);
    std::vector<uint8_t> two((size_t)s.L * s.T, 2);
    EXPECT(build_schedule(s, two.data(), s.L, EVO_GRAN_LAYER, &bad) != EVO_OK);
    // plans: ragged batches, mixed and shuffled ids, one and two samples per tile
    {
      // a workspace too small for the batch is refused
      PlanSpace small;
      small.reserve(4, 8);
      std::vector<int32_t> ids(5, 0);
      EXPECT(plan_into(reg, ids.data(), 5, 1, 8, &small) != EVO_OK);
    }
    for (int batch : {1, 2, 3, 63, 64, 65, 255, 256, 257, 511, 512}) {
      std::vector<int32_t> ids(batch);
      std::uniform_int_distribution<int> u(0, 7);
      for (auto& v : ids) v = u(rng);
      for (int spt : {1, 2}) {
        Plan pl;
        EXPECT(build_plan(s, reg, ids.data(), batch, spt, 8, &pl) == EVO_OK);
        EXPECT((size_t)pl.n_tiles * spt == pl.tile_sample.size());
        std::vector<int> seen(batch, 0);
        for (size_t i = 0; i < pl.tile_sample.size(); ++i) {
          const int j = pl.tile_sample[i];
          if (j < 0) continue;
          EXPECT(j < batch);
          if (j < batch) ++seen[j];
          EXPECT(pl.tile_slot[i] >= 0 && pl.tile_slot[i] < (int)pl.used.size());
        }
        for (int v : seen) EXPECT(v == 1);
        evo_stats st{};
        call_stats(s, reg, ids.data(), batch, pl.tile_sample.data(), pl.n_tiles, spt, 1, &st);
        EXPECT(st.flops_cacheable <= st.flops_full);
        // the allocation-free builder, in arrays sized for a larger batch,
        // gives the same plan
        PlanSpace ps;
        ps.reserve(512, 8);
        EXPECT(plan_into(reg, ids.data(), batch, spt, 8, &ps) == EVO_OK);
        EXPECT(ps.n_tiles == pl.n_tiles && ps.n_used == (int)pl.used.size());
        for (size_t i = 0; i < pl.tile_sample.size(); ++i)
          EXPECT(ps.tile_sample[i] == pl.tile_sample[i] && ps.tile_slot[i] == pl.tile_slot[i]);
        for (size_t i = 0; i < pl.used.size(); ++i) EXPECT(ps.used[i] == pl.used[i]);
      }
    }
  }
}

void bookkeeping_print() {
  // a fixed case whose counts the Python test recomputes with the oracle:
  // Push-T shape, unit lattice with (b, t) set where (7 b + 3 t) % 10 < 3
  evo_policy_desc d = pusht_desc(4, 2, EVO_COLD_COMPUTE);
  Shape s;
  shape_from_desc(&d, &s);
  std::vector<uint8_t> lat((size_t)s.U() * s.T);
  for (int b = 0; b < s.U(); ++b)
    for (int t = 0; t < s.T; ++t) lat[(size_t)b * s.T + t] = ((7 * b + 3 * t) % 10) < 3;
  std::vector<Schedule> reg(2);
  build_schedule(s, lat.data(), s.U(), EVO_GRAN_UNIT, &reg[0]);
  std::vector<uint8_t> all((size_t)s.L * s.T, 1);
  build_schedule(s, all.data(), s.L, EVO_GRAN_LAYER, &reg[1]);
  const int32_t ids[4] = {1, 0, 0, 1};
  evo_stats st{};
  call_stats(s, reg, ids, 4, nullptr, 0, 1, 1, &st);
  std::printf("stats %llu %llu %llu %llu %llu\n", (unsigned long long)st.refreshes_requested,
              (unsigned long long)st.refreshes_effective, (unsigned long long)st.flops_cacheable,
              (unsigned long long)st.flops_always, (unsigned long long)st.flops_full);
}

void eq7(std::mt19937_64& rng) {
  const int rows = 24, T = 100;
  std::vector<float> sc((size_t)rows * T);
  std::uniform_real_distribution<float> uf(0.f, 2.f);
  for (auto& v : sc) v = uf(rng);
  std::vector<double> p(sc.size()), u(sc.size());
  EXPECT(guided_probabilities(sc.data(), sc.size(), 0.05, 2.0, p.data()) == EVO_OK);
  double sum = 0.0;
  for (double v : p) sum += v;
  EXPECT(std::fabs(sum - 1.0) < 1e-12);
  std::uniform_real_distribution<double> ud(1e-12, 1.0 - 1e-12);
  for (auto& v : u) v = ud(rng);
  std::vector<int32_t> pairs(2 * 240);
  EXPECT(guided_sample(p.data(), rows, T, 240, u.data(), pairs.data()) == EVO_OK);
  EXPECT(guided_sample(p.data(), rows, T, rows * T + 1, u.data(), pairs.data()) != EVO_OK);
  // constant scores: all weights zero after min-max normalisation
  std::vector<float> flat(sc.size(), 0.5f);
  EXPECT(guided_probabilities(flat.data(), flat.size(), 0.05, 2.0, p.data()) == EVO_OK);
}

struct Fit {
  int rows, T, K;
  int calls = 0;
};

int quick_fn(void* user, int32_t n, const int32_t* sch, double* out) {
  Fit* f = static_cast<Fit*>(user);
  ++f->calls;
  for (int i = 0; i < n; ++i) {
    // synthetic fitness: fraction of positions in the first quarter of the steps
    int early = 0;
    for (int k = 0; k < f->K; ++k) early += (sch[(size_t)i * f->K + k] % f->T) < f->T / 4;
    out[i] = (double)early / f->K;
  }
  return 0;
}

int formal_fn(void* user, const int32_t* sch, double* out) {
  double v = 0.0;
  quick_fn(user, 1, sch, &v);
  *out = v;
  return 0;
}

void search(std::mt19937_64& rng) {
  const int rows = 24, T = 100;
  for (int early : {0, 1}) {
    evo_ga_config c{};
    c.K = 240; c.pop_size = 30; c.n_elite = 10; c.max_generations = 6; c.tournament = 2; c.n_guided = 15;
    c.mutation_rate = 0.05; c.seed = rng();
    std::vector<double> p((size_t)rows * T, 1.0 / (rows * T));
    Fit f{rows, T, c.K};
    evo_search_result res{};
    std::vector<int32_t> best(c.K), hist((size_t)c.max_generations * c.pop_size * c.K);
    std::vector<double> fh((size_t)c.max_generations * c.pop_size);
    const int rc = evo_ga_search(&c, rows, T, p.data(), quick_fn, early ? formal_fn : nullptr, &f, 0.5, 0.1,
                                 &res, best.data(), hist.data(), fh.data());
    EXPECT(rc == EVO_OK);
    EXPECT(res.generations >= 1 && res.generations <= c.max_generations);
    for (int k = 1; k < c.K; ++k) EXPECT(best[k] > best[k - 1]);
    std::vector<int32_t> pop((size_t)c.pop_size * c.K), next(pop.size());
    EXPECT(evo_ga_initial_population(&c, rows, T, p.data(), pop.data()) == EVO_OK);
    std::vector<double> fit(c.pop_size);
    quick_fn(&f, c.pop_size, pop.data(), fit.data());
    EXPECT(evo_ga_next_generation(&c, rows, T, 1, pop.data(), fit.data(), next.data()) == EVO_OK);
    // refused: K beyond the lattice, a NULL population
    evo_ga_config b = c;
    b.K = rows * T + 1;
    EXPECT(evo_ga_initial_population(&b, rows, T, p.data(), pop.data()) != EVO_OK);
    EXPECT(evo_ga_next_generation(&c, rows, T, 1, nullptr, fit.data(), next.data()) != EVO_OK);
  }
}

}  // namespace

int main() {
  std::mt19937_64 rng(20261202);
  schedules_and_plans(rng);
  bookkeeping_print();
  eq7(rng);
  search(rng);
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("host driver ok\n");
  return 0;
}
