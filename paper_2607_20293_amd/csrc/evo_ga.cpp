// Schedule search on the host: the evolutionary procedure of Sec. 3.2 over
// fixed-budget schedules (Eq. 5), redundancy-guided initial individuals
// (Sec. 3.3, Eq. 7), target-conditioned early stopping (Eq. 8, Eq. 9).
//
// An individual is a sorted array of K distinct flat lattice positions
// p = b*T + t; that array is its canonical signature.  Every random decision
// is one Philox4x64-10 word (Salmon, Moraes, Dror, Shaw, SC 2011) keyed by
// (seed, 0), counter (generation, purpose << 32 | slot, index, 0), so a draw
// is addressed by what it decides and the order of evaluation is free.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <vector>

#include "evo_host.hpp"

namespace evo {
namespace {

enum : uint64_t { kInit = 1, kTour = 2, kCross = 3, kMut = 4, kMutPos = 5, kDrop = 6, kFill = 7 };

inline void mulhilo(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
  const unsigned __int128 p = (unsigned __int128)a * b;
  *hi = (uint64_t)(p >> 64);
  *lo = (uint64_t)p;
}

// first output word of Philox4x64-10 at counter (c0, c1, c2, 0), key (k0, 0)
uint64_t philox_word(uint64_t k0, uint64_t c0, uint64_t c1, uint64_t c2) {
  uint64_t x0 = c0, x1 = c1, x2 = c2, x3 = 0, key0 = k0, key1 = 0;
  for (int r = 0; r < 10; ++r) {
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo(0xD2E7470EE14C6C93ull, x0, &hi0, &lo0);
    mulhilo(0xCA5A826395121157ull, x2, &hi1, &lo1);
    const uint64_t y0 = hi1 ^ x1 ^ key0, y2 = hi0 ^ x3 ^ key1;
    x0 = y0; x1 = lo1; x2 = y2; x3 = lo0;
    key0 += 0x9E3779B97F4A7C15ull;
    key1 += 0xBB67AE8584CAA73Bull;
  }
  return x0;
}

struct Draw {
  uint64_t seed;
  uint64_t gen;
  uint64_t word(uint64_t purpose, uint64_t slot, uint64_t index) const {
    return philox_word(seed, gen, (purpose << 32) | slot, index);
  }
};

// (0, 1): ((w >> 12) + 1/2) 2^-52, exact in double
inline double unit_interval(uint64_t w) { return ((double)(w >> 12) + 0.5) * 0x1p-52; }
// [0, n): high 32 bits scaled by n
inline int32_t below(uint64_t w, uint32_t n) { return (int32_t)(((w >> 32) * (uint64_t)n) >> 32); }

// Completes the sorted set s to K distinct positions of [0, N): draw j adds
// below(word(purpose, slot, j), N) unless present; after 64 N draws (never
// reached in practice) the missing positions are added in ascending order.
// mark: N zero bytes, returned zeroed.
void fill(std::vector<int32_t>& s, int K, int N, const Draw& d, uint64_t purpose, uint64_t slot,
          std::vector<uint8_t>& mark) {
  for (int32_t q : s) mark[q] = 1;
  const size_t start = s.size();
  for (uint64_t j = 0; (int)s.size() < K && j < 64ull * (uint64_t)N; ++j) {
    const int32_t p = below(d.word(purpose, slot, j), (uint32_t)N);
    if (!mark[p]) {
      mark[p] = 1;
      s.push_back(p);
    }
  }
  for (int32_t p = 0; (int)s.size() < K; ++p)
    if (!mark[p]) {
      mark[p] = 1;
      s.push_back(p);
    }
  for (int32_t q : s) mark[q] = 0;
  if (s.size() != start) std::sort(s.begin(), s.end());
}

std::vector<int32_t> ranking(const double* fit, int P) {
  std::vector<int32_t> ord(P);
  for (int i = 0; i < P; ++i) ord[i] = i;
  std::stable_sort(ord.begin(), ord.end(), [fit](int32_t a, int32_t b) { return fit[a] > fit[b]; });
  return ord;
}

int32_t tournament(const evo_ga_config& c, const Draw& d, int child, int parent, const double* fit, int P) {
  int32_t best = -1;
  for (int e = 0; e < c.tournament; ++e) {
    const int32_t idx = below(d.word(kTour, (uint64_t)child, (uint64_t)(parent * c.tournament + e)), (uint32_t)P);
    if (best < 0 || fit[idx] > fit[best] || (fit[idx] == fit[best] && idx < best)) best = idx;
  }
  return best;
}

// crossover, mutation and repair of one child (sets kept as sorted vectors)
void make_child(const evo_ga_config& c, const Draw& d, int child, const int32_t* A, const int32_t* B, int N,
                std::vector<uint8_t>& mark, int32_t* out) {
  const int K = c.K;
  const uint64_t ch = (uint64_t)child;
  // set-level crossover: A & B kept; the r-th position of A ^ B (ascending)
  // kept on bit r % 64 of word(r / 64)
  std::vector<int32_t> s;
  s.reserve(2 * K);
  uint64_t coins = 0;
  int r = 0;
  const auto coin = [&]() {
    if (r % 64 == 0) coins = d.word(kCross, ch, (uint64_t)(r / 64));
    return (coins >> (r++ % 64)) & 1ull;
  };
  int i = 0, j = 0;
  while (i < K || j < K) {
    if (j >= K || (i < K && A[i] < B[j])) {
      if (coin()) s.push_back(A[i]);
      ++i;
    } else if (i >= K || B[j] < A[i]) {
      if (coin()) s.push_back(B[j]);
      ++j;
    } else {
      s.push_back(A[i]);
      ++i;
      ++j;
    }
  }
  // mutation: the r-th position replaced when the 32-bit half r % 2 of
  // word(r / 2) is below floor(rate 2^32)
  const uint64_t thr = (uint64_t)(c.mutation_rate * 4294967296.0);
  uint64_t mw = 0;
  bool moved = false;
  for (size_t q = 0; q < s.size(); ++q) {
    if (q % 2 == 0) mw = d.word(kMut, ch, (uint64_t)(q / 2));
    if (((mw >> (32 * (q % 2))) & 0xFFFFFFFFull) < thr) {
      s[q] = below(d.word(kMutPos, ch, (uint64_t)q), (uint32_t)N);
      moved = true;
    }
  }
  if (moved) {
    std::sort(s.begin(), s.end());
    s.erase(std::unique(s.begin(), s.end()), s.end());
  }
  // repair to exactly K: remove uniformly chosen elements one at a time, or
  // complete with uniform new positions
  for (uint64_t k = 0; (int)s.size() > K; ++k)
    s.erase(s.begin() + below(d.word(kDrop, ch, k), (uint32_t)s.size()));
  if ((int)s.size() < K) fill(s, K, N, d, kFill, ch, mark);
  std::memcpy(out, s.data(), sizeof(int32_t) * K);
}

}  // namespace

int ga_check(const evo_ga_config* c, int rows, int T, const double* probs, bool initial) {
  if (!c) return fail(EVO_E_INVALID, "ga config is NULL");
  if (rows < 1 || T < 1) return fail(EVO_E_INVALID, "rows %d, n_steps %d", rows, T);
  const long long N = (long long)rows * T;
  if (N > (1ll << 30)) return fail(EVO_E_INVALID, "lattice too large");
  if (c->K < 1 || c->K > N) return fail(EVO_E_INVALID, "K = %d outside [1, %lld]", c->K, N);
  if (c->pop_size < 1 || c->pop_size > (1 << 20)) return fail(EVO_E_INVALID, "pop_size %d", c->pop_size);
  if ((long long)c->pop_size * c->K > (1ll << 28))
    return fail(EVO_E_INVALID, "pop_size x K = %lld exceeds 2^28", (long long)c->pop_size * c->K);
  if (c->n_elite < 0 || c->n_elite > c->pop_size)
    return fail(EVO_E_INVALID, "n_elite %d outside [0, pop_size]", c->n_elite);
  if (c->max_generations < 1) return fail(EVO_E_INVALID, "max_generations %d < 1", c->max_generations);
  if (c->tournament < 1) return fail(EVO_E_INVALID, "tournament %d < 1", c->tournament);
  if (c->n_guided < 0 || c->n_guided > c->pop_size)
    return fail(EVO_E_INVALID, "n_guided %d outside [0, pop_size]", c->n_guided);
  if (!(c->mutation_rate >= 0.0 && c->mutation_rate <= 1.0))
    return fail(EVO_E_INVALID, "mutation_rate outside [0, 1]");
  if (initial && c->n_guided > 0) {
    if (!probs) return fail(EVO_E_INVALID, "n_guided > 0 needs the Eq. 7 probabilities");
    long long pos = 0;
    for (long long i = 0; i < N; ++i) {
      if (!(probs[i] >= 0.0) || !std::isfinite(probs[i])) return fail(EVO_E_INVALID, "probability %lld invalid", i);
      pos += probs[i] > 0.0;
    }
    if (pos < c->K) return fail(EVO_E_INVALID, "K = %d exceeds the %lld positions with p > 0", c->K, pos);
  }
  return EVO_OK;
}

int ga_initial(const evo_ga_config& c, int rows, int T, const double* probs, int32_t* pop) {
  const int N = rows * T, K = c.K;
  const Draw d{c.seed, 0};
  std::vector<uint8_t> mark(N, 0);
  std::vector<int32_t> sub;
  std::vector<double> u;
  std::vector<int32_t> pairs;
  for (int i = 0; i < c.pop_size; ++i) {
    int32_t* ind = pop + (size_t)i * K;
    if (i < c.n_guided) {
      u.resize(N);
      pairs.resize(2 * (size_t)K);
      for (int p = 0; p < N; ++p) u[p] = unit_interval(d.word(kInit, (uint64_t)i, (uint64_t)p));
      const int rc = guided_sample(probs, rows, T, K, u.data(), pairs.data());
      if (rc) return rc;
      for (int k = 0; k < K; ++k) ind[k] = pairs[2 * k] * T + pairs[2 * k + 1];
    } else {
      sub.clear();
      fill(sub, K, N, d, kInit, (uint64_t)i, mark);
      std::memcpy(ind, sub.data(), sizeof(int32_t) * K);
    }
  }
  return EVO_OK;
}

int ga_next(const evo_ga_config& c, int rows, int T, int gen, const int32_t* pop, const double* fit,
            int32_t* next) {
  const int N = rows * T, K = c.K, P = c.pop_size;
  const Draw d{c.seed, (uint64_t)gen};
  const std::vector<int32_t> ord = ranking(fit, P);
  for (int e = 0; e < c.n_elite; ++e) std::memcpy(next + (size_t)e * K, pop + (size_t)ord[e] * K, sizeof(int32_t) * K);
  std::vector<uint8_t> mark(N, 0);
  for (int ch = 0; ch < P - c.n_elite; ++ch) {
    const int32_t a = tournament(c, d, ch, 0, fit, P);
    const int32_t b = tournament(c, d, ch, 1, fit, P);
    make_child(c, d, ch, pop + (size_t)a * K, pop + (size_t)b * K, N, mark, next + (size_t)(c.n_elite + ch) * K);
  }
  return EVO_OK;
}

int ga_check_population(const int32_t* pop, int P, int K, int N) {
  for (int i = 0; i < P; ++i) {
    const int32_t* s = pop + (size_t)i * K;
    for (int k = 0; k < K; ++k) {
      if (s[k] < 0 || s[k] >= N) return fail(EVO_E_INVALID, "individual %d position %d out of range", i, k);
      if (k > 0 && s[k] <= s[k - 1])
        return fail(EVO_E_INVALID, "individual %d is not sorted and duplicate-free", i);
    }
  }
  return EVO_OK;
}

int ga_search(const evo_ga_config& c, int rows, int T, const double* probs, const SearchEval& ev, double q_base,
              double delta_acc, evo_search_result* res, int32_t* best_out, int32_t* pop_hist, double* fit_hist) {
  const int K = c.K, P = c.pop_size;
  using Sig = std::vector<int32_t>;
  std::map<Sig, double> memo, formal_memo;
  std::vector<int32_t> pop((size_t)P * K), nxt((size_t)P * K);
  std::vector<double> fit(P);
  evo_search_result r;
  std::memset(&r, 0, sizeof(r));
  r.best_formal = std::nan("");
  int rc = ga_initial(c, rows, T, probs, pop.data());
  if (rc) return rc;
  std::vector<int32_t> batch;
  std::vector<Sig> fresh;
  std::vector<double> vals;
  int32_t best_i = -1;
  for (int gen = 0; gen < c.max_generations; ++gen) {
    if (gen > 0) {
      rc = ga_next(c, rows, T, gen, pop.data(), fit.data(), nxt.data());
      if (rc) return rc;
      pop.swap(nxt);
    }
    fresh.clear();
    for (int i = 0; i < P; ++i) {
      Sig s(pop.begin() + (size_t)i * K, pop.begin() + (size_t)(i + 1) * K);
      if (!memo.count(s) && std::find(fresh.begin(), fresh.end(), s) == fresh.end()) fresh.push_back(std::move(s));
    }
    if (!fresh.empty()) {
      batch.resize(fresh.size() * K);
      for (size_t j = 0; j < fresh.size(); ++j) std::memcpy(&batch[j * K], fresh[j].data(), sizeof(int32_t) * K);
      vals.assign(fresh.size(), 0.0);
      rc = ev.quick((int)fresh.size(), batch.data(), vals.data());
      if (rc) return rc;
      for (size_t j = 0; j < fresh.size(); ++j) memo[fresh[j]] = vals[j];
    }
    r.evaluations += (int32_t)fresh.size();
    r.memo_hits += P - (int32_t)fresh.size();
    for (int i = 0; i < P; ++i) fit[i] = memo[Sig(pop.begin() + (size_t)i * K, pop.begin() + (size_t)(i + 1) * K)];
    if (pop_hist) std::memcpy(pop_hist + (size_t)gen * P * K, pop.data(), sizeof(int32_t) * P * K);
    if (fit_hist) std::memcpy(fit_hist + (size_t)gen * P, fit.data(), sizeof(double) * P);
    r.generations = gen + 1;
    const std::vector<int32_t> ord = ranking(fit.data(), P);
    best_i = ord[0];
    if (ev.formal) {
      for (int32_t i : ord) {
        Sig s(pop.begin() + (size_t)i * K, pop.begin() + (size_t)(i + 1) * K);
        if (!(fit[i] >= q_base) || formal_memo.count(s)) continue;
        double q = 0.0;
        rc = ev.formal(s.data(), &q);
        if (rc) return rc;
        formal_memo[s] = q;
        r.formal_evaluations += 1;
        if (q >= q_base - delta_acc) {
          r.accepted = 1;
          r.best_quick = fit[i];
          r.best_formal = q;
          std::memcpy(best_out, s.data(), sizeof(int32_t) * K);
          *res = r;
          return EVO_OK;
        }
      }
    }
  }
  const Sig s(pop.begin() + (size_t)best_i * K, pop.begin() + (size_t)(best_i + 1) * K);
  r.best_quick = fit[best_i];
  auto f = formal_memo.find(s);
  if (f != formal_memo.end()) r.best_formal = f->second;
  std::memcpy(best_out, s.data(), sizeof(int32_t) * K);
  *res = r;
  return EVO_OK;
}

}  // namespace evo

extern "C" {

int evo_ga_initial_population(const evo_ga_config* cfg, int32_t rows, int32_t n_steps, const double* probs,
                              int32_t* pop_out) {
  return evo::guarded([&]() -> int {
    evo::clear_error();
    int rc = evo::ga_check(cfg, rows, n_steps, probs, true);
    if (rc) return rc;
    if (!pop_out) return evo::fail(EVO_E_INVALID, "pop_out is NULL");
    return evo::ga_initial(*cfg, rows, n_steps, probs, pop_out);
  });
}

int evo_ga_next_generation(const evo_ga_config* cfg, int32_t rows, int32_t n_steps, int32_t generation,
                           const int32_t* pop, const double* fitness, int32_t* next_out) {
  return evo::guarded([&]() -> int {
    evo::clear_error();
    int rc = evo::ga_check(cfg, rows, n_steps, nullptr, false);
    if (rc) return rc;
    if (!pop || !fitness || !next_out) return evo::fail(EVO_E_INVALID, "NULL pointer");
    if (generation < 1) return evo::fail(EVO_E_INVALID, "generation %d < 1", generation);
    for (int i = 0; i < cfg->pop_size; ++i)
      if (std::isnan(fitness[i])) return evo::fail(EVO_E_INVALID, "fitness %d is NaN", i);
    rc = evo::ga_check_population(pop, cfg->pop_size, cfg->K, rows * n_steps);
    if (rc) return rc;
    return evo::ga_next(*cfg, rows, n_steps, generation, pop, fitness, next_out);
  });
}

int evo_ga_search(const evo_ga_config* cfg, int32_t rows, int32_t n_steps, const double* probs,
                  evo_quick_fn quick, evo_formal_fn formal, void* user, double q_base, double delta_acc,
                  evo_search_result* result, int32_t* best_out, int32_t* pop_history, double* fit_history) {
  return evo::guarded([&]() -> int {
    evo::clear_error();
    int rc = evo::ga_check(cfg, rows, n_steps, probs, true);
    if (rc) return rc;
    if (!quick || !result || !best_out) return evo::fail(EVO_E_INVALID, "NULL pointer");
    if (std::isnan(q_base) || std::isnan(delta_acc)) return evo::fail(EVO_E_INVALID, "q_base / delta_acc NaN");
    evo::SearchEval ev;
    ev.quick = [&](int n, const int32_t* sch, double* out) {
      const int r = quick(user, n, sch, out);
      if (r) return evo::fail(EVO_E_STATE, "quick evaluation callback returned %d", r);
      for (int i = 0; i < n; ++i)
        if (std::isnan(out[i])) return evo::fail(EVO_E_INVALID, "quick evaluation returned NaN");
      return (int)EVO_OK;
    };
    if (formal)
      ev.formal = [&](const int32_t* sch, double* out) {
        const int r = formal(user, sch, out);
        if (r) return evo::fail(EVO_E_STATE, "formal evaluation callback returned %d", r);
        return (int)EVO_OK;
      };
    return evo::ga_search(*cfg, rows, n_steps, probs, ev, q_base, delta_acc, result, best_out, pop_history,
                          fit_history);
  });
}

}  // extern "C"
