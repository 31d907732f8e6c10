"""Pins of the schedule-search oracle (oracle/evo_search.py) against things
other than itself: numpy's Philox generator, closed-form selection laws,
distributional properties of the operators, brute force on a tiny lattice,
and the early-stopping rule of Eq. 8 / Eq. 9."""
import itertools

import numpy as np
import pytest

from oracle import evo_search as S


def _chi2_ok(counts, probs, crit):
    counts = np.asarray(counts, np.float64)
    exp = counts.sum() * np.asarray(probs, np.float64)
    return float(np.sum((counts - exp) ** 2 / exp)) < crit


# ---------------------------------------------------------------- generator
@pytest.mark.parametrize("key,ctr", [((0, 0), (0, 0, 0, 0)), ((123, 456), (5, 0, 0, 0)),
                                     ((2 ** 64 - 1, 7), (9, 2 ** 40, 3, 1)), ((77, 0), (1, 2, 3, 4))])
def test_philox_matches_numpy(key, ctr):
    """numpy's Philox (4x64, 10 rounds) emits the block of counter + 1."""
    bg = np.random.Philox(key=np.array(key, np.uint64), counter=np.array(ctr, np.uint64))
    got = [int(x) for x in bg.random_raw(4)]
    nxt = list(ctr)
    nxt[0] += 1
    assert S.philox4x64(nxt, key) == got


def test_uniform_maps():
    assert S.unit_interval(0) == 2.0 ** -53
    assert S.unit_interval(2 ** 64 - 1) == 1.0 - 2.0 ** -53
    assert 0.0 < S.unit_interval(2 ** 64 - 1) < 1.0
    for n in (1, 7, 30, 2400):
        assert S.below(0, n) == 0 and S.below(2 ** 64 - 1, n) == n - 1
    # below() splits the 2^32 high words into n near-equal intervals
    n = 7
    edges = [((j << 32) + n - 1) // n for j in range(n + 1)]
    for j in range(n):
        assert S.below(edges[j] << 32, n) == j and S.below(((edges[j + 1] - 1) << 32) | (2 ** 32 - 1), n) == j


# ---------------------------------------------------------------- initial population
def test_random_individuals_are_uniform_subsets():
    """Uniform K-subsets: every one of the C(5,2) = 10 subsets equally likely
    (chi-square, df 9, 0.999 quantile 27.9)."""
    cfg = S.GAConfig(K=2, seed=11)
    subsets = list(itertools.combinations(range(5), 2))
    counts = np.zeros(len(subsets))
    for i in range(3000):
        ind = S.random_individual(cfg, 5, i)
        assert list(ind) == sorted(set(ind)) and len(ind) == 2
        counts[subsets.index(ind)] += 1
    assert _chi2_ok(counts, np.full(10, 0.1), 27.9)


def test_guided_individuals_follow_eq7_support():
    """probs concentrated on K positions: every guided individual is exactly
    those positions; uniform probs: inclusion frequency K/N."""
    rows, T, K = 3, 8, 5
    p = np.zeros((rows, T))
    support = [1, 4, 9, 17, 23]
    p.reshape(-1)[support] = [0.1, 0.3, 0.2, 0.25, 0.15]
    cfg = S.GAConfig(K=K, pop_size=12, n_guided=12, seed=3)
    pop = S.initial_population(cfg, rows * T, p)
    assert all(list(ind) == support for ind in pop)
    cfg = S.GAConfig(K=K, pop_size=800, n_guided=800, seed=4)
    pop = S.initial_population(cfg, rows * T, np.full((rows, T), 1.0 / (rows * T)))
    freq = np.bincount(np.concatenate(pop), minlength=rows * T) / 800.0
    # Binomial(800, 5/24): sd 0.0144
    assert np.all(np.abs(freq - K / (rows * T)) < 5 * 0.0144)


def test_initial_population_mixes_guided_and_random():
    cfg = S.GAConfig(K=4, pop_size=6, n_guided=2, seed=5)
    p = np.zeros((2, 5))
    p[0, :4] = 0.25
    pop = S.initial_population(cfg, 10, p)
    assert pop[0] == (0, 1, 2, 3) and pop[1] == (0, 1, 2, 3)
    assert all(len(set(ind)) == 4 for ind in pop)


# ---------------------------------------------------------------- operators
@pytest.mark.parametrize("k", [2, 3])
def test_tournament_selection_law(k):
    """With distinct fitness, the i-th best of P wins a size-k tournament
    (entrants with replacement) with probability ((P-i)^k - (P-i-1)^k) / P^k."""
    P = 6
    fit = [0.3, 0.9, 0.1, 0.5, 0.7, 0.2]
    order = sorted(range(P), key=lambda i: -fit[i])
    law = [((P - r) ** k - (P - r - 1) ** k) / P ** k for r in range(P)]
    cfg = S.GAConfig(K=1, tournament=k, seed=21)
    counts = np.zeros(P)
    for c in range(6000):
        w = S.tournament(cfg, 1, c, 0, fit)
        counts[order.index(w)] += 1
    assert _chi2_ok(counts, law, 20.5)          # df 5, 0.999 quantile


def test_tournament_ties_go_to_lower_index():
    """Equal fitness: the lowest drawn index wins, which has the same law by
    index as distinct fitness has by rank."""
    P, k = 5, 2
    cfg = S.GAConfig(K=1, tournament=k, seed=22)
    counts = np.zeros(P)
    for c in range(5000):
        counts[S.tournament(cfg, 2, c, 1, [0.5] * P)] += 1
    law = [((P - i) ** k - (P - i - 1) ** k) / P ** k for i in range(P)]
    assert _chi2_ok(counts, law, 18.5)          # df 4


def test_crossover_is_set_level_uniform():
    cfg = S.GAConfig(K=6, seed=31)
    a, b = (0, 2, 4, 6, 8, 10), (2, 3, 6, 7, 11, 12)
    hits = {p: 0 for p in set(a) ^ set(b)}
    n = 4000
    for c in range(n):
        ch = S.crossover(cfg, 1, c, a, b)
        assert set(a) & set(b) <= ch <= set(a) | set(b)
        for p in hits:
            hits[p] += p in ch
    assert all(abs(h / n - 0.5) < 5 * 0.5 / np.sqrt(n) for h in hits.values())
    assert S.crossover(cfg, 1, 0, a, a) == set(a)


def test_mutation_rate_and_uniform_replacements():
    N, K = 100000, 40
    s = set(range(0, 4 * K, 4))
    cfg = S.GAConfig(K=K, mutation_rate=0.0, seed=41)
    assert S.mutate(cfg, 1, 0, s, N) == s
    cfg = S.GAConfig(K=K, mutation_rate=0.3, seed=41)
    lost, total, repl = 0, 0, []
    for c in range(300):
        out = S.mutate(cfg, 1, c, s, N)
        lost += len(s - out)
        total += K
        repl += sorted(out - s)
    rate = lost / total
    assert abs(rate - 0.3) < 5 * np.sqrt(0.3 * 0.7 / total)
    # replacements uniform over the lattice: 10 equal bins (df 9)
    counts = np.bincount(np.asarray(repl) * 10 // N, minlength=10)
    assert _chi2_ok(counts, np.full(10, 0.1), 27.9)


def test_repair_restores_exactly_k():
    N, K = 50, 8
    cfg = S.GAConfig(K=K, seed=51)
    small = {3, 9, 20}
    big = set(range(0, 40, 3))
    drop_hits = np.zeros(N)
    fill_hits = np.zeros(N)
    n = 3000
    for c in range(n):
        r1 = S.repair(cfg, 2, c, small, N)
        r2 = S.repair(cfg, 2, c, big, N)
        assert len(r1) == K == len(set(r1)) and small <= set(r1) and list(r1) == sorted(r1)
        assert len(r2) == K == len(set(r2)) and set(r2) <= big
        fill_hits[list(set(r1) - small)] += 1
        drop_hits[list(r2)] += 1
        assert S.repair(cfg, 2, c, set(r1), N) == r1
    # fill: 5 of the 47 missing positions, uniformly; drop: keep 8 of 14, uniformly
    miss = [p for p in range(N) if p not in small]
    assert np.all(np.abs(fill_hits[miss] / n - 5 / 47) < 5 * np.sqrt((5 / 47) * (42 / 47) / n))
    keep = sorted(big)
    assert np.all(np.abs(drop_hits[keep] / n - 8 / 14) < 5 * np.sqrt((8 / 14) * (6 / 14) / n))


def test_next_generation_keeps_elites_in_rank_order():
    cfg = S.GAConfig(K=3, pop_size=8, n_elite=3, seed=61)
    N = 12
    pop = [S.random_individual(cfg, N, i) for i in range(8)]
    fit = [0.2, 0.9, 0.5, 0.9, 0.1, 0.7, 0.3, 0.0]
    nxt = S.next_generation(cfg, N, 1, pop, fit)
    assert nxt[:3] == [pop[1], pop[3], pop[5]]      # 0.9 (index 1 before 3), 0.7
    assert len(nxt) == 8 and all(len(set(c)) == 3 and list(c) == sorted(c) for c in nxt)


# ---------------------------------------------------------------- the search loop
def _table_fitness(N, seed):
    rng = np.random.default_rng(seed)
    tab = rng.permutation(N) / N            # distinct, exact in binary
    return lambda sch: float(sum(tab[p] for p in sch))


def test_search_memoises_and_never_regresses():
    N, K = 40, 6
    f = _table_fitness(N, 1)
    seen = []

    def quick(batch):
        for s in batch:
            assert s not in seen
            seen.append(s)
        return [f(s) for s in batch]

    cfg = S.GAConfig(K=K, pop_size=10, n_elite=3, max_generations=12, n_guided=0, mutation_rate=0.1, seed=7)
    res = S.search(cfg, N, quick)
    best = [max(fs) for fs in res.fitness]
    assert all(b2 >= b1 for b1, b2 in zip(best, best[1:]))
    assert res.evaluations == len(seen) and res.evaluations + res.memo_hits == 10 * 12
    assert res.generations == 12 and not res.accepted and res.best_quick == best[-1]
    for g in range(1, 12):
        prev, cur = res.fitness[g - 1], res.populations[g]
        top = [res.populations[g - 1][i] for i in S.ranking(prev)[:3]]
        assert cur[:3] == top


@pytest.mark.parametrize("seed", [0, 1, 2, 3, 4])
def test_search_reaches_brute_force_optimum(seed):
    """C(10, 3) = 120 schedules with distinct fitness: the search finds the
    brute-force maximum."""
    N, K = 10, 3
    f = _table_fitness(N * 7, seed + 100)
    tab = {s: f(tuple(p * 7 + (p * p) % 7 for p in s)) for s in itertools.combinations(range(N), K)}
    opt = max(tab, key=tab.get)
    cfg = S.GAConfig(K=K, pop_size=12, n_elite=4, max_generations=25, n_guided=0, mutation_rate=0.2,
                     seed=seed)
    res = S.search(cfg, N, lambda batch: [tab[s] for s in batch])
    assert res.best == opt


def test_early_stopping_eq8_eq9():
    """Candidates reaching q_base in the quick evaluation get one formal
    evaluation each, best first; the first passing Eq. 9 ends the search."""
    N, K = 30, 4
    f = _table_fitness(N, 3)
    quick_vals = {}

    def quick(batch):
        out = []
        for s in batch:
            v = 1.0 if f(s) > 2.6 else 0.5
            quick_vals[s] = v
            out.append(v)
        return out

    formal_calls = []

    def formal(s):
        formal_calls.append(s)
        return 0.9 if len(formal_calls) >= 3 else 0.7     # the first two fail Eq. 9

    cfg = S.GAConfig(K=K, pop_size=10, n_elite=3, max_generations=30, n_guided=0, seed=9)
    res = S.search(cfg, N, quick, formal=formal, q_base=1.0, delta_acc=0.15)
    assert res.accepted and res.best == formal_calls[-1] and res.best_formal == 0.9
    assert len(formal_calls) == 3 == res.formal_evaluations == len(set(formal_calls))
    assert all(quick_vals[s] >= 1.0 for s in formal_calls)
    g = res.generations - 1
    assert res.best in res.populations[g]
    # no formal evaluation before the first generation holding a qualifying candidate
    first = min(i for i, fs in enumerate(res.fitness) if max(fs) >= 1.0)
    assert res.generations - 1 >= first
    # never accepted: runs every generation and returns the best of the last one
    res2 = S.search(cfg, N, quick, formal=lambda s: 0.0, q_base=1.0, delta_acc=0.15)
    assert not res2.accepted and res2.generations == 30
    assert res2.best == res2.populations[-1][S.ranking(res2.fitness[-1])[0]]


def test_success_rate_closed_form():
    full = np.zeros((4, 3, 2))
    cached = full.copy()
    cached[1, 0, 0] = 0.5
    cached[2, 2, 1] = -0.1
    cached[3, 1, 1] = 0.1 + 1e-6
    assert S.success_rate(full, full, 0.0) == 1.0
    assert S.success_rate(cached, full, 0.1) == 0.5
    assert S.success_rate(cached, full, 0.5) == 1.0
