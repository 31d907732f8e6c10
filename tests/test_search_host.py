"""The library's schedule search on the host (evo_ga_initial_population,
evo_ga_next_generation, evo_ga_search) against the oracle of Sec. 3.2 /
Eq. 8-9, bit for bit: same populations, same fitness, same result, on the
same seeds and the same (host) fitness functions."""
import numpy as np
import pytest

from oracle import evo_redundancy as R
from oracle import evo_search as S
from paper_2607_20293_amd import evo


def _cfgs(K, **kw):
    return S.GAConfig(K=K, **kw), evo.GAConfig.make(K, **kw)


def _probs(rows, T, seed):
    d = np.random.default_rng(seed).random((rows, T)) ** 2
    return R.guided_probabilities(d, 0.05, 2.0)


@pytest.mark.parametrize("rows,T,K,n_guided,seed", [(24, 100, 240, 15, 0), (6, 10, 20, 3, 7), (8, 100, 80, 30, 3),
                                                   (5, 7, 35, 0, 2**63 + 5)])
def test_initial_population_matches_oracle(rows, T, K, n_guided, seed):
    oc, lc = _cfgs(K, pop_size=30, n_guided=n_guided, seed=seed)
    p = _probs(rows, T, seed % 1000)
    want = np.array(S.initial_population(oc, rows * T, p if n_guided else None), np.int32)
    got = evo.ga_initial_population(lc, rows, T, p if n_guided else None)
    assert np.array_equal(got, want)


def _fitness_with_ties(N, seed):
    """Integer-valued fitness (exact in fp64) with many ties."""
    tab = np.random.default_rng(seed).integers(0, 5, N)
    return lambda sch: float(int(tab[list(sch)].sum()) % 11) / 10.0


@pytest.mark.parametrize("rows,T,K,tour,mut,elite", [(24, 100, 240, 2, 0.05, 10), (6, 10, 20, 3, 0.3, 4),
                                                     (4, 6, 23, 1, 1.0, 0), (3, 5, 2, 4, 0.0, 30)])
def test_generations_match_oracle(rows, T, K, tour, mut, elite):
    N = rows * T
    oc, lc = _cfgs(K, pop_size=30, n_elite=elite, tournament=tour, mutation_rate=mut, n_guided=0, seed=17)
    f = _fitness_with_ties(N, 5)
    pop = [tuple(x) for x in evo.ga_initial_population(lc, rows, T)]
    assert pop == S.initial_population(oc, N)
    for g in range(1, 12):
        fit = [f(s) for s in pop]
        want = S.next_generation(oc, N, g, pop, fit)
        got = evo.ga_next_generation(lc, rows, T, g, np.array(pop, np.int32), np.array(fit))
        assert [tuple(x) for x in got] == want, g
        pop = want


@pytest.mark.parametrize("early", [False, True])
def test_search_loop_matches_oracle(early):
    rows, T, K = 24, 100, 240
    N = rows * T
    p = _probs(rows, T, 9)
    oc, lc = _cfgs(K, n_guided=15, seed=123)
    tab = np.random.default_rng(4).random(N)

    def quick(batch):
        return [float(np.floor(8 * tab[list(s)].mean() * 3) / 8) for s in batch]

    thr = 1.5

    def formal(s):
        return float(tab[list(s)].mean() * 3 > thr)

    want = S.search(oc, N, quick, probs=p, formal=formal if early else None, q_base=0.75, delta_acc=0.0)
    got = evo.ga_search(lc, rows, T, lambda b: quick([tuple(x) for x in b]),
                        (lambda s: formal(tuple(s))) if early else None, probs=p, q_base=0.75, delta_acc=0.0)
    assert got["generations"] == want.generations
    assert got["evaluations"] == want.evaluations and got["memo_hits"] == want.memo_hits
    assert got["formal_evaluations"] == want.formal_evaluations
    assert bool(got["accepted"]) == want.accepted
    assert tuple(got["best"]) == want.best and got["best_quick"] == want.best_quick
    if want.best_formal is None:
        assert np.isnan(got["best_formal"])
    else:
        assert got["best_formal"] == want.best_formal
    for g in range(want.generations):
        assert [tuple(x) for x in got["populations"][g]] == want.populations[g]
        assert list(got["fitness"][g]) == want.fitness[g]


def test_callback_error_and_invalid_configs():
    lc = evo.GAConfig.make(4, pop_size=6, n_elite=2, max_generations=3, n_guided=0)
    with pytest.raises(ZeroDivisionError):
        evo.ga_search(lc, 2, 5, lambda b: [1 / 0 for _ in b])
    for bad in (dict(K=0), dict(K=11), dict(pop_size=0), dict(n_elite=7), dict(max_generations=0),
                dict(tournament=0), dict(n_guided=7), dict(mutation_rate=1.5)):
        kw = dict(K=4, pop_size=6, n_elite=2, max_generations=3, n_guided=0)
        kw.update(bad)
        with pytest.raises(evo.EvoError):
            evo.ga_initial_population(evo.GAConfig.make(**kw), 2, 5)
    with pytest.raises(evo.EvoError, match="2\\^28"):
        evo.ga_initial_population(evo.GAConfig.make(1 << 24, pop_size=30, n_guided=0), 1 << 12, 1 << 12)
    with pytest.raises(evo.EvoError, match="probabilities"):
        evo.ga_initial_population(evo.GAConfig.make(4, pop_size=6, n_elite=2, n_guided=2), 2, 5)
    p = np.zeros((2, 5))
    p[0, :3] = 1 / 3
    with pytest.raises(evo.EvoError, match="exceeds"):
        evo.ga_initial_population(evo.GAConfig.make(4, pop_size=6, n_elite=2, n_guided=2), 2, 5, p)
    pop = evo.ga_initial_population(lc, 2, 5)
    bad = pop.copy()
    bad[0, :2] = bad[0, 1::-1]
    with pytest.raises(evo.EvoError, match="sorted"):
        evo.ga_next_generation(lc, 2, 5, 1, bad, np.zeros(6))
    with pytest.raises(evo.EvoError, match="NaN"):
        evo.ga_next_generation(lc, 2, 5, 1, pop, np.full(6, np.nan))
