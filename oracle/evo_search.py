"""CPU oracle of EVO's schedule search (arXiv 2607.20293, Sec. 3.2
"evolutionary procedure" with Eq. 4 and Eq. 5, Sec. 3.3 "Redundancy-aware
Initialization" and "Target-conditioned Early Stopping" with Eq. 7, Eq. 8 and
Eq. 9, population settings of Sec. 4.1).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
baseline may import this module.  It shares no code with the HIP library and
imports nothing from the product package.

What it computes:

* A candidate is a schedule S: exactly K distinct positions of the
  block x step lattice (Eq. 5), held as the sorted flat indices p = b*T + t.
  The sorted tuple is its canonical signature.
* Fitness (Eq. 4) is supplied by the caller (the rollout success rate in the
  paper; a synthetic stand-in in the tests).  Evaluated schedules are
  memoised by signature and never evaluated twice.
* Initial population (Sec. 3.3): n_guided individuals drawn from Eq. 7's
  distribution (K positions without replacement), the rest uniformly random
  K-subsets of the lattice.
* One generation (Sec. 3.2): the n_elite best individuals carry over
  (elitism); each other child takes two parents by tournament selection,
  set-level crossover of the parents, mutation that resamples positions from
  the full lattice, and repair back to exactly K unique positions.
* Early stopping (Eq. 8, Eq. 9): after a generation is evaluated, candidates
  whose quick score reaches q_base get a formal evaluation (each signature at
  most once), best first; the first with formal score >= q_base - delta_acc
  is accepted and the search ends.

Readings where the paper is silent (listed in the design notes):
* Randomness comes from the counter-based generator Philox4x64-10 (Salmon,
  Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011),
  keyed by (seed, 0) with counter (generation, purpose << 32 | slot, index, 0);
  the first output word is used.  Every draw is addressed by the decision it
  makes (an individual or child, and a rank or draw number within it).
* Uniform in (0, 1): ((w >> 12) + 1/2) * 2^-52 (exact in fp64).  Uniform integer in [0, n):
  ((w >> 32) * n) >> 32.  Bernoulli(1/2): the top bit of w.
* Random individuals: uniform K-subsets, by `fill` from the empty set:
  draw j adds position below(word(j), N) unless present.
* Tournament: `tournament` entrants drawn with replacement from the
  population; the highest fitness wins, ties to the lower population index.
* Crossover (always applied): positions in both parents are kept; each
  position in exactly one parent is kept with probability 1/2 (one bit of a
  word per position, by rank).
* Mutation: each position of the child is, with probability mutation_rate
  (a 32-bit half-word against floor(rate * 2^32)), replaced by a position
  drawn uniformly from the whole lattice.
* Repair: duplicates merge (sets); a surplus is removed one uniformly chosen
  element at a time; a shortfall is completed by uniform draws of positions
  not yet present.
* Ranking: fitness descending, ties to the lower population index.  The next
  population is the n_elite best in that order followed by the children.
* max_generations counts evaluated populations, the initial one included.
  Without acceptance the search returns the best individual of the last
  population.

Every function is pinned in tests/test_search_pins.py against numpy's Philox
generator, closed forms, distributional laws and brute force.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import evo_redundancy as R

MASK64 = (1 << 64) - 1
_PHILOX_MUL = (0xD2E7470EE14C6C93, 0xCA5A826395121157)
_PHILOX_WEYL = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)

INIT, TOUR, CROSS, MUT, MUTPOS, DROP, FILL = 1, 2, 3, 4, 5, 6, 7


def philox4x64(ctr: Sequence[int], key: Sequence[int]) -> List[int]:
    """Philox4x64 with 10 rounds (Salmon et al. 2011): four 64-bit counter
    words, two key words; each round multiplies words 0 and 2 by the two
    constants, recombines high/low halves with the key, and the key advances
    by the Weyl constants between rounds."""
    c = [int(x) & MASK64 for x in ctr]
    k = [int(x) & MASK64 for x in key]
    for rnd in range(10):
        p0 = _PHILOX_MUL[0] * c[0]
        p1 = _PHILOX_MUL[1] * c[2]
        hi0, lo0 = p0 >> 64, p0 & MASK64
        hi1, lo1 = p1 >> 64, p1 & MASK64
        c = [hi1 ^ c[1] ^ k[0], lo1, hi0 ^ c[3] ^ k[1], lo0]
        if rnd < 9:
            k = [(k[0] + _PHILOX_WEYL[0]) & MASK64, (k[1] + _PHILOX_WEYL[1]) & MASK64]
    return c


def word(seed: int, gen: int, purpose: int, slot: int, index: int) -> int:
    return philox4x64((gen, (purpose << 32) | slot, index, 0), (seed, 0))[0]


def unit_interval(w: int) -> float:
    return ((w >> 12) + 0.5) * 2.0 ** -52


def below(w: int, n: int) -> int:
    return ((w >> 32) * n) >> 32


@dataclass
class GAConfig:
    K: int
    pop_size: int = 30
    n_elite: int = 10
    max_generations: int = 30
    tournament: int = 2
    n_guided: int = 15
    mutation_rate: float = 0.05
    seed: int = 0


def fill(seed: int, gen: int, purpose: int, slot: int, s: set, K: int, N: int) -> set:
    """Uniform completion to K distinct positions: draw j = 0, 1, ... adds
    below(word(j), N) unless present.  After 64 N draws (never reached in
    practice) the missing positions are added in ascending order."""
    out = set(s)
    j = 0
    while len(out) < K and j < 64 * N:
        out.add(below(word(seed, gen, purpose, slot, j), N))
        j += 1
    p = 0
    while len(out) < K:
        out.add(p)
        p += 1
    return out


def random_individual(cfg: GAConfig, N: int, i: int) -> Tuple[int, ...]:
    return tuple(sorted(fill(cfg.seed, 0, INIT, i, set(), cfg.K, N)))


def guided_individual(cfg: GAConfig, probs: np.ndarray, i: int) -> Tuple[int, ...]:
    rows, T = probs.shape
    u = np.array([unit_interval(word(cfg.seed, 0, INIT, i, p)) for p in range(rows * T)]).reshape(rows, T)
    pairs = R.guided_sample(probs, cfg.K, u)
    return tuple(int(b) * T + int(t) for b, t in pairs)


def initial_population(cfg: GAConfig, N: int, probs: Optional[np.ndarray] = None) -> List[Tuple[int, ...]]:
    """Sec. 3.3: n_guided individuals from Eq. 7 (probs [rows][T]), the rest
    uniform random."""
    if cfg.n_guided > 0:
        assert probs is not None and probs.size == N
    return [guided_individual(cfg, probs, i) if i < cfg.n_guided else random_individual(cfg, N, i)
            for i in range(cfg.pop_size)]


def ranking(fit: Sequence[float]) -> List[int]:
    return sorted(range(len(fit)), key=lambda i: (-fit[i], i))


def tournament(cfg: GAConfig, gen: int, child: int, parent: int, fit: Sequence[float]) -> int:
    best = -1
    for e in range(cfg.tournament):
        idx = below(word(cfg.seed, gen, TOUR, child, parent * cfg.tournament + e), len(fit))
        if best < 0 or fit[idx] > fit[best] or (fit[idx] == fit[best] and idx < best):
            best = idx
    return best


def crossover(cfg: GAConfig, gen: int, child: int, a: Sequence[int], b: Sequence[int]) -> set:
    """Positions in both parents are kept; the r-th position (ascending) of
    those in exactly one parent is kept on bit r mod 64 of word(r div 64)."""
    A, B = set(a), set(b)
    out = A & B
    for r, p in enumerate(sorted(A ^ B)):
        if (word(cfg.seed, gen, CROSS, child, r // 64) >> (r % 64)) & 1:
            out.add(p)
    return out


def mutate(cfg: GAConfig, gen: int, child: int, s: set, N: int) -> set:
    """The r-th position (ascending) is replaced, when the 32-bit half
    r mod 2 of word(r div 2) is below floor(mutation_rate * 2^32), by
    below(word'(r), N) (purpose MUTPOS)."""
    thr = int(cfg.mutation_rate * 2.0 ** 32)
    out = set()
    for r, q in enumerate(sorted(s)):
        h = (word(cfg.seed, gen, MUT, child, r // 2) >> (32 * (r % 2))) & 0xFFFFFFFF
        out.add(below(word(cfg.seed, gen, MUTPOS, child, r), N) if h < thr else q)
    return out


def repair(cfg: GAConfig, gen: int, child: int, s: set, N: int) -> Tuple[int, ...]:
    """Back to exactly K: a surplus loses, one at a time, the element at
    index below(word(j), size) of the ascending list (purpose DROP, draw
    j = 0, 1, ...); a shortfall is completed by `fill` (purpose FILL)."""
    K = cfg.K
    ss = sorted(s)
    j = 0
    while len(ss) > K:
        del ss[below(word(cfg.seed, gen, DROP, child, j), len(ss))]
        j += 1
    if len(ss) < K:
        ss = sorted(fill(cfg.seed, gen, FILL, child, set(ss), K, N))
    return tuple(ss)


def make_child(cfg: GAConfig, gen: int, child: int, pop: Sequence[Sequence[int]], fit: Sequence[float],
               N: int) -> Tuple[int, ...]:
    a = tournament(cfg, gen, child, 0, fit)
    b = tournament(cfg, gen, child, 1, fit)
    s = crossover(cfg, gen, child, pop[a], pop[b])
    s = mutate(cfg, gen, child, s, N)
    return repair(cfg, gen, child, s, N)


def next_generation(cfg: GAConfig, N: int, gen: int, pop: Sequence[Sequence[int]],
                    fit: Sequence[float]) -> List[Tuple[int, ...]]:
    """Population `gen` (>= 1) from population gen-1 and its fitness."""
    order = ranking(fit)
    elites = [tuple(pop[i]) for i in order[:cfg.n_elite]]
    children = [make_child(cfg, gen, c, pop, fit, N) for c in range(cfg.pop_size - cfg.n_elite)]
    return elites + children


@dataclass
class SearchResult:
    best: Tuple[int, ...]
    best_quick: float
    best_formal: Optional[float]
    accepted: bool
    generations: int
    evaluations: int
    memo_hits: int
    formal_evaluations: int
    populations: List[List[Tuple[int, ...]]]
    fitness: List[List[float]]


def search(cfg: GAConfig, N: int, quick: Callable[[List[Tuple[int, ...]]], Sequence[float]],
           probs: Optional[np.ndarray] = None,
           formal: Optional[Callable[[Tuple[int, ...]], float]] = None,
           q_base: float = 1.0, delta_acc: float = 0.0) -> SearchResult:
    """Sec. 3.2 with Eq. 8 / Eq. 9.  quick(list of schedules) returns their
    quick fitness (called only for signatures not evaluated before, in
    population order); formal(schedule) the formal score (None: no early
    stopping)."""
    memo: Dict[Tuple[int, ...], float] = {}
    formal_memo: Dict[Tuple[int, ...], float] = {}
    pops, fits = [], []
    evaluations = memo_hits = 0
    pop = initial_population(cfg, N, probs)
    fit: List[float] = []
    for gen in range(cfg.max_generations):
        if gen > 0:
            pop = next_generation(cfg, N, gen, pop, fit)
        new: List[Tuple[int, ...]] = []
        for s in pop:
            if s not in memo and s not in new:
                new.append(s)
        if new:
            vals = list(quick(new))
            assert len(vals) == len(new)
            for s, v in zip(new, vals):
                memo[s] = float(v)
        evaluations += len(new)
        memo_hits += len(pop) - len(new)
        fit = [memo[s] for s in pop]
        pops.append(list(pop))
        fits.append(list(fit))
        if formal is not None:
            for i in ranking(fit):
                s = pop[i]
                if fit[i] >= q_base and s not in formal_memo:
                    formal_memo[s] = float(formal(s))
                    if formal_memo[s] >= q_base - delta_acc:
                        return SearchResult(s, fit[i], formal_memo[s], True, gen + 1, evaluations, memo_hits,
                                            len(formal_memo), pops, fits)
    i = ranking(fit)[0]
    return SearchResult(pop[i], fit[i], formal_memo.get(pop[i]), False, cfg.max_generations, evaluations,
                        memo_hits, len(formal_memo), pops, fits)


def success_rate(cached: np.ndarray, full: np.ndarray, tau: float) -> float:
    """Synthetic stand-in for Eq. 4's success indicator: episode n succeeds
    when the cached action chunk stays within tau (max-abs) of the uncached
    chunk of the same observation and noise.  The deviation is formed in
    fp64 and the decision taken in fp32, the precision of the GPU path."""
    dev = np.max(np.abs(np.asarray(cached, np.float64) - np.asarray(full, np.float64)), axis=(1, 2))
    return float(np.count_nonzero(dev.astype(np.float32) <= np.float32(tau))) / dev.shape[0]
