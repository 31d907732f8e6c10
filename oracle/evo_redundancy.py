"""CPU fp64 oracle of EVO's redundancy-aware initialisation (arXiv
2607.20293, Sec. 3.3 "Redundancy-aware Initialization", Eq. 6 and Eq. 7).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
baseline may import this module.  It shares no code with the HIP library and
imports nothing from the product package.

What it computes:

* Activations (Sec. 3.3): a_{r,b,t}, the residual of cacheable unit b at
  denoising step t of action query r, collected from the uncached policy
  (every unit evaluated at every step).  Here a query is one sample of a
  batch (its own observation and noise); the activation is the unit's
  [H][d] residual flattened to one vector.
* Dissimilarity score (Eq. 6): for every unit b and step t, the mean over
  the other steps t' of one minus the cosine similarity between a_{r,b,t}
  and a_{r,b,t'}, averaged over the queries r.
* Guided sampling (Eq. 7): the scores are normalised to w in [0, 1] and a
  position (b, t) is drawn with probability proportional to (eps + w)^gamma.

Readings where the paper is silent (listed in the design notes):
* a zero activation vector has no direction; its cosine with anything is
  taken as 0 (dissimilarity 1);
* the normalisation of d into w is min-max over all positions (all zeros if
  d is constant);
* eps and gamma are parameters (the paper gives no values);
* an initial individual takes K distinct positions, drawn one after another
  without replacement from Eq. 7's distribution.  This is computed with the
  Gumbel-top-K construction (key = log p + Gumbel noise from a given uniform
  per position; the K largest keys, ties to the lower flat index), which has
  exactly that distribution; the uniforms are an input.

Every function is pinned in tests/test_redundancy_pins.py against closed
forms, special cases, a library routine and brute force.
"""
from __future__ import annotations

import numpy as np

from . import evo_oracle as O


def collect_activations(shape, P, obs: np.ndarray, noise: np.ndarray, clip: bool = True) -> np.ndarray:
    """a[r][b][t][:] for r < n queries (Sec. 3.3): the uncached policy's unit
    residuals, flattened [H*d].  P: fp64 parameters (prepare_params)."""
    tr = {}
    O.denoise_group(shape, P, obs, noise, np.ones((3 * shape.n_layers, shape.n_steps), bool), clip=clip,
                    cache=False, trace=tr)
    r = tr["r"]                                   # [T][U][n][H][d]
    T, U, n = r.shape[0], r.shape[1], r.shape[2]
    return np.ascontiguousarray(r.transpose(2, 1, 0, 3, 4).reshape(n, U, T, -1))


def cosine(u: np.ndarray, v: np.ndarray) -> float:
    """<u, v> / (|u| |v|); 0 when either vector is zero (reading)."""
    nu = float(np.sqrt(np.dot(u, u)))
    nv = float(np.sqrt(np.dot(v, v)))
    if nu == 0.0 or nv == 0.0:
        return 0.0
    return float(np.dot(u, v)) / (nu * nv)


def redundancy_scores(acts: np.ndarray) -> np.ndarray:
    """Eq. 6: d[b][t] = E_r[ 1/(T-1) sum_{t' != t} (1 - cos(a_{r,b,t}, a_{r,b,t'})) ].
    acts: [R][U][T][V] (any float type, computed in fp64)."""
    a = np.asarray(acts, np.float64)
    R, U, T = a.shape[0], a.shape[1], a.shape[2]
    d = np.zeros((U, T))
    for b in range(U):
        for t in range(T):
            tot = 0.0
            for r in range(R):
                s = 0.0
                for t2 in range(T):
                    if t2 != t:
                        s += 1.0 - cosine(a[r, b, t], a[r, b, t2])
                tot += s / (T - 1)
            d[b, t] = tot / R
    return d


def normalize_scores(d: np.ndarray) -> np.ndarray:
    """Min-max normalisation of the scores into w in [0, 1] (reading)."""
    d = np.asarray(d, np.float64)
    lo, hi = float(d.min()), float(d.max())
    if hi <= lo:
        return np.zeros_like(d)
    return (d - lo) / (hi - lo)


def guided_probabilities(d: np.ndarray, eps: float, gamma: float) -> np.ndarray:
    """Eq. 7: p[b][t] = (eps + w[b][t])^gamma / sum (eps + w)^gamma, w the
    normalised scores."""
    w = normalize_scores(d)
    q = (eps + w) ** gamma
    return q / q.sum()


def guided_sample(p: np.ndarray, K: int, u: np.ndarray) -> np.ndarray:
    """K distinct positions drawn without replacement from p (flattened
    [rows][T]), Gumbel-top-K with the uniforms u (same shape, in (0, 1)).
    Returns int32 pairs [K][2] = (row, step), sorted by flat index."""
    p = np.asarray(p, np.float64)
    rows, T = p.shape
    flat_p = p.reshape(-1)
    if K < 0 or K > int(np.count_nonzero(flat_p > 0.0)):
        raise ValueError("K must not exceed the number of positions with non-zero probability")
    flat_u = np.asarray(u, np.float64).reshape(-1)
    keys = []
    for i in range(flat_p.size):
        if flat_p[i] > 0.0:
            keys.append((np.log(flat_p[i]) - np.log(-np.log(flat_u[i])), -i))
        else:
            keys.append((-np.inf, -i))
    order = sorted(range(flat_p.size), key=lambda i: keys[i], reverse=True)
    chosen = sorted(order[:K])
    return np.array([[i // T, i % T] for i in chosen], np.int32).reshape(-1, 2)
