"""Pins of the redundancy oracle (Sec. 3.3, Eq. 6 and Eq. 7) against closed
forms, special cases, scipy's cosine distance and brute-force enumeration."""
import itertools

import numpy as np
import pytest
from scipy.spatial.distance import cdist

from oracle import evo_oracle as O
from oracle import evo_redundancy as RD
from paper_2607_20293_amd import inputs as I


def test_identical_activations_have_zero_dissimilarity():
    v = np.random.default_rng(0).standard_normal(12)
    acts = np.broadcast_to(v, (2, 3, 5, 12)).copy()
    assert np.allclose(RD.redundancy_scores(acts), 0.0, atol=1e-15)


def test_orthogonal_activations_have_unit_dissimilarity():
    T = 6
    acts = np.zeros((1, 2, T, T))
    for t in range(T):
        acts[0, :, t, t] = 1.0 + t          # orthogonal directions, any length
    assert np.allclose(RD.redundancy_scores(acts), 1.0)


def test_two_steps_closed_form():
    # T = 2: d[b][0] = d[b][1] = 1 - cos(a0, a1); antiparallel gives 2
    a0 = np.array([1.0, 2.0, 2.0])
    a1 = np.array([2.0, -1.0, 0.0])
    acts = np.stack([a0, a1])[None, None]
    c = (1 * 2 + 2 * -1 + 2 * 0) / (3.0 * np.sqrt(5.0))
    assert np.allclose(RD.redundancy_scores(acts), 1.0 - c)
    acts2 = np.stack([a0, -a0])[None, None]
    assert np.allclose(RD.redundancy_scores(acts2), 2.0)


def test_three_steps_hand_computed():
    e = np.eye(3)
    acts = np.stack([e[0], e[0] + e[1], e[1]])[None, None]      # 45 degrees apart, then orthogonal
    c = 1.0 / np.sqrt(2.0)
    want = np.array([(1 - c + 1 - 0) / 2, (1 - c + 1 - c) / 2, (1 - 0 + 1 - c) / 2])
    assert np.allclose(RD.redundancy_scores(acts)[0], want)


def test_scale_invariance_and_rollout_mean():
    rng = np.random.default_rng(1)
    acts = rng.standard_normal((3, 2, 7, 10))
    scales = rng.uniform(0.1, 10.0, size=(3, 2, 7, 1))
    assert np.allclose(RD.redundancy_scores(acts), RD.redundancy_scores(acts * scales))
    per_r = np.stack([RD.redundancy_scores(acts[r:r + 1]) for r in range(3)])
    assert np.allclose(RD.redundancy_scores(acts), per_r.mean(axis=0))


def test_matches_scipy_cosine_distance():
    rng = np.random.default_rng(2)
    acts = rng.standard_normal((2, 3, 9, 16))
    want = np.zeros((3, 9))
    for r in range(2):
        for b in range(3):
            D = cdist(acts[r, b], acts[r, b], "cosine")         # 1 - cos, zero diagonal
            want[b] += D.sum(axis=1) / 8
    want /= 2
    assert np.allclose(RD.redundancy_scores(acts), want, atol=1e-12)


def test_zero_vector_reading():
    acts = np.zeros((1, 1, 3, 4))
    acts[0, 0, 1] = [1.0, 0.0, 0.0, 0.0]
    acts[0, 0, 2] = [1.0, 0.0, 0.0, 0.0]
    # step 0 is zero: its cosines count as 0 -> dissimilarity 1 to both others
    assert np.allclose(RD.redundancy_scores(acts)[0], [1.0, 0.5, 0.5])


def test_guided_probabilities():
    rng = np.random.default_rng(3)
    d = rng.uniform(0.2, 0.9, size=(4, 5))
    p = RD.guided_probabilities(d, 0.05, 2.0)
    assert abs(p.sum() - 1.0) < 1e-15 and (p > 0).all()
    w = (d - d.min()) / (d.max() - d.min())
    i, j = np.unravel_index(np.argmax(d), d.shape), np.unravel_index(np.argmin(d), d.shape)
    assert np.isclose(p[i] / p[j], ((0.05 + 1.0) / 0.05) ** 2.0)     # normalised extremes are 1 and 0
    assert np.allclose(p, (0.05 + w) ** 2 / ((0.05 + w) ** 2).sum())
    assert np.allclose(RD.guided_probabilities(d, 0.3, 0.0), 1.0 / 20)    # gamma 0: uniform
    assert np.allclose(RD.guided_probabilities(np.full((2, 3), 0.7), 0.1, 3.0), 1.0 / 6)  # constant d
    order = np.argsort(d, axis=None)
    assert np.all(np.diff(p.reshape(-1)[order]) >= 0)                 # monotone in d


def test_guided_sample_support_and_uniqueness():
    rng = np.random.default_rng(4)
    p = np.zeros((3, 8))
    support = [(0, 1), (1, 7), (2, 0), (2, 5)]
    for i, (b, t) in enumerate(support):
        p[b, t] = (i + 1) / 10.0
    for s in range(20):
        u = rng.uniform(size=p.shape)
        got = RD.guided_sample(p, 4, u)
        assert sorted(map(tuple, got)) == sorted(support)            # K = support size: all of it
        got2 = RD.guided_sample(p, 2, u)
        assert len({tuple(x) for x in got2}) == 2 and all(tuple(x) in support for x in got2)
    with pytest.raises(ValueError):
        RD.guided_sample(p, 5, rng.uniform(size=p.shape))


def test_guided_sample_law_matches_sequential_draws():
    """Brute force on 4 positions, K = 2: the probability of each unordered
    pair under sequential sampling without replacement is
    p_i p_j / (1 - p_i) + p_j p_i / (1 - p_j); the Gumbel-top-K draws reproduce
    it."""
    p = np.array([[0.1, 0.2, 0.3, 0.4]])
    want = {}
    for i, j in itertools.combinations(range(4), 2):
        a, b = p[0, i], p[0, j]
        want[(i, j)] = a * b / (1 - a) + b * a / (1 - b)
    rng = np.random.default_rng(5)
    N = 40000
    cnt = dict.fromkeys(want, 0)
    for _ in range(N):
        got = RD.guided_sample(p, 2, rng.uniform(size=p.shape))
        cnt[(int(got[0, 1]), int(got[1, 1]))] += 1
    for key, pr in want.items():
        assert abs(cnt[key] / N - pr) < 4.5 * np.sqrt(pr * (1 - pr) / N), (key, cnt[key] / N, pr)


def test_collected_activations_are_the_uncached_residuals():
    """The uncached policy's trace equals the all-refresh cached run's trace
    (Eq. 1 with S = B x T), and step 0's first unit equals the residual
    computed directly."""
    s = I.TINY
    P = O.prepare_params(I.split_weights(s, I.make_weights(s, 0, "perturbed")), "fp32")
    obs, noise = I.make_obs(s, 2, 0), I.make_noise(s, 2, 0)
    acts = RD.collect_activations(s, P, obs, noise)
    assert acts.shape == (2, 3 * s.n_layers, s.n_steps, s.horizon * s.d_model)
    tr = {}
    O.denoise_group(s, P, obs, noise, np.ones((3 * s.n_layers, s.n_steps), bool), trace=tr)
    assert np.array_equal(acts, tr["r"].transpose(2, 1, 0, 3, 4).reshape(acts.shape))
    mem = np.concatenate([np.broadcast_to(O.sinusoid(s.n_steps - 1, s.d_model), (2, 1, s.d_model)),
                          np.asarray(obs, np.float64) @ P["W_obs"].T + P["b_obs"]], axis=1) + P["P_mem"]
    h = np.asarray(noise[0], np.float64) @ P["W_in"].T + P["b_in"] + P["P_act"]
    r0 = O.unit_residual(0, h, mem, P, s.n_heads)
    assert np.allclose(acts[:, 0, 0], r0.reshape(2, -1))
