"""evo_denoise_noalloc (working data in the device's fixed scratch array)
against evo_denoise on the same policy and inputs, through the C ABI: two
calls in a row, the second with a smaller batch, on the team variant, on
one-workgroup tiles and on two-sample tiles; bookkeeping equal; the call
captured into a HIP graph and replayed; a batch too large for the array
refused before anything runs."""
import numpy as np
import pytest

from oracle import evo_oracle as O
from paper_2607_20293_amd import evo
from paper_2607_20293_amd import inputs as I
from tests.gpu_util import compare, device, say

pytestmark = pytest.mark.gpu


def _policy(shape, wts, dtype, max_batch, n_sched, env=None):
    import os
    old = {k: os.environ.get(k) for k in (env or {})}
    os.environ.update(env or {})
    try:
        return evo.Policy(shape, wts, dtype=dtype, max_batch=max_batch, max_schedules=n_sched)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def _both(pol, shape, obs, noise, ids):
    import torch
    dev = device()
    o = torch.from_numpy(np.ascontiguousarray(obs)).to(dev)
    n = torch.from_numpy(np.ascontiguousarray(noise)).to(dev)
    B = obs.shape[0]
    ref = pol.denoise(o, n, ids)
    pol.synchronize()
    st_ref = pol.stats()
    out = torch.full((B, shape.horizon, shape.action_dim), float("nan"), device=dev)
    pol.denoise_noalloc(o, n, ids, out)
    pol.synchronize()
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), ref.cpu().numpy().astype(np.float64), pol.stats(), st_ref


@pytest.mark.parametrize("case", ["team", "single", "two_sample"])
def test_noalloc_matches_denoise_twice(case):
    if case == "two_sample":
        s, dtype, env, batches = I.TINY, "fp32", None, (9, 4)
    elif case == "team":
        s, dtype, env, batches = I.PUSHT, "bf16", None, (64, 5)
    else:
        s, dtype, env, batches = I.PUSHT, "bf16", {"EVO_TEAM": "0"}, (100, 7)
    B0 = batches[0]
    wts = I.make_weights(s, 5, "perturbed")
    rng = np.random.default_rng([5, 3])
    lats = [I.lattice_bernoulli(s.n_layers, s.n_steps, p, rng) for p in (0.15, 0.4, 0.8)]
    pol = _policy(s, wts, dtype, B0, 3, env)
    for j, lt in enumerate(lats):
        pol.set_schedule(j, lt, O.GRAN_LAYER)
    for k, B in enumerate(batches):
        say(f"[gpu] noalloc {case}: call {k} batch {B}")
        obs, noise = I.make_obs(s, B, 10 + k), I.make_noise(s, B, 10 + k)
        ids = rng.integers(0, 3, B).astype(np.int32)
        got, ref, st, st_ref = _both(pol, s, obs, noise, ids)
        assert np.all(np.isfinite(got))
        compare(got, ref, dtype, f"noalloc vs denoise ({case}, batch {B})")
        say(f"  bitwise equal: {np.array_equal(got, ref)}")
        for key in ("refreshes_requested", "refreshes_effective", "flops_cacheable", "flops_always",
                    "flops_full", "flops_kernel", "n_tiles", "n_workgroups", "weight_bytes"):
            assert st[key] == st_ref[key], key
        with pytest.raises(evo.EvoError) as e:
            pol.read_cache(0, 0)
        assert e.value.code == -2   # EVO_E_STATE: the cache lives in the scratch array
    pol.close()


@pytest.mark.parametrize("case", ["team", "two_sample"])
def test_noalloc_captured_in_a_graph_replays(case):
    """evo_denoise_noalloc enqueued while a stream is captured into a HIP
    graph: three replays, with eager calls of the same policy and
    synchronisations between them, each bitwise equal to the eager result
    (the replays read the plan that the policy's pinned staging buffers hold
    when they run; the eager calls in between restage the same bytes)."""
    import torch
    if case == "team":
        s, dtype, B = I.PUSHT, "bf16", 2
    else:
        s, dtype, B = I.TINY, "fp32", 9
    wts = I.make_weights(s, 6, "perturbed")
    rng = np.random.default_rng([6, 3])
    lats = [I.lattice_bernoulli(s.n_layers, s.n_steps, p, rng) for p in (0.2, 0.5)]
    pol = _policy(s, wts, dtype, B, 2)
    for j, lt in enumerate(lats):
        pol.set_schedule(j, lt, O.GRAN_LAYER)
    dev = device()
    obs = torch.from_numpy(np.ascontiguousarray(I.make_obs(s, B, 21))).to(dev)
    noise = torch.from_numpy(np.ascontiguousarray(I.make_noise(s, B, 21))).to(dev)
    ids = rng.integers(0, 2, B).astype(np.int32)
    shape = (B, s.horizon, s.action_dim)
    ref = torch.zeros(shape, device=dev)
    pol.denoise_noalloc(obs, noise, ids, ref)
    pol.synchronize()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    out = torch.zeros(shape, device=dev)
    g = torch.cuda.CUDAGraph()
    say(f"[gpu] noalloc graph capture ({case}, batch {B})")
    with torch.cuda.graph(g, stream=side):
        pol.denoise_noalloc(obs, noise, ids, out, stream=side)
    for rep in range(3):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {rep}"
        eager = torch.zeros(shape, device=dev)
        pol.denoise_noalloc(obs, noise, ids, eager)
        pol.synchronize()
        torch.cuda.synchronize()
        assert torch.equal(eager, ref), f"eager call after replay {rep}"
    del g
    pol.close()


def test_noalloc_refuses_a_batch_beyond_the_scratch():
    import torch
    s = I.PUSHT
    B = 240   # one-sample tiles, fp16 caches: about 200 samples of this policy fit
    pol = _policy(s, I.make_weights(s, 0), "bf16", B, 1, {"EVO_TEAM": "0"})
    pol.set_schedule(0, I.make_lattice("dirichlet", s.n_layers, s.n_steps, 0.25, 0), O.GRAN_LAYER)
    dev = device()
    obs = torch.from_numpy(I.make_obs(s, B, 0)).to(dev)
    noise = torch.from_numpy(I.make_noise(s, B, 0)).to(dev)
    out = torch.zeros((B, s.horizon, s.action_dim), device=dev)
    with pytest.raises(evo.EvoError) as e:
        pol.denoise_noalloc(obs, noise, np.zeros(B, np.int32), out)
    assert e.value.code == -5 and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert float(out.abs().max()) == 0.0       # nothing ran
    assert evo.lib().evo_noalloc_scratch_bytes() == 64 << 20
    pol.close()
