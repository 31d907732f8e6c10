"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on
the same seeded inputs, plus the invariants of the cached loop that hold on
the device (determinism, per-query reset, sample independence, cache
contents).  Bars: fp32 max-abs <= 1e-4; bf16 normwise relative <= 3e-2;
bookkeeping bit-exact."""
import os

import numpy as np
import pytest

from oracle import evo_oracle as O
from paper_2607_20293_amd import evo
from paper_2607_20293_amd import inputs as I
from tests.conftest import printed_unit_lattice
from tests.gpu_util import check_stats, compare, device, load_stored, run_gpu, run_oracle, say

pytestmark = pytest.mark.gpu


def _policy(shape, weights, dtype, max_batch, max_sched, cold=O.COLD_COMPUTE, clip=True, team=True, env=None):
    """team=False creates the policy with the small-batch team variant
    switched off (EVO_TEAM=0 is read at creation); env: further variables
    set only while the policy is created."""
    device()
    env = dict(env or {})
    if not team:
        env["EVO_TEAM"] = "0"
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        return evo.Policy(shape, weights, dtype=dtype, max_batch=max_batch, max_schedules=max_sched,
                          cold_policy=cold, clip=clip)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def _case(name, shape, weights, obs, noise, lattices, ids, dtype, gran=O.GRAN_LAYER,
          cold=O.COLD_COMPUTE, samples=None, max_batch=None, clip=True, team=True, env=None):
    say(f"[gpu] {name}: dtype={dtype} batch={obs.shape[0]} schedules={len(lattices)} gran={gran} cold={cold} "
        f"team={team} env={env}")
    B = obs.shape[0]
    pol = _policy(shape, weights, dtype, max_batch or B, len(lattices), cold, clip, team, env)
    for j, lt in enumerate(lattices):
        pol.set_schedule(j, lt, gran)
    got, gst = run_gpu(pol, obs, noise, ids)
    ref, ost = run_oracle(shape, weights, obs, noise, lattices, ids, gran, cold, dtype, samples, clip)
    sel = got if samples is None else got[list(samples)]
    err = compare(sel, ref, dtype, name)
    check_stats(gst, ost)
    return pol, got, gst, err


# ---------------------------------------------------------------- workloads
def test_tiny_fp32_b1_config():
    w = I.WORKLOADS["tiny_fp32_b1"]
    inp = I.make_inputs(w)
    pol, *_ = _case("tiny_fp32_b1", w.shape, inp.weights, inp.obs, inp.noise, inp.lattices, inp.ids, "fp32")
    pol.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_tiny_perturbed_ragged_mixed(dtype):
    """batch 5 (two samples per tile -> a half-empty last tile), three
    schedules mixed within tiles, non-zero biases and LN affine."""
    s = I.TINY
    wts = I.make_weights(s, 1, "perturbed")
    obs, noise = I.make_obs(s, 5, 1), I.make_noise(s, 5, 1)
    rng = np.random.default_rng([1, 3])
    lats = [I.lattice_bernoulli(2, 10, p, rng) for p in (0.2, 0.5, 0.9)]
    ids = np.array([2, 0, 1, 0, 2], np.int32)
    pol, *_ = _case(f"tiny_{dtype}_mixed", s, wts, obs, noise, lats, ids, dtype)
    pol.close()


def test_tiny_wide_weights_fp32():
    """Larger weights: sharper attention and larger residuals."""
    s = I.TINY
    wts = I.make_weights(s, 2, "wide")
    obs, noise = I.make_obs(s, 2, 2), I.make_noise(s, 2, 2)
    lats = [I.lattice_bernoulli(2, 10, 0.5, np.random.default_rng(5))]
    pol, *_ = _case("tiny_wide", s, wts, obs, noise, lats, np.zeros(2, np.int32), "fp32")
    pol.close()


@pytest.mark.parametrize("name", ["pusht_fp32_b1_d25", "pusht_fp32_b1_all", "pusht_bf16_b1_d25",
                                  "pusht_bf16_b1_all"])
def test_pusht_b1(name):
    w = I.WORKLOADS[name]
    inp = I.make_inputs(w)
    pol, *_ = _case(name, w.shape, inp.weights, inp.obs, inp.noise, inp.lattices, inp.ids, w.dtype)
    pol.close()


@pytest.mark.parametrize("name", ["pusht_fp32_b1_d25", "pusht_bf16_b1_d25"])
def test_pusht_b1_single_workgroup(name):
    """The same batch-1 queries with the team variant switched off: one
    workgroup per tile."""
    w = I.WORKLOADS[name]
    inp = I.make_inputs(w)
    pol, got, gst, _ = _case(name + "_noteam", w.shape, inp.weights, inp.obs, inp.noise, inp.lattices, inp.ids,
                             w.dtype, team=False)
    assert gst["n_workgroups"] == gst["n_tiles"] == 1
    pol.close()


@pytest.mark.parametrize("size", [4, 2])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_team_variant_matches_single_workgroup(dtype, size):
    """Small batches run `size` workgroups per one-sample tile (self-
    attention heads and d_ff chunks split among them, partial residuals summed
    through memory; the folded cross-attention is evaluated whole by each;
    automatic choice: fp32 teams of 4 up to n_cu/4 samples, then teams of 2
    up to n_cu/2, bf16 teams of 2 up to n_cu/2; each size forced here with
    EVO_TEAM=<size>).  Both variants match the oracle on a ragged
    batch with mixed unit-granular schedules, and each other to summation
    order."""
    s = I.PUSHT
    wts = I.make_weights(s, 6, "perturbed")
    B = 7
    obs, noise = I.make_obs(s, B, 6), I.make_noise(s, B, 6)
    rng = np.random.default_rng([6, 3])
    lats = [I.lattice_bernoulli(3 * s.n_layers, s.n_steps, p, rng) for p in (0.1, 0.3, 0.6)]
    ids = np.array([0, 1, 2, 2, 1, 0, 1], np.int32)
    pol_t, got_t, st_t, _ = _case(f"team{size}_{dtype}", s, wts, obs, noise, lats, ids, dtype, gran=O.GRAN_UNIT,
                                  samples=[0, 3, 6], env={"EVO_TEAM": str(size)})
    pol_1, got_1, st_1, _ = _case(f"noteam_{dtype}", s, wts, obs, noise, lats, ids, dtype, gran=O.GRAN_UNIT,
                                  samples=[0, 3, 6], team=False)
    assert st_t["n_tiles"] == st_1["n_tiles"] == B
    assert st_1["n_workgroups"] == B
    assert st_t["n_workgroups"] in (B, size * B)
    if st_t["n_workgroups"] == size * B:
        assert st_t["cache_bytes_written"] == size * st_1["cache_bytes_written"]
    d = float(np.max(np.abs(got_t - got_1)))
    say(f"  team vs single workgroup: max-abs diff {d:.3e}")
    if dtype == "fp32":
        assert d <= 1e-4
    # repeated team calls are bitwise reproducible
    again, _ = run_gpu(pol_t, obs, noise, ids)
    assert np.array_equal(again, got_t)
    pol_t.close()
    pol_1.close()


@pytest.mark.parametrize("size", [4, 2])
def test_team_wait_timeout_is_reported(size):
    """Error path of the team variant, forced from the host: team member 0
    withholds its partial residuals (test hook) and the other members' waits
    give up after 64 polls.  The kernel still finishes; evo_synchronize
    reports the failure once and clears it; a policy created normally
    afterwards is unaffected."""
    import torch
    s = I.PUSHT
    wts = I.make_weights(s, 7, "perturbed")
    obs, noise = I.make_obs(s, 1, 7), I.make_noise(s, 1, 7)
    lat = I.lattice_bernoulli(3 * s.n_layers, s.n_steps, 0.2, np.random.default_rng(7))
    say(f"[gpu] team of {size}: wait timeout, forced from the host")
    pol = _policy(s, wts, "bf16", 1, 1, env={"EVO_TEAM_SPIN_LIMIT": "64", "EVO_TEAM": str(size)})
    pol.debug_team_withhold(True)
    pol.set_schedule(0, lat, O.GRAN_UNIT)
    dev = device()
    pol.denoise(torch.from_numpy(obs).to(dev), torch.from_numpy(noise).to(dev), None)
    st = pol.stats()
    if st["n_workgroups"] == st["n_tiles"]:
        pol.synchronize()
        pol.close()
        pytest.skip("the team variant is not used on this device")
    assert st["n_workgroups"] == size * st["n_tiles"]
    with pytest.raises(evo.EvoError) as e:
        pol.synchronize()
    assert e.value.code == -4 and "team barrier" in str(e.value)
    pol.synchronize()  # reported once, then cleared
    pol.close()
    pol2 = _policy(s, wts, "bf16", 1, 1)
    pol2.set_schedule(0, lat, O.GRAN_UNIT)
    got, st2 = run_gpu(pol2, obs, noise, np.zeros(1, np.int32))
    ref, _ = run_oracle(s, wts, obs, noise, [lat], np.zeros(1, np.int32), O.GRAN_UNIT, O.COLD_COMPUTE, "bf16")
    compare(got, ref, "bf16", "after a forced timeout")
    pol2.close()


def _case_stored(name, expect_tiles=None):
    """A full-size workload on the GPU against the oracle's chunks stored by
    tests/golden/make_oracle_outputs.py (every sample of the batch, or the
    stored spread subset), each sample checked on its own against the bar;
    bookkeeping against the oracle's integer counts."""
    w = I.WORKLOADS[name]
    inp = I.make_inputs(w)
    g = load_stored(name)
    samples = [int(j) for j in g["samples"]]
    say(f"[gpu] {name}: dtype={w.dtype} batch={w.batch}, {len(samples)} stored oracle samples")
    pol = _policy(w.shape, inp.weights, w.dtype, w.batch, len(inp.lattices))
    for j, lt in enumerate(inp.lattices):
        pol.set_schedule(j, lt, O.GRAN_LAYER)
    got, gst = run_gpu(pol, inp.obs, inp.noise, inp.ids)
    errs = [compare(got[j], g["chunks"][i], w.dtype, None) for i, j in enumerate(samples)]
    worst = int(np.argmax(errs))
    say(f"  {name}: worst sample {samples[worst]}: {'max-abs' if w.dtype == 'fp32' else 'rel'} "
        f"{errs[worst]:.3e}; median {float(np.median(errs)):.3e}")
    check_stats(gst, O.bookkeeping(w.shape, inp.lattices, inp.ids))
    if expect_tiles is not None:
        assert gst["n_tiles"] == expect_tiles
    pol.close()
    return errs


@pytest.mark.parametrize("name", ["pusht_fp32_b64_d25", "pusht_bf16_b64_d25", "pusht_bf16_b64_all"])
def test_pusht_b64_every_sample(name):
    _case_stored(name)


def test_image_b256_every_sample():
    _case_stored("image_bf16_b256_d12")


@pytest.mark.parametrize("name", ["bimanual_bf16_b128_d20", "bimanual_bf16_b128_all"])
def test_bimanual_b128_samples(name):
    """Every sample of the 20% lattice; 32 all-refresh samples spread over
    the batch (every XCD's tile range, every residue of the sample index
    mod 8)."""
    _case_stored(name)


def test_population_b512_every_sample():
    """512 samples, 64 schedules (10-40% density), per-sample ids."""
    _case_stored("population_bf16_b512")


# ---------------------------------------------------------------- invariants
def test_determinism_reset_and_independence():
    """Same inputs -> bitwise-same chunk; a call in between does not leak
    (caches are reset per query); a sample's chunk does not depend on the
    other samples of the batch or on its tile position.  The kernel variant
    is chosen by batch size (for fp32, teams of 4 up to n_cu/4 samples), and
    variants sum partial residuals in different orders, so the variant is
    fixed here (EVO_TEAM=2 serves both batch sizes)."""
    w = I.WORKLOADS["pusht_bf16_b64_d25"]
    s = w.shape
    inp = I.make_inputs(w)
    lats = I.population_lattices(s.n_layers, s.n_steps, 4, 0)
    ids = np.arange(64, dtype=np.int32) % 4
    say("[gpu] determinism/reset/independence pusht bf16 b64")
    pol = _policy(s, inp.weights, "bf16", 64, 4, env={"EVO_TEAM": "2"})
    for j, lt in enumerate(lats):
        pol.set_schedule(j, lt, O.GRAN_LAYER)
    a1, st = run_gpu(pol, inp.obs, inp.noise, ids)
    assert st["n_workgroups"] in (64, 128)
    obs2, noise2 = I.make_obs(s, 64, 9), I.make_noise(s, 64, 9)
    run_gpu(pol, obs2, noise2, ids[::-1].copy())
    a2, _ = run_gpu(pol, inp.obs, inp.noise, ids)
    assert np.array_equal(a1, a2)
    for n in (0, 13, 63):
        one, _ = run_gpu(pol, inp.obs[n:n + 1], inp.noise[:, n:n + 1], ids[n:n + 1])
        assert np.array_equal(one[0], a1[n]), n
    pol.close()


def test_two_sample_tiles_match_single_sample_tiles():
    """Population-sized batches use two samples per workgroup; the chunk of a
    sample matches its single-sample-tile result."""
    w = I.WORKLOADS["population_bf16_b512"]
    s = w.shape
    inp = I.make_inputs(w)
    say("[gpu] two-sample tiles vs single-sample tiles")
    pol = _policy(s, inp.weights, "bf16", 512, 64, team=False)
    for j, lt in enumerate(inp.lattices):
        pol.set_schedule(j, lt, O.GRAN_LAYER)
    big, st = run_gpu(pol, inp.obs, inp.noise, inp.ids)
    assert st["n_tiles"] == 256
    for n in (3, 77, 400):
        one, st1 = run_gpu(pol, inp.obs[n:n + 1], inp.noise[:, n:n + 1], inp.ids[n:n + 1])
        assert st1["n_tiles"] == 1
        np.testing.assert_allclose(one[0], big[n], rtol=0, atol=1e-5)
    pol.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_step0_only_cache_holds_step0_residuals(dtype):
    """Only step 0 refreshed (unit-granular): after the query every unit's
    cache holds r_{b,0}; the chunk matches the oracle."""
    s = I.PUSHT
    wts = I.make_weights(s, 3, "perturbed")
    obs, noise = I.make_obs(s, 1, 3), I.make_noise(s, 1, 3)
    lat = np.zeros((3 * s.n_layers, s.n_steps), np.uint8)
    lat[:, 0] = 1
    pol, got, gst, _ = _case(f"step0_only_{dtype}", s, wts, obs, noise, [lat], np.zeros(1, np.int32), dtype,
                             gran=O.GRAN_UNIT)
    P = O.prepare_params(I.split_weights(s, wts), dtype)
    eff = O.effective_lattice(O.expand_lattice(lat, O.GRAN_UNIT, s.n_layers), O.COLD_COMPUTE)
    tr = {}
    O.denoise_group(s, P, obs, noise, eff, trace=tr)
    worst = 0.0
    for b in range(3 * s.n_layers):
        c = pol.read_cache(b, 0).astype(np.float64)
        r0 = tr["r"][0, b, 0]
        e = float(np.max(np.abs(c - r0)))
        scale = max(float(np.max(np.abs(r0))), 1e-6)
        worst = max(worst, e / scale)
        assert (e <= 1e-4) if dtype == "fp32" else (e / scale <= 3e-2), (b, e)
    say(f"  cache readback worst relative error {worst:.2e}")
    per_wg = gst["n_workgroups"] // gst["n_tiles"]
    elt = 2 if dtype == "bf16" else 4   # fp16 caches with bf16 operands, fp32 with fp32
    assert gst["cache_bytes_written"] == 3 * s.n_layers * s.horizon * s.d_model * elt * per_wg
    pol.close()


@pytest.mark.parametrize("gran", [O.GRAN_UNIT, O.GRAN_LAYER])
def test_fp16_cache_saturates(gran):
    """With bf16 operands the residual caches hold fp16: a cached residual
    beyond the fp16 range reads back as +-65504 (a saturating store, never
    an infinity) and values inside it to fp16 rounding.  Only step 0 is
    refreshed, so the caches hold step-0 residuals; the first layer's
    self-attention output bias puts three columns at 1e5, -2e5 and 3e4.
    Layer-granular schedules cache the layer's summed residual in unit 2."""
    s = I.PUSHT
    wts = I.make_weights(s, 5, "perturbed")
    I.split_weights(s, wts)["l0.b_o"][[3, 7, 11]] = [1e5, -2e5, 3e4]
    obs, noise = I.make_obs(s, 1, 5), I.make_noise(s, 1, 5)
    rows = 3 * s.n_layers if gran == O.GRAN_UNIT else s.n_layers
    lat = np.zeros((rows, s.n_steps), np.uint8)
    lat[:, 0] = 1
    say(f"[gpu] fp16 cache saturation, granularity {gran}")
    pol = _policy(s, wts, "bf16", 1, 1)
    pol.set_schedule(0, lat, gran)
    got, _ = run_gpu(pol, obs, noise, np.zeros(1, np.int32))
    assert np.all(np.isfinite(got))
    P = O.prepare_params(I.split_weights(s, wts), "bf16")
    eff = O.effective_lattice(O.expand_lattice(lat, gran, s.n_layers), O.COLD_COMPUTE)
    tr = {}
    O.denoise_group(s, P, obs, noise, eff, trace=tr)
    if gran == O.GRAN_UNIT:
        unit, ref = 0, tr["r"][0, 0, 0]
    else:
        unit, ref = 2, tr["r"][0, 0, 0] + tr["r"][0, 1, 0] + tr["r"][0, 2, 0]
    c = pol.read_cache(unit, 0).astype(np.float64)
    pol.close()
    assert np.all(np.isfinite(c))
    big = np.abs(ref) > 65504.0
    assert big[:, 3].all() and big[:, 7].all() and big.sum() == 2 * s.horizon
    assert np.array_equal(c[big], np.sign(ref[big]) * 65504.0)
    large = (np.abs(ref) > 1000.0) & ~big   # the 3e4 column: fp16 spacing 16 there
    assert large[:, 11].all()
    assert np.max(np.abs(c[large] - ref[large]) / np.abs(ref[large])) <= 3e-2
    rest = ~big & ~large
    scale = float(np.max(np.abs(ref[rest])))
    err = float(np.max(np.abs(c[rest] - ref[rest])))
    say(f"  saturated {int(big.sum())} values; other columns relative error {err / scale:.2e}")
    assert err <= 3e-2 * scale


@pytest.mark.parametrize("cold", [O.COLD_COMPUTE, O.COLD_ZERO])
def test_printed_schedules(cold):
    """The paper's printed 24 x 100 unit schedules (three tasks, BAC and
    EVO; most EVO rows skip step 0) on the 8-layer policy."""
    s = I.PUSHT
    wts = I.make_weights(s, 4, "perturbed")
    lats = [printed_unit_lattice(tag, m) for tag in ("pusht", "kitchen", "lift_ph") for m in ("BAC", "EVO")]
    B = len(lats)
    obs, noise = I.make_obs(s, B, 4), I.make_noise(s, B, 4)
    ids = np.arange(B, dtype=np.int32)
    for dtype in ("fp32", "bf16"):
        pol, *_ = _case(f"printed_{dtype}_cold{cold}", s, wts, obs, noise, lats, ids, dtype, gran=O.GRAN_UNIT,
                        cold=cold)
        pol.close()


def test_comparison_schedule_families():
    """Fixed-interval synchronous refresh (EfficientVLA, M = 8 and 10) and
    block-wise fixed budgets (M = 10 per unit), unit- and layer-granular, on
    the 8-layer policy, one sample per schedule."""
    s = I.PUSHT
    wts = I.make_weights(s, 5, "perturbed")
    U, T = 3 * s.n_layers, s.n_steps
    rng = np.random.default_rng(5)
    for gran, rows in ((O.GRAN_UNIT, U), (O.GRAN_LAYER, s.n_layers)):
        lats = [I.lattice_fixed_interval(rows, T, 8), I.lattice_fixed_interval(rows, T, 10),
                I.lattice_blockwise_budget(rows, T, 10, rng)]
        B = len(lats)
        obs, noise = I.make_obs(s, B, 5), I.make_noise(s, B, 5)
        ids = np.arange(B, dtype=np.int32)
        for dtype in ("fp32", "bf16"):
            pol, *_ = _case(f"families_{dtype}_gran{gran}", s, wts, obs, noise, lats, ids, dtype, gran=gran)
            pol.close()


def test_hand_lattice_most_recent_unit():
    """One unit refreshed at steps {0, 2, 6} only, every other unit always."""
    s = I.TINY
    wts = I.make_weights(s, 6, "perturbed")
    obs, noise = I.make_obs(s, 2, 6), I.make_noise(s, 2, 6)
    lat = np.ones((6, 10), np.uint8)
    lat[4] = 0
    lat[4, [0, 2, 6]] = 1
    pol, *_ = _case("hand_lattice", s, wts, obs, noise, [lat], np.zeros(2, np.int32), "fp32", gran=O.GRAN_UNIT)
    pol.close()


def test_cold_zero_without_step0():
    s = I.TINY
    wts = I.make_weights(s, 7, "perturbed")
    obs, noise = I.make_obs(s, 2, 7), I.make_noise(s, 2, 7)
    lat = (np.random.default_rng(7).random((6, 10)) < 0.4).astype(np.uint8)
    lat[:, 0] = 0
    pol, *_ = _case("cold_zero", s, wts, obs, noise, [lat], np.zeros(2, np.int32), "fp32", gran=O.GRAN_UNIT,
                    cold=O.COLD_ZERO)
    pol.close()


def test_no_clip_fp32():
    s = I.TINY
    wts = I.make_weights(s, 8, "perturbed")
    obs, noise = I.make_obs(s, 2, 8), I.make_noise(s, 2, 8)
    lats = [I.lattice_bernoulli(2, 10, 0.5, np.random.default_rng(8))]
    say("[gpu] no clip fp32")
    pol = _policy(s, wts, "fp32", 2, 1, clip=False)
    pol.set_schedule(0, lats[0], O.GRAN_LAYER)
    got, _ = run_gpu(pol, obs, noise, np.zeros(2, np.int32))
    ref, _ = run_oracle(s, wts, obs, noise, lats, np.zeros(2, np.int32), O.GRAN_LAYER, O.COLD_COMPUTE, "fp32",
                        clip=False)
    rel = float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))
    say(f"  no-clip relative error {rel:.2e}")
    assert rel <= 1e-5
    pol.close()


def test_pairs_entry_point_equals_lattice():
    s = I.TINY
    wts = I.make_weights(s, 9, "perturbed")
    obs, noise = I.make_obs(s, 1, 9), I.make_noise(s, 1, 9)
    lat = I.lattice_bernoulli(6, 10, 0.4, np.random.default_rng(9))
    say("[gpu] pairs entry point")
    pol = _policy(s, wts, "fp32", 1, 2)
    pol.set_schedule(0, lat, O.GRAN_UNIT)
    pol.set_schedule_pairs(1, np.argwhere(lat > 0), O.GRAN_UNIT)
    a, _ = run_gpu(pol, obs, noise, np.array([0], np.int32))
    b, _ = run_gpu(pol, obs, noise, np.array([1], np.int32))
    assert np.array_equal(a, b)
    with pytest.raises(evo.EvoError):
        pol.set_schedule_pairs(1, [[0, 0], [0, 0]], O.GRAN_UNIT)
    pol.close()


def test_errors_leave_policy_usable():
    import torch
    s = I.TINY
    wts = I.make_weights(s, 0)
    say("[gpu] error paths")
    pol = _policy(s, wts, "fp32", 2, 2)
    pol.set_schedule(0, np.ones((2, 10), np.uint8), O.GRAN_LAYER)
    dev = device()
    obs = torch.zeros((2, s.n_obs, s.obs_dim), device=dev)
    noise = torch.zeros((s.n_steps, 2, s.horizon, s.action_dim), device=dev)
    with pytest.raises(evo.EvoError) as e:
        pol.denoise(obs, noise, np.array([0, 1], np.int32))      # schedule 1 not registered
    assert e.value.code == -2
    with pytest.raises(evo.EvoError) as e:
        pol.denoise(obs, noise, np.array([0, 5], np.int32))      # id out of range
    assert e.value.code == -1
    big_obs = torch.zeros((3, s.n_obs, s.obs_dim), device=dev)
    big_noise = torch.zeros((s.n_steps, 3, s.horizon, s.action_dim), device=dev)
    with pytest.raises(evo.EvoError) as e:
        pol.denoise(big_obs, big_noise, None)                    # batch > max_batch
    assert e.value.code == -1
    with pytest.raises(evo.EvoError):
        pol.set_schedule(0, np.ones((2, 9), np.uint8), O.GRAN_LAYER)
    out = pol.denoise(obs, noise, None)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    pol.close()


def test_automatic_team_choice():
    """The automatic team size follows the measured crossovers: bf16 runs
    teams of 2 up to n_cu/2 samples; fp32 runs teams of 4 up to n_cu/4
    samples, then teams of 2 up to n_cu/2; larger batches run one workgroup
    per tile (stats report workgroups per tile)."""
    import torch
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    s = I.PUSHT
    wts = I.make_weights(s, 0)
    lt = I.make_lattice("dirichlet", s.n_layers, s.n_steps, 0.25, 0)
    cases = [("bf16", 1, 2), ("bf16", n_cu // 4, 2), ("bf16", n_cu // 2, 2), ("bf16", n_cu // 2 + 1, 1),
             ("fp32", 1, 4), ("fp32", n_cu // 4, 4), ("fp32", n_cu // 4 + 1, 2), ("fp32", n_cu // 2 + 1, 1)]
    for dtype, B, want in cases:
        say(f"[gpu] automatic team choice: {dtype} batch {B}")
        pol = _policy(s, wts, dtype, B, 1)
        pol.set_schedule(0, lt, O.GRAN_LAYER)
        _, st = run_gpu(pol, I.make_obs(s, B, 0), I.make_noise(s, B, 0), np.zeros(B, np.int32))
        pol.close()
        per = st["n_workgroups"] // st["n_tiles"]
        assert st["n_tiles"] == B, (dtype, B, st["n_tiles"])
        assert per == want, f"{dtype} batch {B}: {per} workgroups per tile, expected {want}"


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_one_workgroup_per_tile_is_batch_independent(dtype):
    """With one workgroup per tile (teams switched off), a sample's chunk is
    the same bits at batch 8 and n_cu - 1 (one-sample tiles) and at
    n_cu + 64 (two-sample tiles, the sample's partner differing with the
    batch): the variants sum every product in the same order.  The
    schedule search runs this way."""
    import torch
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    s = I.PUSHT
    wts = I.make_weights(s, 6, "perturbed")
    Bmax = n_cu + 64
    obs, noise = I.make_obs(s, Bmax, 6), I.make_noise(s, Bmax, 6)
    rng = np.random.default_rng([6, 3])
    lats = [I.lattice_bernoulli(s.n_layers, s.n_steps, p, rng) for p in (0.2, 0.5)]
    ids = rng.integers(0, 2, Bmax).astype(np.int32)
    outs = {}
    for B in (8, n_cu - 1, Bmax):
        say(f"[gpu] one workgroup per tile: {dtype} batch {B}")
        pol = _policy(s, wts, dtype, B, 2, team=False)
        for j, lt in enumerate(lats):
            pol.set_schedule(j, lt, O.GRAN_LAYER)
        got, st = run_gpu(pol, obs[:B], noise[:, :B], ids[:B])
        pol.close()
        assert st["n_workgroups"] == st["n_tiles"] == (B if B < n_cu else (B + 1) // 2)
        outs[B] = got
    for B in (n_cu - 1, Bmax):
        assert np.array_equal(outs[B][:8], outs[8]), B
    assert np.array_equal(outs[Bmax][:n_cu - 1], outs[n_cu - 1])
    ref, _ = run_oracle(s, wts, obs[:8], noise[:, :8], lats, ids[:8], O.GRAN_LAYER, O.COLD_COMPUTE, dtype)
    compare(outs[8], ref, dtype, f"{dtype} batch 8, one workgroup per tile")


def test_replacing_a_schedule_between_calls():
    """The plan upload is skipped when the plan bytes are unchanged, so a
    schedule replaced under the same id (same batch, same ids) must still
    take effect: each call matches the oracle of the schedule registered at
    the time, also across a layer -> unit granularity change, and returning
    to the first schedule gives the first call's bits again."""
    s = I.TINY
    wts = I.make_weights(s, 7, "perturbed")
    obs, noise = I.make_obs(s, 3, 7), I.make_noise(s, 3, 7)
    ids = np.zeros(3, np.int32)
    rng = np.random.default_rng([7, 3])
    lat_a = I.lattice_bernoulli(s.n_layers, s.n_steps, 0.3, rng)
    lat_b = I.lattice_bernoulli(3 * s.n_layers, s.n_steps, 0.6, rng)
    pol = _policy(s, wts, "fp32", 3, 1)
    seq = [(lat_a, O.GRAN_LAYER), (lat_b, O.GRAN_UNIT), (lat_a, O.GRAN_LAYER)]
    outs = []
    for lat, gran in seq:
        say(f"[gpu] replace schedule 0: granularity {gran}")
        pol.set_schedule(0, lat, gran)
        got, _ = run_gpu(pol, obs, noise, ids)
        ref, _ = run_oracle(s, wts, obs, noise, [lat], ids, gran, O.COLD_COMPUTE, "fp32")
        compare(got, ref, "fp32", f"schedule granularity {gran}")
        outs.append(got)
    pol.close()
    assert not np.array_equal(outs[0], outs[1])
    assert np.array_equal(outs[0], outs[2])


def test_calls_on_two_streams_are_ordered():
    """A call on another stream than the previous call waits for it (the
    plan, caches and observation keys/values are per-policy buffers): two
    back-to-back calls on two streams, with no host synchronisation between
    them, both match the oracle."""
    import torch
    device()
    s = I.TINY
    wts = I.make_weights(s, 8, "perturbed")
    lat = I.lattice_bernoulli(s.n_layers, s.n_steps, 0.5, np.random.default_rng([8, 3]))
    pol = _policy(s, wts, "fp32", 2, 1)
    pol.set_schedule(0, lat, O.GRAN_LAYER)
    ids = np.zeros(2, np.int32)
    ins = [(I.make_obs(s, 2, 81 + k), I.make_noise(s, 2, 81 + k)) for k in range(2)]
    dev = torch.device("cuda:0")
    t_in = [(torch.from_numpy(o).to(dev), torch.from_numpy(n).to(dev)) for o, n in ins]
    outs = [torch.empty((2, s.horizon, s.action_dim), dtype=torch.float32, device=dev) for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority
    torch.cuda.synchronize()
    for k in range(2):
        pol.denoise(t_in[k][0], t_in[k][1], ids, out=outs[k], stream=streams[k])
    torch.cuda.synchronize()
    pol.synchronize()
    for k in range(2):
        ref, _ = run_oracle(s, wts, ins[k][0], ins[k][1], [lat], ids, O.GRAN_LAYER, O.COLD_COMPUTE, "fp32")
        compare(outs[k].cpu().numpy(), ref, "fp32", f"stream {k}")
    pol.close()


@pytest.mark.parametrize("cold", [O.COLD_ZERO, O.COLD_COMPUTE])
def test_empty_schedule(cold):
    """K = 0 (Eq. 3 with no pairs): with the zero cold-cache reading no unit
    is ever evaluated (every residual is zero, the chunk comes from the
    embedding, head and sampler alone); with the compute reading every unit
    runs at step 0 only.  Both match the oracle."""
    s = I.TINY
    wts = I.make_weights(s, 9, "perturbed")
    obs, noise = I.make_obs(s, 2, 9), I.make_noise(s, 2, 9)
    ids = np.zeros(2, np.int32)
    pol = _policy(s, wts, "fp32", 2, 1, cold=cold)
    pol.set_schedule_pairs(0, np.zeros((0, 2), np.int32), O.GRAN_UNIT)
    got, st = run_gpu(pol, obs, noise, ids)
    empty = np.zeros((3 * s.n_layers, s.n_steps), np.uint8)
    ref, ost = run_oracle(s, wts, obs, noise, [empty], ids, O.GRAN_UNIT, cold, "fp32")
    compare(got, ref, "fp32", f"empty schedule, cold {cold}")
    check_stats(st, ost)
    assert st["refreshes_effective"] == (0 if cold == O.COLD_ZERO else 2 * 3 * s.n_layers)
    pol.close()


def test_empty_batch_is_refused():
    """A batch of zero samples (or frames) is refused before any device work."""
    import torch
    dev = device()
    s = I.TINY
    pol = _policy(s, I.make_weights(s, 0), "fp32", 2, 1)
    pol.set_schedule(0, np.ones((2, 10), np.uint8), O.GRAN_LAYER)
    obs = torch.zeros((0, s.n_obs, s.obs_dim), device=dev)
    noise = torch.zeros((s.n_steps, 0, s.horizon, s.action_dim), device=dev)
    with pytest.raises(evo.EvoError) as e:
        pol.denoise(obs, noise, None)
    assert e.value.code == -1
    pol.close()
    en = I.ENC_TINY
    enc = evo.Encoder(en, I.make_encoder_weights(en, 0), "fp32", max_batch=2)
    with pytest.raises(evo.EvoError) as e:
        enc.encode(torch.zeros((0, en.height, en.width, en.in_ch), device=dev))
    assert e.value.code == -1
    enc.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_maximum_step_count(dtype):
    """170 reverse steps (the largest count the two-sample tiles hold), a
    ragged batch of 3 and a 30% lattice, against the oracle."""
    from dataclasses import replace
    s = replace(I.TINY, n_steps=170)
    wts = I.make_weights(s, 10, "perturbed")
    obs, noise = I.make_obs(s, 3, 10), I.make_noise(s, 3, 10)
    lat = I.lattice_bernoulli(s.n_layers, s.n_steps, 0.3, np.random.default_rng([10, 3]))
    pol, *_ = _case(f"tiny_T170_{dtype}", s, wts, obs, noise, [lat], np.zeros(3, np.int32), dtype)
    pol.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("base", ["tiny", "pusht"])
def test_maximum_obs_tokens_and_action_dim(base, dtype):
    """7 observation tokens (8 memory tokens) and 16 action dims, the largest
    compiled, on a ragged batch of 3 with a mixed pair of schedules (the
    Push-T shape at batch 3 runs the small-batch team variant)."""
    from dataclasses import replace
    s = replace(I.TINY if base == "tiny" else I.PUSHT, n_obs=7, action_dim=16)
    wts = I.make_weights(s, 11, "perturbed")
    obs, noise = I.make_obs(s, 3, 11), I.make_noise(s, 3, 11)
    rng = np.random.default_rng([11, 3])
    lats = [I.lattice_bernoulli(s.n_layers, s.n_steps, p, rng) for p in (0.3, 0.7)]
    pol, *_ = _case(f"{base}_obs7_a16_{dtype}", s, wts, obs, noise, lats, np.array([1, 0, 1], np.int32), dtype)
    pol.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("n_obs,batch", [(3, 3), (3, 301), (4, 3)])
def test_cross_attention_fold_boundary(n_obs, batch, dtype):
    """Width-256 cross-attention at the boundary of its folded form: 3
    observation tokens fill all 16 folded score columns (4 heads x 4 memory
    tokens), 4 fall back to the projected unit.  Batch 3 runs the small-batch
    teams (every member evaluates the folded unit), batch 301 two-sample
    tiles with a half-empty last tile (oracle on the first, a middle and the
    last sample); two schedules mixed."""
    from dataclasses import replace
    s = replace(I.PUSHT, n_obs=n_obs)
    wts = I.make_weights(s, 13, "perturbed")
    obs, noise = I.make_obs(s, batch, 13), I.make_noise(s, batch, 13)
    rng = np.random.default_rng([13, n_obs])
    lats = [I.lattice_bernoulli(s.n_layers, s.n_steps, p, rng) for p in (0.25, 0.6)]
    ids = (np.arange(batch) % 2).astype(np.int32)
    samples = None if batch <= 3 else [0, batch // 2, batch - 1]
    pol, *_ = _case(f"pusht_obs{n_obs}_b{batch}_{dtype}", s, wts, obs, noise, lats, ids, dtype, samples=samples)
    pol.close()
