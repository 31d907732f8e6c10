"""GPU parity of the redundancy-aware initialisation (Sec. 3.3, Eq. 6/7):
activations recorded by the HIP path, the Gram-based dissimilarity scores,
and the guided positions they lead to, against the fp64 oracle."""
import numpy as np
import pytest

from oracle import evo_oracle as O
from oracle import evo_redundancy as RD
from paper_2607_20293_amd import evo
from paper_2607_20293_amd import inputs as I
from tests.gpu_util import device, say

pytestmark = pytest.mark.gpu


def _policy(shape, wts, dtype, B):
    device()
    return evo.Policy(shape, wts, dtype=dtype, max_batch=B, max_schedules=1)


def _collect(shape, wts, dtype, B, seed, lat=None, fill=0.0):
    import torch
    dev = device()
    pol = _policy(shape, wts, dtype, B)
    U, T = 3 * shape.n_layers, shape.n_steps
    pol.set_schedule(0, np.ones((U, T), np.uint8) if lat is None else lat, O.GRAN_UNIT)
    obs, noise = I.make_obs(shape, B, seed), I.make_noise(shape, B, seed)
    acts = torch.full((B, U, T, shape.horizon, shape.d_model), fill, dtype=torch.float32, device=dev)
    out = pol.denoise(torch.from_numpy(obs).to(dev), torch.from_numpy(noise).to(dev), None, acts=acts)
    pol.synchronize()
    return pol, obs, noise, out.cpu().numpy(), acts


@pytest.mark.parametrize("name,dtype,B", [("tiny", "fp32", 3), ("pusht", "fp32", 2), ("pusht", "bf16", 1)])
def test_collected_activations_match_oracle(name, dtype, B):
    s = I.TINY if name == "tiny" else I.PUSHT
    wts = I.make_weights(s, 21, "perturbed")
    say(f"[gpu] activations {name} {dtype} batch {B}")
    pol, obs, noise, _, acts = _collect(s, wts, dtype, B, 21)
    got = acts.cpu().numpy().reshape(B, 3 * s.n_layers, s.n_steps, -1).astype(np.float64)
    P = O.prepare_params(I.split_weights(s, wts), dtype)
    want = RD.collect_activations(s, P, obs, noise)
    err = float(np.max(np.abs(got - want)))
    scale = float(np.max(np.abs(want)))
    say(f"  max-abs {err:.3e} (scale {scale:.3e})")
    if dtype == "fp32":
        assert err <= 1e-4
    else:
        assert err / scale <= 3e-2
    pol.close()


def test_unevaluated_positions_are_left_untouched():
    s = I.TINY
    wts = I.make_weights(s, 22, "perturbed")
    lat = I.lattice_bernoulli(3 * s.n_layers, s.n_steps, 0.4, np.random.default_rng(22))
    pol, obs, noise, _, acts = _collect(s, wts, "fp32", 2, 22, lat=lat, fill=7.0)
    got = acts.cpu().numpy().reshape(2, 3 * s.n_layers, s.n_steps, -1)
    P = O.prepare_params(I.split_weights(s, wts), "fp32")
    eff = O.effective_lattice(O.expand_lattice(lat, O.GRAN_UNIT, s.n_layers), O.COLD_COMPUTE)
    tr = {}
    O.denoise_group(s, P, obs, noise, eff, trace=tr)
    ref = tr["r"].transpose(2, 1, 0, 3, 4).reshape(got.shape)
    m = eff.astype(bool)
    assert np.all(got[:, ~m] == 7.0)
    assert np.max(np.abs(got[:, m] - ref[:, m])) <= 1e-4
    pol.close()


@pytest.mark.parametrize("name,R", [("tiny", 3), ("pusht", 3)])
def test_scores_kernel_on_oracle_activations(name, R):
    """The Gram kernel alone: the oracle's activations (rounded to fp32) in,
    Eq. 6 scores out, against the oracle's scores of the same fp32 values.
    One activation vector is zeroed to exercise the zero-norm reading."""
    import torch
    s = I.TINY if name == "tiny" else I.PUSHT
    wts = I.make_weights(s, 23, "perturbed")
    P = O.prepare_params(I.split_weights(s, wts), "fp32")
    acts = RD.collect_activations(s, P, I.make_obs(s, R, 23), I.make_noise(s, R, 23)).astype(np.float32)
    acts[1, 2, 3] = 0.0
    want = RD.redundancy_scores(acts)
    pol = _policy(s, wts, "fp32", R)
    got = pol.redundancy_scores(torch.from_numpy(acts).to(device())).cpu().numpy()
    pol.synchronize()
    err = float(np.max(np.abs(got - want)))
    say(f"[gpu] scores kernel {name} R={R}: max-abs {err:.3e}")
    assert err <= 2e-5
    pol.close()


def test_scores_and_guided_schedule_end_to_end():
    """Activations recorded by the HIP path -> scores on the GPU -> Eq. 7 on
    the host -> K guided positions -> a schedule the library runs; against
    the oracle's chain on the same inputs."""
    import torch
    s = I.PUSHT
    R = 2
    wts = I.make_weights(s, 24, "perturbed")
    pol, obs, noise, _, acts = _collect(s, wts, "fp32", R, 24)
    sc = pol.redundancy_scores(acts).cpu().numpy()
    P = O.prepare_params(I.split_weights(s, wts), "fp32")
    want = RD.redundancy_scores(RD.collect_activations(s, P, obs, noise))
    err = float(np.max(np.abs(sc - want)))
    say(f"[gpu] end-to-end scores: max-abs {err:.3e}")
    assert err <= 1e-4
    p = evo.guided_probabilities(sc, 0.05, 2.0)
    assert np.allclose(p, RD.guided_probabilities(want, 0.05, 2.0), rtol=5e-3, atol=0)
    pairs = evo.guided_sample(p, 240, np.random.default_rng(24).uniform(size=p.shape))
    pol.set_schedule_pairs(0, pairs, O.GRAN_UNIT)
    out = pol.denoise(torch.from_numpy(obs).to(device()), torch.from_numpy(noise).to(device()))
    pol.synchronize()
    assert torch.isfinite(out).all()
    assert pol.stats()["refreshes_requested"] == 240 * R
    pol.close()
