"""GPU parity of the observation encoder (evo_create_encoder / evo_encode)
against the fp64 oracle (oracle/evo_encoder.py) on seeded synthetic images:
fp32 operands max-abs <= 1e-4 of features of order one, bf16 operands
normwise relative <= 3e-2 (the oracle rounds the same weights to bf16; the
kernel also rounds the activations it multiplies).  Sizes: a tiny network
with ragged tiles (channels and pixel counts not multiples of 64) and the
96x96 network at a small batch; strided output rows."""
from dataclasses import replace

import numpy as np
import pytest

from oracle import evo_encoder as E
from oracle import evo_oracle as O
from paper_2607_20293_amd import inputs as I
from tests.gpu_util import compare

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _run(e, dtype, batch, seed, variant="perturbed", stride=None):
    torch = _torch()
    from paper_2607_20293_amd import evo
    w = I.make_encoder_weights(e, seed, variant)
    imgs = I.make_images(e, batch, seed)
    enc = evo.Encoder(e, w, dtype, max_batch=max(batch, 2))
    x = torch.from_numpy(imgs).cuda()
    if stride is None:
        out = enc.encode(x)
    else:
        buf = torch.full((batch, stride), 7.0, device="cuda")
        out = enc.encode(x, out=buf[:, 1:1 + e.out_dim])
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    if stride is not None:
        rest = torch.cat([buf[:, :1], buf[:, 1 + e.out_dim:]], 1).cpu().numpy()
        assert np.all(rest == 7.0), "elements outside the feature columns were written"
    enc.close()
    want = E.encode(e, I.split_encoder_weights(e, w), imgs, dtype)
    return got, want


def _rel(got, want):
    return float(np.linalg.norm(got - want) / np.linalg.norm(want))


@pytest.mark.parametrize("batch", [1, 3])
def test_encoder_tiny_fp32(batch):
    got, want = _run(I.ENC_TINY, "fp32", batch, 11)
    print("tiny fp32 max-abs", np.max(np.abs(got - want)))
    assert np.max(np.abs(got - want)) <= 1e-4


@pytest.mark.parametrize("batch", [1, 3])
def test_encoder_tiny_bf16(batch):
    got, want = _run(I.ENC_TINY, "bf16", batch, 12)
    print("tiny bf16 rel", _rel(got, want))
    assert _rel(got, want) <= 3e-2


def test_encoder_pusht_fp32_strided_rows():
    got, want = _run(I.ENC_PUSHT, "fp32", 2, 13, stride=600)
    print("pusht fp32 max-abs", np.max(np.abs(got - want)))
    assert np.max(np.abs(got - want)) <= 1e-4


def test_encoder_pusht_bf16():
    got, want = _run(I.ENC_PUSHT, "bf16", 2, 14)
    print("pusht bf16 rel", _rel(got, want))
    assert _rel(got, want) <= 3e-2


def test_encoder_robomimic_bf16_default_affine():
    got, want = _run(I.ENC_ROBOMIMIC, "bf16", 2, 15, variant="default")
    print("robomimic bf16 rel", _rel(got, want))
    assert _rel(got, want) <= 3e-2


def test_encoder_batch_independent():
    """An image's features do not depend on the other images of the batch,
    on its position in it or on the batch size (bit-exact, one encoder, with
    maps large enough for several GroupNorm chunks and late layers whose
    convolutions split K)."""
    torch = _torch()
    from paper_2607_20293_amd import evo
    e = I.ENC_PUSHT
    imgs = I.make_images(e, 10, 3)
    enc = evo.Encoder(e, I.make_encoder_weights(e, 3, "perturbed"), "bf16", max_batch=10)
    run = lambda idx: enc.encode(torch.from_numpy(np.ascontiguousarray(imgs[idx])).cuda()).cpu().numpy()
    a = run([0, 1, 2, 3])
    b = run([4, 1, 5, 6])
    c = run([1, 7, 8, 9])
    assert np.array_equal(a[1], b[1]) and np.array_equal(a[1], c[0])
    enc.close()
    for dtype in ("fp32", "bf16"):
        enc = evo.Encoder(e, I.make_encoder_weights(e, 3, "perturbed"), dtype, max_batch=10)
        one = run([1])[0]
        three = run([5, 1, 7])[1]
        ten = run(list(range(10)))[1]
        assert np.array_equal(one, ten) and np.array_equal(one, three), dtype
        enc.close()


def test_encoder_rejects_bad_arguments():
    torch = _torch()
    from paper_2607_20293_amd import evo
    e = I.ENC_TINY
    enc = evo.Encoder(e, I.make_encoder_weights(e, 3), "fp32", max_batch=2)
    x = torch.from_numpy(I.make_images(e, 3, 3)).cuda()
    with pytest.raises(evo.EvoError):
        enc.encode(x)                       # batch above max_batch
    with pytest.raises(evo.EvoError):
        evo.Encoder(e, I.make_encoder_weights(e, 3)[:-1], "fp32")
    # a misaligned view of the images is refused before anything runs
    flat = torch.zeros(1 + 2 * e.height * e.width * e.in_ch, device="cuda")
    view = flat[1:].view(2, e.height, e.width, e.in_ch)
    with pytest.raises(evo.EvoError, match="aligned"):
        enc.encode(view)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_encode_then_denoise_matches_oracle_chain(dtype):
    """The whole action query: camera frames -> encoder features written into
    the observation rows beside the proprioceptive columns -> cached
    denoising, against the oracle's encoder followed by the oracle's loop."""
    torch = _torch()
    from paper_2607_20293_amd import evo
    e = I.ENC_TINY
    s = replace(I.TINY, obs_dim=e.out_dim + 4)
    B = 3
    ew = I.make_encoder_weights(e, 21, "perturbed")
    pw = I.make_weights(s, 21, "perturbed")
    imgs = I.make_images(e, B * s.n_obs, 21)   # frame t of sample b is image b * n_obs + t
    obs = I.make_obs(s, B, 21)                 # the last 4 columns stay (proprioception)
    noise = I.make_noise(s, B, 21)
    lats = [I.lattice_bernoulli(s.n_layers, s.n_steps, 0.4, np.random.default_rng(21))]
    ids = np.zeros(B, np.int32)

    enc = evo.Encoder(e, ew, dtype, max_batch=B * s.n_obs)
    pol = evo.Policy(s, pw, dtype=dtype, max_batch=B, max_schedules=1)
    pol.set_schedule(0, lats[0], evo.GRAN_LAYER)
    obs_d = torch.from_numpy(obs).cuda()
    enc.encode(torch.from_numpy(imgs).cuda(), out=obs_d.view(B * s.n_obs, s.obs_dim)[:, :e.out_dim])
    got = pol.denoise(obs_d, torch.from_numpy(noise).cuda(), ids).cpu().numpy()
    assert np.array_equal(obs_d[:, :, e.out_dim:].cpu().numpy(), obs[:, :, e.out_dim:])
    pol.close()
    enc.close()

    f = E.encode(e, I.split_encoder_weights(e, ew), imgs, dtype)
    obs_ref = obs.astype(np.float64)
    obs_ref[:, :, :e.out_dim] = f.reshape(B, s.n_obs, e.out_dim)
    ref, _ = O.denoise(s, I.split_weights(s, pw), obs_ref, noise, lats, ids, granularity=O.GRAN_LAYER,
                       cold_policy=O.COLD_COMPUTE, clip=True, dtype=dtype)
    compare(got, ref, dtype, f"encode+denoise {dtype}")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_encoder_large_tiles_sampled_frames(dtype):
    """A batch large enough that no convolution splits K (thousands of
    output tiles, ragged in channels nowhere and in pixels at the last
    stage), checked on sampled frames: frames are independent, so the
    oracle runs on those frames alone."""
    torch = _torch()
    from paper_2607_20293_amd import evo
    e = I.EncoderShape(64, 64, stem_ch=64, widths=(128, 256), blocks=(1, 1), gn_group=16)
    B, pick = 256, [0, 77, 255]
    w = I.make_encoder_weights(e, 31, "perturbed")
    imgs = I.make_images(e, B, 31)
    enc = evo.Encoder(e, w, dtype, max_batch=B)
    got = enc.encode(torch.from_numpy(imgs).cuda()).cpu().numpy().astype(np.float64)[pick]
    enc.close()
    want = E.encode(e, I.split_encoder_weights(e, w), imgs[pick], dtype)
    if dtype == "fp32":
        print("large tiles fp32 max-abs", np.max(np.abs(got - want)))
        assert np.max(np.abs(got - want)) <= 1e-4
    else:
        print("large tiles bf16 rel", _rel(got, want))
        assert _rel(got, want) <= 3e-2


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_encoder_odd_shape(dtype):
    """Odd image sizes (ragged maps at every stage), one input channel (the
    element-wise gather), GroupNorm groups of 4 channels, two blocks in the
    first stage (identity shortcuts)."""
    e = I.EncoderShape(37, 29, in_ch=1, stem_ch=8, widths=(8, 16), blocks=(2, 1), gn_group=4)
    got, want = _run(e, dtype, 2, 32)
    if dtype == "fp32":
        print("odd fp32 max-abs", np.max(np.abs(got - want)))
        assert np.max(np.abs(got - want)) <= 1e-4
    else:
        print("odd bf16 rel", _rel(got, want))
        assert _rel(got, want) <= 3e-2


def test_image_policy_query_matches_oracle_chain():
    """The image policy's own configuration: 84x84 frames, 512 features
    written into observation rows of 521 floats (an odd row stride, the
    9 proprioceptive columns kept), then the cached loop with a 25% lattice
    in bf16; two samples against the oracle encoder followed by the oracle
    loop."""
    torch = _torch()
    from paper_2607_20293_amd import evo
    e, s = I.ENC_ROBOMIMIC, I.IMAGE
    assert s.obs_dim - e.out_dim == 9
    B = 2
    ew, pw = I.make_encoder_weights(e, 41, "perturbed"), I.make_weights(s, 41, "perturbed")
    imgs = I.make_images(e, B * s.n_obs, 41)
    obs, noise = I.make_obs(s, B, 41), I.make_noise(s, B, 41)
    lats = [I.make_lattice("dirichlet", s.n_layers, s.n_steps, 0.25, 41)]
    ids = np.zeros(B, np.int32)
    enc = evo.Encoder(e, ew, "bf16", max_batch=B * s.n_obs)
    pol = evo.Policy(s, pw, dtype="bf16", max_batch=B, max_schedules=1)
    pol.set_schedule(0, lats[0], evo.GRAN_LAYER)
    obs_d = torch.from_numpy(obs).cuda()
    enc.encode(torch.from_numpy(imgs).cuda(), out=obs_d.view(B * s.n_obs, s.obs_dim)[:, :e.out_dim])
    got = pol.denoise(obs_d, torch.from_numpy(noise).cuda(), ids).cpu().numpy()
    assert np.array_equal(obs_d[:, :, e.out_dim:].cpu().numpy(), obs[:, :, e.out_dim:])
    pol.close()
    enc.close()
    f = E.encode(e, I.split_encoder_weights(e, ew), imgs, "bf16")
    obs_ref = obs.astype(np.float64)
    obs_ref[:, :, :e.out_dim] = f.reshape(B, s.n_obs, e.out_dim)
    ref, _ = O.denoise(s, I.split_weights(s, pw), obs_ref, noise, lats, ids, granularity=O.GRAN_LAYER,
                       cold_policy=O.COLD_COMPUTE, clip=True, dtype="bf16")
    compare(got, ref, "bf16", "image policy query bf16")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_encoder_bench_batch_sampled_frames(dtype):
    """The benchmark's encode: 512 frames of 84x84 (the image policy's 256
    chunks x 2 observation steps) on an encoder planned for 512 frames, which
    runs the stem's GroupNorm in two passes and every other GroupNorm as one
    kernel over several groups per workgroup; frames spread over the batch
    against the oracle on those frames alone."""
    torch = _torch()
    from paper_2607_20293_amd import evo
    e = I.ENC_ROBOMIMIC
    B, pick = 512, [0, 200, 511]
    w = I.make_encoder_weights(e, 33, "perturbed")
    imgs = I.make_images(e, B, 33)
    enc = evo.Encoder(e, w, dtype, max_batch=B)
    got = enc.encode(torch.from_numpy(imgs).cuda()).cpu().numpy().astype(np.float64)[pick]
    enc.close()
    want = E.encode(e, I.split_encoder_weights(e, w), imgs[pick], dtype)
    if dtype == "fp32":
        print("bench batch fp32 max-abs", np.max(np.abs(got - want)))
        assert np.max(np.abs(got - want)) <= 1e-4
    else:
        print("bench batch bf16 rel", _rel(got, want))
        assert _rel(got, want) <= 3e-2
