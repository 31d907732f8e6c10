"""GPU parity of the observation encoder (evo_create_encoder / evo_encode)
against the fp64 oracle (oracle/evo_encoder.py) on seeded synthetic images:
fp32 operands max-abs <= 1e-4 of features of order one, bf16 operands
normwise relative <= 3e-2 (the oracle rounds the same weights to bf16; the
kernel also rounds the activations it multiplies).  Sizes: a tiny network
with ragged tiles (channels and pixel counts not multiples of 64) and the
96x96 network at a small batch; strided output rows."""
import numpy as np
import pytest

from oracle import evo_encoder as E
from paper_2607_20293_amd import inputs as I

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
    """An image's features do not depend on the other images of the batch
    (same kernels, different batch sizes, bit-exact)."""
    torch = _torch()
    from paper_2607_20293_amd import evo
    e = I.ENC_TINY
    enc = evo.Encoder(e, I.make_encoder_weights(e, 3, "perturbed"), "bf16", max_batch=70)
    x = torch.from_numpy(I.make_images(e, 70, 3)).cuda()
    big = enc.encode(x).cpu().numpy()
    small = enc.encode(x[5:6].contiguous()).cpu().numpy()
    assert np.array_equal(big[5:6], small)


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
