"""Pins of the observation-encoder oracle (oracle/evo_encoder.py) against
torch's float64 CPU operators (an independent implementation): convolution,
GroupNorm, max pooling, and the whole network rebuilt from torch.nn layers
with the same weights.  Plus closed forms: a 1x1 convolution is a matrix
product per pixel, GroupNorm output has zero mean and unit variance per
group, and the FLOP count of a single convolution."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import evo_encoder as E
from paper_2607_20293_amd import inputs as I


def _nchw(x):
    return torch.from_numpy(np.ascontiguousarray(np.transpose(np.asarray(x, np.float64), (0, 3, 1, 2))))


def _oihw(w):
    return torch.from_numpy(np.ascontiguousarray(np.transpose(np.asarray(w, np.float64), (0, 3, 1, 2))))


def _nhwc(t):
    return np.transpose(t.numpy(), (0, 2, 3, 1))


@pytest.mark.parametrize("k,stride,pad,cin,cout,hw", [(7, 2, 3, 3, 8, 19), (3, 1, 1, 5, 4, 9), (3, 2, 1, 6, 7, 10),
                                                     (1, 2, 0, 4, 6, 11), (1, 1, 0, 3, 2, 5)])
def test_conv2d_matches_torch(k, stride, pad, cin, cout, hw):
    rng = np.random.default_rng(k * 100 + stride * 10 + cin)
    x = rng.standard_normal((2, hw, hw + 1, cin))
    w = rng.standard_normal((cout, k, k, cin))
    want = _nhwc(F.conv2d(_nchw(x), _oihw(w), stride=stride, padding=pad))
    got = E.conv2d(x, w, stride, pad)
    assert got.shape == want.shape
    assert np.max(np.abs(got - want)) < 1e-12


def test_conv1x1_is_a_matrix_product():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 4, 5, 6))
    w = rng.standard_normal((3, 1, 1, 6))
    assert np.allclose(E.conv2d(x, w, 1, 0), np.einsum("nhwc,oc->nhwo", x, w[:, 0, 0, :]), rtol=0, atol=1e-13)


def test_group_norm_matches_torch_and_normalises():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 5, 6, 32)) * 3 + 1
    g, b = rng.standard_normal(32), rng.standard_normal(32)
    want = _nhwc(F.group_norm(_nchw(x), 32 // 8, torch.from_numpy(g), torch.from_numpy(b), eps=1e-5))
    got = E.group_norm(x, 8, g, b)
    assert np.max(np.abs(got - want)) < 1e-12
    y = E.group_norm(x, 8, np.ones(32), np.zeros(32)).reshape(3, 30, 4, 8)
    assert np.allclose(y.mean(axis=(1, 3)), 0, atol=1e-12)
    assert np.allclose(y.var(axis=(1, 3)), 1, atol=1e-4)      # var / (var + eps)


def test_max_pool_matches_torch():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 9, 8, 3))
    want = _nhwc(F.max_pool2d(_nchw(x), 3, 2, 1))
    assert np.array_equal(E.max_pool(x), want)


def _torch_encoder(e, P):
    """The same network from torch.nn layers (float64), weights copied."""
    import torch.nn as nn

    def conv(name, stride, pad):
        w = _oihw(P[name])
        m = nn.Conv2d(w.shape[1], w.shape[0], w.shape[2], stride, pad, bias=False).double()
        m.weight.data.copy_(w)
        return m

    def gn(name, c):
        m = nn.GroupNorm(c // e.gn_group, c, eps=1e-5).double()
        m.weight.data.copy_(torch.from_numpy(np.asarray(P[name + "_g"], np.float64)))
        m.bias.data.copy_(torch.from_numpy(np.asarray(P[name + "_b"], np.float64)))
        return m

    class Block(nn.Module):
        def __init__(self, p, cin, c, stride):
            super().__init__()
            self.ca, self.na = conv(p + "a", stride, 1), gn(p + "a", c)
            self.cb, self.nb = conv(p + "b", 1, 1), gn(p + "b", c)
            self.proj = (p + "d") in P
            if self.proj:
                self.cd, self.nd = conv(p + "d", stride, 0), gn(p + "d", c)

        def forward(self, x):
            y = torch.relu(self.na(self.ca(x)))
            y = self.nb(self.cb(y))
            s = self.nd(self.cd(x)) if self.proj else x
            return torch.relu(y + s)

    layers = [conv("stem", 2, 3), gn("stem", e.stem_ch), nn.ReLU(), nn.MaxPool2d(3, 2, 1)]
    cin = e.stem_ch
    for si, (c, nb) in enumerate(zip(e.widths, e.blocks)):
        for bi in range(nb):
            layers.append(Block(f"s{si}b{bi}.", cin, c, 2 if (si > 0 and bi == 0) else 1))
            cin = c
    layers += [nn.AdaptiveAvgPool2d(1), nn.Flatten()]
    return nn.Sequential(*layers)


@pytest.mark.parametrize("shape", ["tiny", "pusht"])
def test_encoder_matches_torch_network(shape):
    e = I.ENC_TINY if shape == "tiny" else I.ENC_PUSHT
    P = I.split_encoder_weights(e, I.make_encoder_weights(e, 1, "perturbed"))
    imgs = I.make_images(e, 2, 1)
    got = E.encode(e, P, imgs)
    with torch.no_grad():
        want = _torch_encoder(e, P)(_nchw(imgs)).numpy()
    assert got.shape == (2, e.out_dim)
    assert np.max(np.abs(got - want)) < 1e-10
    # bf16 mode: identical to fp64 on bf16-rounded convolution weights
    Pb = {k: (E.O.to_bf16(np.asarray(v, np.float64)) if np.asarray(v).ndim == 4 else v) for k, v in P.items()}
    assert np.max(np.abs(E.encode(e, P, imgs, "bf16") - E.encode(e, Pb, imgs))) == 0.0


def test_conv_flops_closed_form():
    e = I.EncoderShape(8, 8, stem_ch=4, widths=(4,), blocks=(1,), gn_group=4)
    # stem 4x4 out: 2*16*4*49*3; pooled 2x2; block: two 3x3 convs 2*4*4*36 each
    assert E.conv_flops(e, 3) == 3 * (2 * 16 * 4 * 147 + 2 * (2 * 4 * 4 * 36))
