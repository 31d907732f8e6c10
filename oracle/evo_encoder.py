"""CPU fp64 oracle of the observation encoder that turns camera images into
the visual part of the policy's observation tokens.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
baseline may import this module.  It shares no code with the HIP library and
imports nothing from the product package.

The paper keeps the pretrained policy's observation encoder unchanged
(Sec. 3.1, Sec. 3.4) and times action generation with visual encoding
included (appendix, wall-clock table), but prints no architecture for it.
Reading (listed in the design notes): the encoder of the image-based
diffusion policies it evaluates, a ResNet-18-topology network with GroupNorm
in place of BatchNorm and global average pooling, no final linear layer:

* stem: 7x7 stride-2 convolution (padding 3), GroupNorm, ReLU, 3x3 stride-2
  max pooling (padding 1);
* stages of basic blocks: y = ReLU(GN(conv3x3(ReLU(GN(conv3x3(x))))) + s(x)),
  where s is the identity, or GN(conv1x1 stride 2(x)) for the first block of
  a stage that halves the resolution or changes the width;
* global average pooling over the final feature map.

Convolutions have no bias; GroupNorm uses the population variance over each
group's channels and all pixels, eps 1e-5, then a per-channel gain and
shift.  Arithmetic is float64; in 'bf16' mode the convolution weights are
first rounded to bf16 (round to nearest even), like the denoiser's matrices.

Every function is pinned in tests/test_encoder_pins.py against torch's
float64 convolution, GroupNorm and pooling and a torch module built from its
layers.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import evo_oracle as O


def conv2d(x: np.ndarray, w: np.ndarray, stride: int, pad: int) -> np.ndarray:
    """x [N][H][W][Cin], w [Cout][kh][kw][Cin] -> [N][Ho][Wo][Cout]:
    y[n,i,j,o] = sum_{a,b,c} xpad[n, i*stride + a, j*stride + b, c] w[o,a,b,c]."""
    x = np.asarray(x, np.float64)
    w = np.asarray(w, np.float64)
    N, H, W, C = x.shape
    Co, kh, kw, Ci = w.shape
    assert Ci == C
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    Ho = (H + 2 * pad - kh) // stride + 1
    Wo = (W + 2 * pad - kw) // stride + 1
    cols = np.empty((N, Ho, Wo, kh, kw, C))
    for a in range(kh):
        for b in range(kw):
            cols[:, :, :, a, b, :] = xp[:, a:a + stride * (Ho - 1) + 1:stride, b:b + stride * (Wo - 1) + 1:stride, :]
    return (cols.reshape(N * Ho * Wo, kh * kw * C) @ w.reshape(Co, -1).T).reshape(N, Ho, Wo, Co)


def group_norm(x: np.ndarray, group: int, g: np.ndarray, b: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """Per sample and group of `group` consecutive channels: (x - mean) /
    sqrt(var + eps) over the group's channels and all pixels, then x g + b."""
    x = np.asarray(x, np.float64)
    N, H, W, C = x.shape
    xg = x.reshape(N, H * W, C // group, group)
    mu = xg.mean(axis=(1, 3), keepdims=True)
    var = ((xg - mu) ** 2).mean(axis=(1, 3), keepdims=True)
    y = ((xg - mu) / np.sqrt(var + eps)).reshape(N, H, W, C)
    return y * np.asarray(g, np.float64) + np.asarray(b, np.float64)


def relu(x: np.ndarray) -> np.ndarray:
    return np.maximum(x, 0.0)


def max_pool(x: np.ndarray, k: int = 3, stride: int = 2, pad: int = 1) -> np.ndarray:
    """Max over k x k windows (stride, padding excluded from the max)."""
    N, H, W, C = x.shape
    xp = np.pad(np.asarray(x, np.float64), ((0, 0), (pad, pad), (pad, pad), (0, 0)), constant_values=-np.inf)
    Ho = (H + 2 * pad - k) // stride + 1
    Wo = (W + 2 * pad - k) // stride + 1
    y = np.full((N, Ho, Wo, C), -np.inf)
    for a in range(k):
        for b in range(k):
            y = np.maximum(y, xp[:, a:a + stride * (Ho - 1) + 1:stride, b:b + stride * (Wo - 1) + 1:stride, :])
    return y


def prepare(e, params: Dict[str, np.ndarray], dtype: str) -> Dict[str, np.ndarray]:
    out = {}
    for name, v in params.items():
        v = np.asarray(v, np.float64)
        if dtype == "bf16" and v.ndim == 4:
            v = O.to_bf16(v)
        out[name] = v
    return out


def encode(e, params: Dict[str, np.ndarray], images: np.ndarray, dtype: str = "fp32") -> np.ndarray:
    """Features [N][out_dim] of images [N][H][W][in_ch]."""
    P = prepare(e, params, dtype)
    G = e.gn_group
    x = relu(group_norm(conv2d(images, P["stem"], 2, 3), G, P["stem_g"], P["stem_b"]))
    x = max_pool(x)
    cin = e.stem_ch
    for si, (c, nb) in enumerate(zip(e.widths, e.blocks)):
        for bi in range(nb):
            p = f"s{si}b{bi}."
            stride = 2 if (si > 0 and bi == 0) else 1
            y = relu(group_norm(conv2d(x, P[p + "a"], stride, 1), G, P[p + "a_g"], P[p + "a_b"]))
            y = group_norm(conv2d(y, P[p + "b"], 1, 1), G, P[p + "b_g"], P[p + "b_b"])
            if (p + "d") in P:
                s = group_norm(conv2d(x, P[p + "d"], stride, 0), G, P[p + "d_g"], P[p + "d_b"])
            else:
                s = x
            x = relu(y + s)
            cin = c
    return x.mean(axis=(1, 2))


def conv_flops(e, batch: int) -> int:
    """2 FLOPs per multiply-add of every convolution (the encoder's matrix
    work; normalisation and pooling are not counted)."""
    H, W = e.height, e.width
    tot = 0

    def out_hw(h, w, k, s, p):
        return (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1

    h, w = out_hw(H, W, 7, 2, 3)
    tot += 2 * h * w * e.stem_ch * 49 * e.in_ch
    h, w = out_hw(h, w, 3, 2, 1)
    cin = e.stem_ch
    for si, (c, nb) in enumerate(zip(e.widths, e.blocks)):
        for bi in range(nb):
            stride = 2 if (si > 0 and bi == 0) else 1
            ho, wo = out_hw(h, w, 3, stride, 1)
            tot += 2 * ho * wo * c * 9 * cin + 2 * ho * wo * c * 9 * c
            if stride != 1 or cin != c:
                tot += 2 * ho * wo * c * cin
            h, w, cin = ho, wo, c
    return tot * batch
