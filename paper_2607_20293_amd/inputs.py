"""Seeded synthetic inputs for the cached denoising loop: shapes, weights,
observations, noise and refresh lattices.

This module is shared by the CPU oracle's tests and by the GPU path's tests
and benchmark.  It holds no arithmetic of the method itself: it only draws
random numbers and lays them out.  Nothing here may depend on the oracle or
on the HIP library.

Workload shapes stand in for the paper's manipulation benchmarks (RoboMimic,
Push-T, Block Push, Kitchen; Sec. 4.1), whose data and checkpoints are not
available: every tensor is synthetic, drawn from the seeds below.

Seed streams (numpy ``default_rng`` with a sequence seed):
  [seed, 0]     weights, in the flat order of ``weight_layout``
  [seed, 1]     observation features, N(0, 1)
  [seed, 2]     sampler noise, N(0, 1)
  [seed, 3, j]  refresh lattice j
  [seed, 4]     sample -> schedule assignment
  [seed, 5]     observation-encoder weights
  [seed, 6]     images
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, List, Tuple

import numpy as np


@dataclass(frozen=True)
class PolicyShape:
    """Shape of a transformer diffusion policy (decoder-only denoiser with
    cross-attention to observation tokens), Sec. 3.1: an L-layer decoder
    whose self-attention, cross-attention and feed-forward residual branches
    are the B = 3L cacheable units."""
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    horizon: int
    action_dim: int
    n_obs: int
    obs_dim: int
    n_steps: int

    @property
    def n_units(self) -> int:
        return 3 * self.n_layers

    @property
    def n_mem(self) -> int:
        # memory tokens: one diffusion-time token + the observation tokens
        return 1 + self.n_obs


@dataclass(frozen=True)
class Workload:
    name: str
    shape: PolicyShape
    batch: int
    dtype: str                      # "fp32" | "bf16"
    schedule: str                   # lattice recipe name
    density: float = 1.0
    n_schedules: int = 1
    samples_per_schedule: int = 0   # >0: per-sample schedule ids
    extra: Dict[str, object] = field(default_factory=dict)


TINY = PolicyShape(n_layers=2, d_model=64, n_heads=2, d_ff=256, horizon=8,
                   action_dim=2, n_obs=2, obs_dim=20, n_steps=10)
PUSHT = PolicyShape(n_layers=8, d_model=256, n_heads=4, d_ff=1024, horizon=16,
                    action_dim=2, n_obs=2, obs_dim=20, n_steps=100)
IMAGE = PolicyShape(n_layers=8, d_model=256, n_heads=4, d_ff=1024, horizon=16,
                    action_dim=10, n_obs=2, obs_dim=521, n_steps=100)
BIMANUAL = PolicyShape(n_layers=12, d_model=768, n_heads=12, d_ff=3072, horizon=32,
                       action_dim=14, n_obs=4, obs_dim=1024, n_steps=100)

# The five workloads.  Names describe what they are.
WORKLOADS: Dict[str, Workload] = {
    "tiny_fp32_b1": Workload("tiny_fp32_b1", TINY, 1, "fp32", "bernoulli", 0.5),
    "pusht_fp32_b1_all": Workload("pusht_fp32_b1_all", PUSHT, 1, "fp32", "all"),
    "pusht_fp32_b1_d25": Workload("pusht_fp32_b1_d25", PUSHT, 1, "fp32", "dirichlet", 0.25),
    "pusht_bf16_b1_d25": Workload("pusht_bf16_b1_d25", PUSHT, 1, "bf16", "dirichlet", 0.25),
    "pusht_bf16_b1_all": Workload("pusht_bf16_b1_all", PUSHT, 1, "bf16", "all"),
    "pusht_fp32_b64_d25": Workload("pusht_fp32_b64_d25", PUSHT, 64, "fp32", "dirichlet", 0.25),
    "pusht_bf16_b64_d25": Workload("pusht_bf16_b64_d25", PUSHT, 64, "bf16", "dirichlet", 0.25),
    "pusht_bf16_b64_all": Workload("pusht_bf16_b64_all", PUSHT, 64, "bf16", "all"),
    "image_bf16_b256_d12": Workload("image_bf16_b256_d12", IMAGE, 256, "bf16", "uniform", 0.125),
    "bimanual_bf16_b128_all": Workload("bimanual_bf16_b128_all", BIMANUAL, 128, "bf16", "all"),
    "bimanual_bf16_b128_d20": Workload("bimanual_bf16_b128_d20", BIMANUAL, 128, "bf16", "uniform", 0.20),
    "population_bf16_b512": Workload("population_bf16_b512", PUSHT, 512, "bf16", "population",
                                     n_schedules=64, samples_per_schedule=8),
}


# --------------------------------------------------------------------------
# weights
# --------------------------------------------------------------------------
def weight_layout(s: PolicyShape) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Flat parameter order: (name, shape, kind).  kind is one of
    'mat' (projection / positional table), 'bias', 'ln_g', 'ln_b'.
    Linear layers are stored [out][in]."""
    d, A, H, S = s.d_model, s.action_dim, s.horizon, s.n_mem
    out: List[Tuple[str, Tuple[int, ...], str]] = [
        ("W_in", (d, A), "mat"), ("b_in", (d,), "bias"),
        ("P_act", (H, d), "mat"),
        ("W_obs", (d, s.obs_dim), "mat"), ("b_obs", (d,), "bias"),
        ("P_mem", (S, d), "mat"),
    ]
    for l in range(s.n_layers):
        p = f"l{l}."
        out += [
            (p + "ln1_g", (d,), "ln_g"), (p + "ln1_b", (d,), "ln_b"),
            (p + "W_qkv", (3 * d, d), "mat"), (p + "b_qkv", (3 * d,), "bias"),
            (p + "W_o", (d, d), "mat"), (p + "b_o", (d,), "bias"),
            (p + "ln2_g", (d,), "ln_g"), (p + "ln2_b", (d,), "ln_b"),
            (p + "W_q", (d, d), "mat"), (p + "b_q", (d,), "bias"),
            (p + "W_kv", (2 * d, d), "mat"), (p + "b_kv", (2 * d,), "bias"),
            (p + "W_o2", (d, d), "mat"), (p + "b_o2", (d,), "bias"),
            (p + "ln3_g", (d,), "ln_g"), (p + "ln3_b", (d,), "ln_b"),
            (p + "W_1", (s.d_ff, d), "mat"), (p + "b_1", (s.d_ff,), "bias"),
            (p + "W_2", (d, s.d_ff), "mat"), (p + "b_2", (d,), "bias"),
        ]
    out += [("lnf_g", (d,), "ln_g"), ("lnf_b", (d,), "ln_b"),
            ("W_out", (A, d), "mat"), ("b_out", (A,), "bias")]
    return out


def n_weight_floats(s: PolicyShape) -> int:
    return int(sum(int(np.prod(shp)) for _, shp, _ in weight_layout(s)))


def make_weights(s: PolicyShape, seed: int = 0, variant: str = "default",
                 std: float = 0.02) -> np.ndarray:
    """Flat float32 parameter vector in ``weight_layout`` order.

    variant 'default': matrices and positional tables N(0, std^2), biases 0,
    LayerNorm gain 1 and shift 0.
    variant 'perturbed': additionally biases and LN shifts N(0, std^2) and
    LN gains 1 + N(0, std^2), so that every affine path carries signal.
    variant 'wide': as 'perturbed' with std scaled by 5 for matrices (larger
    activations, stronger attention contrast).
    """
    rng = np.random.default_rng([seed, 0])
    out = np.empty(n_weight_floats(s), np.float32)
    mstd = np.float32(std * (5.0 if variant == "wide" else 1.0))
    off = 0
    for _, shp, kind in weight_layout(s):
        n = int(np.prod(shp))
        v = out[off:off + n]
        off += n
        if kind == "mat":
            rng.standard_normal(out=v, dtype=np.float32)
            v *= mstd
        elif variant == "default":
            v[:] = 1.0 if kind == "ln_g" else 0.0
        else:
            rng.standard_normal(out=v, dtype=np.float32)
            v *= np.float32(std)
            if kind == "ln_g":
                v += np.float32(1.0)
    return out


def split_weights(s: PolicyShape, flat: np.ndarray) -> Dict[str, np.ndarray]:
    """Named views of the flat vector (no arithmetic)."""
    out, off = {}, 0
    for name, shp, _ in weight_layout(s):
        n = int(np.prod(shp))
        out[name] = flat[off:off + n].reshape(shp)
        off += n
    assert off == flat.size
    return out


# --------------------------------------------------------------------------
# observations and noise
# --------------------------------------------------------------------------
def make_obs(s: PolicyShape, batch: int, seed: int = 0) -> np.ndarray:
    """[batch][n_obs][obs_dim] float32, N(0,1)."""
    rng = np.random.default_rng([seed, 1])
    return rng.standard_normal((batch, s.n_obs, s.obs_dim), dtype=np.float32)


def make_noise(s: PolicyShape, batch: int, seed: int = 0) -> np.ndarray:
    """[n_steps][batch][horizon][action_dim] float32, N(0,1).
    Slice 0 is the initial sample x_T; slice t+1 is the noise added after
    reverse step t (the last slice that is read is n_steps-1)."""
    rng = np.random.default_rng([seed, 2])
    return rng.standard_normal((s.n_steps, batch, s.horizon, s.action_dim), dtype=np.float32)


# --------------------------------------------------------------------------
# refresh lattices (uint8 [rows][n_steps], rows = L (layer) or 3L (unit))
# --------------------------------------------------------------------------
def lattice_all(rows: int, T: int) -> np.ndarray:
    return np.ones((rows, T), np.uint8)


def lattice_bernoulli(rows: int, T: int, p: float, rng) -> np.ndarray:
    lat = (rng.random((rows, T)) < p).astype(np.uint8)
    lat[:, 0] = 1
    return lat


def lattice_uniform_k(rows: int, T: int, K: int, rng) -> np.ndarray:
    """Exactly K refreshes: step 0 of every row, the other K-rows drawn
    uniformly without replacement from the rows x (T-1) later positions."""
    assert rows <= K <= rows * T
    lat = np.zeros((rows, T), np.uint8)
    lat[:, 0] = 1
    pick = rng.choice(rows * (T - 1), size=K - rows, replace=False)
    lat[pick // (T - 1), 1 + pick % (T - 1)] = 1
    return lat


def lattice_dirichlet_k(rows: int, T: int, K: int, rng) -> np.ndarray:
    """Exactly K refreshes, step 0 forced; per-row shares of the remaining
    K-rows drawn from Dirichlet(1), rounded by largest remainder, capped at
    T-1 per row (overflow handed to rows with room, largest share first);
    each row's steps drawn without replacement from 1..T-1."""
    assert rows <= K <= rows * T
    extra = K - rows
    w = rng.dirichlet(np.ones(rows))
    raw = w * extra
    cnt = np.floor(raw).astype(np.int64)
    rem = extra - int(cnt.sum())
    order = np.argsort(-(raw - cnt), kind="stable")
    cnt[order[:rem]] += 1
    cap = T - 1
    over = int(np.maximum(cnt - cap, 0).sum())
    cnt = np.minimum(cnt, cap)
    for r in np.argsort(-w, kind="stable"):
        if over == 0:
            break
        room = cap - int(cnt[r])
        take = min(room, over)
        cnt[r] += take
        over -= take
    assert int(cnt.sum()) == extra
    lat = np.zeros((rows, T), np.uint8)
    lat[:, 0] = 1
    for r in range(rows):
        steps = rng.choice(np.arange(1, T), size=int(cnt[r]), replace=False)
        lat[r, steps] = 1
    return lat


def lattice_fixed_interval(rows: int, T: int, M: int) -> np.ndarray:
    """The comparison schedule the paper attributes to EfficientVLA (Sec. 1,
    Sec. 4.1): every unit refreshed synchronously, M times per query at a
    fixed interval: steps floor(i * T / M), i = 0 .. M-1 (step 0 included)."""
    assert 1 <= M <= T
    lat = np.zeros((rows, T), np.uint8)
    lat[:, [(i * T) // M for i in range(M)]] = 1
    return lat


def lattice_blockwise_budget(rows: int, T: int, M: int, rng) -> np.ndarray:
    """A block-wise fixed budget (the search space the paper attributes to
    BAC, Sec. 2): exactly M refreshes per unit, step 0 and M-1 further steps
    drawn without replacement per unit."""
    assert 1 <= M <= T
    lat = np.zeros((rows, T), np.uint8)
    lat[:, 0] = 1
    for r in range(rows):
        lat[r, rng.choice(np.arange(1, T), size=M - 1, replace=False)] = 1
    return lat


def read_printed_schedules(path: str) -> Dict[str, Dict[str, List[int]]]:
    """{method: {unit name: [steps]}} from a text file of printed refresh
    schedules, one line per (unit, method): unit name, method, comma-separated
    refreshed steps."""
    out: Dict[str, Dict[str, List[int]]] = {}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            steps = [int(x) for x in parts[2].split(",")] if len(parts) > 2 else []
            out.setdefault(parts[1], {})[parts[0]] = steps
    return out


def printed_lattice(path: str, method: str, n_layers: int, T: int) -> np.ndarray:
    """Unit-granular lattice [3L][T] (rows layer-major SA, CA, FFN) of one
    method's printed schedule."""
    sch = read_printed_schedules(path)[method]
    lat = np.zeros((3 * n_layers, T), np.uint8)
    for l in range(n_layers):
        for u, nm in enumerate(("SA", "CA", "FFN")):
            for t in sch[f"layers.{l}.{nm}"]:
                lat[3 * l + u, t] = 1
    return lat


def make_lattice(kind: str, rows: int, T: int, density: float, seed: int, j: int = 0) -> np.ndarray:
    rng = np.random.default_rng([seed, 3, j])
    if kind == "all":
        return lattice_all(rows, T)
    if kind == "bernoulli":
        return lattice_bernoulli(rows, T, density, rng)
    K = int(round(density * rows * T))
    if kind == "uniform":
        return lattice_uniform_k(rows, T, K, rng)
    if kind == "dirichlet":
        return lattice_dirichlet_k(rows, T, K, rng)
    raise ValueError(kind)


def population_lattices(rows: int, T: int, n: int, seed: int,
                        lo: float = 0.10, hi: float = 0.40) -> List[np.ndarray]:
    """n Dirichlet lattices at densities spread uniformly over [lo, hi]."""
    out = []
    for j in range(n):
        rho = lo + (hi - lo) * j / max(n - 1, 1)
        K = int(round(rows * T * rho))
        out.append(lattice_dirichlet_k(rows, T, max(K, rows), np.random.default_rng([seed, 3, j])))
    return out


def population_ids(n_sched: int, per: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng([seed, 4])
    ids = np.repeat(np.arange(n_sched, dtype=np.int32), per)
    rng.shuffle(ids)
    return ids


@dataclass
class Inputs:
    workload: Workload
    weights: np.ndarray
    obs: np.ndarray
    noise: np.ndarray
    lattices: List[np.ndarray]      # layer-granular [L][T] uint8
    ids: np.ndarray                 # int32 [batch]


def make_inputs(w: Workload, seed: int = 0, batch: int | None = None,
                variant: str = "default") -> Inputs:
    s = w.shape
    B = w.batch if batch is None else batch
    weights = make_weights(s, seed, variant)
    obs = make_obs(s, B, seed)
    noise = make_noise(s, B, seed)
    if w.schedule == "population":
        lats = population_lattices(s.n_layers, s.n_steps, w.n_schedules, seed)
        ids = population_ids(w.n_schedules, w.samples_per_schedule, seed)
        if B != ids.size:
            ids = ids[:B] if B < ids.size else np.resize(ids, B)
    else:
        lats = [make_lattice(w.schedule, s.n_layers, s.n_steps, w.density, seed)]
        ids = np.zeros(B, np.int32)
    return Inputs(w, weights, obs, noise, lats, ids.astype(np.int32))


def with_batch(w: Workload, batch: int) -> Workload:
    return replace(w, batch=batch)


# --------------------------------------------------------------------------
# observation encoder (images -> the visual part of an observation token)
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class EncoderShape:
    """A ResNet-18-topology image encoder with GroupNorm and global average
    pooling: a 7x7 stride-2 stem convolution, 3x3 stride-2 max pooling, then
    stages of basic blocks (two 3x3 convolutions and a shortcut; the first
    block of stages 2.. halves the resolution and projects the shortcut with
    a 1x1 stride-2 convolution).  GroupNorm uses groups of `gn_group`
    channels.  Images are NHWC [N][height][width][in_ch]."""
    height: int
    width: int
    in_ch: int = 3
    stem_ch: int = 64
    widths: Tuple[int, ...] = (64, 128, 256, 512)
    blocks: Tuple[int, ...] = (2, 2, 2, 2)
    gn_group: int = 16

    @property
    def out_dim(self) -> int:
        return self.widths[-1]


ENC_PUSHT = EncoderShape(96, 96)                # Push-T camera images
ENC_ROBOMIMIC = EncoderShape(84, 84)            # RoboMimic camera images
ENC_TINY = EncoderShape(20, 20, stem_ch=16, widths=(16, 32, 32, 64), blocks=(1, 1, 1, 1), gn_group=8)


def encoder_layout(e: EncoderShape) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Flat parameter order: (name, shape, kind), kind 'conv' ([out][kh][kw][in])
    or 'gn_g' / 'gn_b'.  Blocks are named s<stage>b<block>: conv a, conv b and,
    where the shortcut changes shape, conv d."""
    out: List[Tuple[str, Tuple[int, ...], str]] = [
        ("stem", (e.stem_ch, 7, 7, e.in_ch), "conv"),
        ("stem_g", (e.stem_ch,), "gn_g"), ("stem_b", (e.stem_ch,), "gn_b")]
    cin = e.stem_ch
    for si, (c, nb) in enumerate(zip(e.widths, e.blocks)):
        for bi in range(nb):
            p = f"s{si}b{bi}."
            stride = 2 if (si > 0 and bi == 0) else 1
            out += [(p + "a", (c, 3, 3, cin), "conv"), (p + "a_g", (c,), "gn_g"), (p + "a_b", (c,), "gn_b"),
                    (p + "b", (c, 3, 3, c), "conv"), (p + "b_g", (c,), "gn_g"), (p + "b_b", (c,), "gn_b")]
            if stride != 1 or cin != c:
                out += [(p + "d", (c, 1, 1, cin), "conv"), (p + "d_g", (c,), "gn_g"), (p + "d_b", (c,), "gn_b")]
            cin = c
    return out


def n_encoder_floats(e: EncoderShape) -> int:
    return int(sum(int(np.prod(shp)) for _, shp, _ in encoder_layout(e)))


def make_encoder_weights(e: EncoderShape, seed: int = 0, variant: str = "default") -> np.ndarray:
    """Flat float32 encoder parameters (seed stream [seed, 5]): convolution
    weights N(0, 2 / fan_in); GroupNorm gain 1 and shift 0, or with
    'perturbed' gain 1 + N(0, 0.1^2) and shift N(0, 0.1^2)."""
    rng = np.random.default_rng([seed, 5])
    out = np.empty(n_encoder_floats(e), np.float32)
    off = 0
    for _, shp, kind in encoder_layout(e):
        n = int(np.prod(shp))
        v = out[off:off + n]
        off += n
        if kind == "conv":
            rng.standard_normal(out=v, dtype=np.float32)
            v *= np.float32(np.sqrt(2.0 / (shp[1] * shp[2] * shp[3])))
        elif variant == "default":
            v[:] = 1.0 if kind == "gn_g" else 0.0
        else:
            rng.standard_normal(out=v, dtype=np.float32)
            v *= np.float32(0.1)
            if kind == "gn_g":
                v += np.float32(1.0)
    return out


def split_encoder_weights(e: EncoderShape, flat: np.ndarray) -> Dict[str, np.ndarray]:
    out, off = {}, 0
    for name, shp, _ in encoder_layout(e):
        n = int(np.prod(shp))
        out[name] = flat[off:off + n].reshape(shp)
        off += n
    assert off == flat.size
    return out


def make_images(e: EncoderShape, batch: int, seed: int = 0) -> np.ndarray:
    """[batch][height][width][in_ch] float32 in [0, 1) (seed stream [seed, 6])."""
    rng = np.random.default_rng([seed, 6])
    return rng.random((batch, e.height, e.width, e.in_ch), dtype=np.float32)
