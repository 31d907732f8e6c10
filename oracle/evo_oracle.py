"""CPU fp64 oracle of the schedule-driven cached denoising loop of EVO
(arXiv 2607.20293, "Evolving Cache Schedules for Fast Diffusion Policy
Inference").

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
baseline may import this module.  It shares no code with the HIP library and
imports nothing from the product package; the product path never calls it.

What it computes, and where each piece comes from:

* Cached execution (Sec. 3.1, Eq. 1): every cacheable unit b keeps one cache
  c_b.  At a scheduled position (b, t) in S the unit's residual branch is
  evaluated, used and stored in c_b; at any other position the unit adds the
  residual it cached at its most recent refresh.  Caches are reset at the
  start of each action query (Sec. 3.1 and Sec. 3.4).
* Cacheable units (Sec. 3.1): the self-attention, cross-attention and
  feed-forward residual branches of every decoder layer, B = 3L units.
* Schedule (Eq. 2 / Eq. 3): a subset S of the unit x step lattice.
* Denoising steps (Sec. 3.1): T reverse steps, t = 0 is the first step from
  noise; the diffusion timestep of step t is k = T-1-t.
* Everything else (the denoiser layer, the sampler) is the unchanged policy
  (Sec. 3.1 end, Sec. 3.4).  The paper prints no dimensions or constants for
  it, so the model follows the readings listed in the design notes: pre-norm
  decoder layers (LayerNorm inside each branch, eps 1e-5), causal
  self-attention over the action tokens, unmasked cross-attention to memory
  tokens [time token; observation tokens] + learned positions, exact-erf GELU,
  sinusoidal time embedding, a final LayerNorm and linear head predicting
  epsilon, and a DDPM sampler with the squared-cosine beta schedule
  (s = 0.008, beta capped at 0.999), fixed-small posterior variance and x0
  clipping to [-1, 1].

Arithmetic is float64 throughout.  In 'bf16' mode the projection matrices
that the GPU path multiplies in bf16 (W_obs, W_qkv, W_o, W_q, W_kv, W_o2,
W_1, W_2) are first rounded to bf16 (round to nearest even); all other
parameters stay as given.  All randomness (initial sample and per-step
noise) is an input.

Every function here is pinned by a CPU test against something other than
itself (closed forms, special cases, brute force, torch's reference decoder
layer); see tests/test_oracle_pins.py.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np
from scipy.special import erf

GRAN_LAYER = 0
GRAN_UNIT = 1
COLD_COMPUTE = 0
COLD_ZERO = 1

SA, CA, FFN = 0, 1, 2
UNIT_NAMES = ("SA", "CA", "FFN")

BF16_MATS = ("W_obs", "W_qkv", "W_o", "W_q", "W_kv", "W_o2", "W_1", "W_2")


# ---------------------------------------------------------------------------
# elementary pieces of the unchanged policy
# ---------------------------------------------------------------------------
def to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned
    as float64.  bfloat16 keeps the top 16 bits of the IEEE float32 pattern."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    r = r.astype(np.uint32)
    nan = np.isnan(np.asarray(a, dtype=np.float32))
    r = np.where(nan, np.uint32(0x7FC00000), r)
    return r.view(np.float32).astype(np.float64)


def layer_norm(v: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """LayerNorm over the last axis with the population variance."""
    mu = v.mean(axis=-1, keepdims=True)
    var = ((v - mu) ** 2).mean(axis=-1, keepdims=True)
    return (v - mu) / np.sqrt(var + eps) * g + b


def gelu(v: np.ndarray) -> np.ndarray:
    """GELU with the exact Gaussian CDF: v * Phi(v)."""
    return v * 0.5 * (1.0 + erf(v / math.sqrt(2.0)))


def softmax(z: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(z, axis=axis, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=axis, keepdims=True)


def sinusoid(k: int, d: int) -> np.ndarray:
    """Sinusoidal embedding of the integer diffusion timestep k:
    [sin(k w_j) for j < d/2] ++ [cos(k w_j) for j < d/2],
    w_j = exp(-ln(1e4) * j / (d/2 - 1))."""
    half = d // 2
    w = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / (half - 1))
    a = float(k) * w
    return np.concatenate([np.sin(a), np.cos(a)])


def ddpm_table(T: int, s: float = 0.008, beta_cap: float = 0.999) -> Dict[str, np.ndarray]:
    """DDPM constants for a T-step squared-cosine schedule, indexed by the
    diffusion timestep i = 0..T-1.

    f(u) = cos^2(((u + s)/(1 + s)) * pi/2);
    beta_i = min(1 - f((i+1)/T) / f(i/T), beta_cap);
    alpha_i = 1 - beta_i;  abar_i = prod_{j<=i} alpha_j;  abar_prev_0 = 1.
    Posterior q(x_{i-1} | x_i, x0) (DDPM): mean = c0_i x0 + ct_i x_i with
    c0_i = sqrt(abar_prev_i) beta_i / (1 - abar_i) and
    ct_i = sqrt(alpha_i) (1 - abar_prev_i) / (1 - abar_i); the fixed-small
    variance is (1 - abar_prev_i)/(1 - abar_i) beta_i, floored at 1e-20.
    """
    def f(u):
        return math.cos((u + s) / (1.0 + s) * math.pi / 2.0) ** 2

    beta = np.array([min(1.0 - f((i + 1) / T) / f(i / T), beta_cap) for i in range(T)])
    alpha = 1.0 - beta
    abar = np.cumprod(alpha)
    abar_prev = np.concatenate([[1.0], abar[:-1]])
    c0 = np.sqrt(abar_prev) * beta / (1.0 - abar)
    ct = np.sqrt(alpha) * (1.0 - abar_prev) / (1.0 - abar)
    var = np.maximum((1.0 - abar_prev) / (1.0 - abar) * beta, 1e-20)
    return dict(beta=beta, alpha=alpha, abar=abar, abar_prev=abar_prev,
                c0=c0, ct=ct, sigma=np.sqrt(var))


def ddpm_step(x: np.ndarray, eps: np.ndarray, k: int, z: Optional[np.ndarray],
              tab: Dict[str, np.ndarray], clip: bool = True) -> np.ndarray:
    """One reverse step at diffusion timestep k for an epsilon-predicting
    model: estimate x0, clip it, take the posterior mean, add sigma_k z
    unless k == 0."""
    abar = tab["abar"][k]
    x0 = (x - math.sqrt(1.0 - abar) * eps) / math.sqrt(abar)
    if clip:
        x0 = np.clip(x0, -1.0, 1.0)
    out = tab["c0"][k] * x0 + tab["ct"][k] * x
    if k > 0:
        out = out + tab["sigma"][k] * z
    return out


# ---------------------------------------------------------------------------
# the three residual branches (cacheable units, Sec. 3.1)
# ---------------------------------------------------------------------------
def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int,
              causal: bool) -> np.ndarray:
    """Multi-head scaled dot-product attention.  q: [..., Nq, d],
    k, v: [..., Nk, d]; head h uses columns h*dh .. (h+1)*dh-1; scale
    1/sqrt(dh); with causal=True query i sees keys j <= i."""
    d = q.shape[-1]
    dh = d // n_heads
    outs = []
    for hd in range(n_heads):
        sl = slice(hd * dh, (hd + 1) * dh)
        s = q[..., sl] @ np.swapaxes(k[..., sl], -1, -2) / math.sqrt(dh)
        if causal:
            nq, nk = s.shape[-2], s.shape[-1]
            mask = np.triu(np.ones((nq, nk), bool), k=1)
            s = np.where(mask, -np.inf, s)
        outs.append(softmax(s, axis=-1) @ v[..., sl])
    return np.concatenate(outs, axis=-1)


def self_attention_branch(h: np.ndarray, P: Dict[str, np.ndarray], l: int, n_heads: int) -> np.ndarray:
    """SA residual branch: W_o . causal_attn(LN1(h)) + b_o."""
    p = f"l{l}."
    x = layer_norm(h, P[p + "ln1_g"], P[p + "ln1_b"])
    qkv = x @ P[p + "W_qkv"].T + P[p + "b_qkv"]
    d = h.shape[-1]
    o = attention(qkv[..., :d], qkv[..., d:2 * d], qkv[..., 2 * d:], n_heads, causal=True)
    return o @ P[p + "W_o"].T + P[p + "b_o"]


def cross_attention_branch(h: np.ndarray, mem: np.ndarray, P: Dict[str, np.ndarray], l: int,
                           n_heads: int) -> np.ndarray:
    """CA residual branch: queries from LN2(h), keys/values from the memory
    tokens (not normalised), no mask."""
    p = f"l{l}."
    d = h.shape[-1]
    x = layer_norm(h, P[p + "ln2_g"], P[p + "ln2_b"])
    q = x @ P[p + "W_q"].T + P[p + "b_q"]
    kv = mem @ P[p + "W_kv"].T + P[p + "b_kv"]
    o = attention(q, kv[..., :d], kv[..., d:], n_heads, causal=False)
    return o @ P[p + "W_o2"].T + P[p + "b_o2"]


def feed_forward_branch(h: np.ndarray, P: Dict[str, np.ndarray], l: int) -> np.ndarray:
    """FFN residual branch: W_2 . GELU(W_1 . LN3(h) + b_1) + b_2."""
    p = f"l{l}."
    x = layer_norm(h, P[p + "ln3_g"], P[p + "ln3_b"])
    return gelu(x @ P[p + "W_1"].T + P[p + "b_1"]) @ P[p + "W_2"].T + P[p + "b_2"]


def unit_residual(b: int, h: np.ndarray, mem: np.ndarray, P, n_heads: int) -> np.ndarray:
    """r_{b,t}: residual output of unit b = 3l + u (u: 0 SA, 1 CA, 2 FFN)."""
    l, u = divmod(b, 3)
    if u == SA:
        return self_attention_branch(h, P, l, n_heads)
    if u == CA:
        return cross_attention_branch(h, mem, P, l, n_heads)
    return feed_forward_branch(h, P, l)


# ---------------------------------------------------------------------------
# schedules (Eq. 2 / Eq. 3) and the cold-cache reading
# ---------------------------------------------------------------------------
def expand_lattice(lat: np.ndarray, granularity: int, n_layers: int) -> np.ndarray:
    """Unit-level lattice [3L][T] bool.  A layer-granular row applies to the
    SA, CA and FFN units of that layer."""
    lat = np.asarray(lat)
    if granularity == GRAN_LAYER:
        assert lat.shape[0] == n_layers
        return np.repeat(lat.astype(bool), 3, axis=0)
    assert lat.shape[0] == 3 * n_layers
    return lat.astype(bool)


def pairs_to_lattice(pairs: Sequence[Sequence[int]], rows: int, T: int) -> np.ndarray:
    """Eq. 3: an individual is K unique (b, t) positions.  Duplicates or
    out-of-range positions are rejected."""
    lat = np.zeros((rows, T), np.uint8)
    for b, t in pairs:
        if not (0 <= b < rows and 0 <= t < T):
            raise ValueError("position out of range")
        if lat[b, t]:
            raise ValueError("duplicate position")
        lat[b, t] = 1
    return lat


def effective_lattice(unit_lat: np.ndarray, cold_policy: int) -> np.ndarray:
    """Positions actually refreshed.  A unit reused before its first refresh
    has no cached residual; with COLD_COMPUTE it is computed at step 0
    (S' = S u (B x {0})), with COLD_ZERO its empty cache contributes zero and
    S' = S."""
    eff = unit_lat.astype(bool).copy()
    if cold_policy == COLD_COMPUTE:
        eff[:, 0] = True
    return eff


# ---------------------------------------------------------------------------
# the cached denoising loop (Eq. 1)
# ---------------------------------------------------------------------------
def prepare_params(P: Dict[str, np.ndarray], dtype: str) -> Dict[str, np.ndarray]:
    out = {}
    for name, v in P.items():
        base = name.split(".")[-1]
        if dtype == "bf16" and base in BF16_MATS:
            out[name] = to_bf16(v)
        else:
            out[name] = np.asarray(v, dtype=np.float64)
    return out


def denoise_group(shape, P: Dict[str, np.ndarray], obs: np.ndarray, noise: np.ndarray,
                  eff: np.ndarray, clip: bool = True, cache: bool = True,
                  trace: Optional[dict] = None) -> np.ndarray:
    """Cached DDPM sampling for a group of samples that share one effective
    unit lattice ``eff`` [3L][T].  Samples never interact: every operation
    acts on each sample's own [H][d] rows.

    obs: [n][n_obs][obs_dim]; noise: [T][n][H][A] (slice 0 is x_T, slice t+1
    the noise added after step t).  P: fp64 parameters (prepare_params).
    With cache=False every unit is evaluated at every step (the uncached
    policy) and ``eff`` is ignored.
    trace (optional dict) receives 'r' [T][3L][n][H][d] of residuals used,
    'computed' [T][3L] bools, and 'eps' [T][n][H][A].
    """
    L, d, T = shape.n_layers, shape.d_model, shape.n_steps
    U = 3 * L
    tab = ddpm_table(T)
    obs = np.asarray(obs, np.float64)
    n = obs.shape[0]
    # observation tokens, once per action query
    m_obs = obs @ P["W_obs"].T + P["b_obs"]                       # [n][n_obs][d]
    x = np.asarray(noise[0], np.float64).copy()                  # [n][H][A]
    c = [None] * U                                                # caches reset per query
    if trace is not None:
        trace["r"] = np.zeros((T, U, n, shape.horizon, d))
        trace["computed"] = np.zeros((T, U), bool)
        trace["eps"] = np.zeros((T, n, shape.horizon, shape.action_dim))
    for t in range(T):
        k = T - 1 - t
        time_tok = sinusoid(k, d)
        mem = np.concatenate([np.broadcast_to(time_tok, (n, 1, d)), m_obs], axis=1) + P["P_mem"]
        h = x @ P["W_in"].T + P["b_in"] + P["P_act"]
        for b in range(U):
            if (not cache) or eff[b, t]:
                r = unit_residual(b, h, mem, P, shape.n_heads)
                c[b] = r
                if trace is not None:
                    trace["computed"][t, b] = True
            elif c[b] is not None:
                r = c[b]
            else:                                   # cold cache, COLD_ZERO reading
                r = np.zeros_like(h)
            if trace is not None:
                trace["r"][t, b] = r
            h = h + r
        eps = layer_norm(h, P["lnf_g"], P["lnf_b"]) @ P["W_out"].T + P["b_out"]
        if trace is not None:
            trace["eps"][t] = eps
        z = np.asarray(noise[t + 1], np.float64) if k > 0 else None
        x = ddpm_step(x, eps, k, z, tab, clip)
    return x


def denoise(shape, params: Dict[str, np.ndarray], obs: np.ndarray, noise: np.ndarray,
            lattices: List[np.ndarray], ids: np.ndarray, granularity: int = GRAN_LAYER,
            cold_policy: int = COLD_COMPUTE, clip: bool = True, dtype: str = "fp32",
            samples: Optional[Sequence[int]] = None):
    """Action chunks [B][H][A] (or for the listed ``samples`` only) and the
    integer bookkeeping of the call.  Sample n follows lattice ids[n]."""
    P = prepare_params(params, dtype)
    B = obs.shape[0]
    sel = list(range(B)) if samples is None else list(samples)
    effs = [effective_lattice(expand_lattice(lt, granularity, shape.n_layers), cold_policy)
            for lt in lattices]
    out = np.zeros((len(sel), shape.horizon, shape.action_dim))
    ids = np.asarray(ids)
    for sid in sorted(set(int(ids[n]) for n in sel)):
        pos = [i for i, n in enumerate(sel) if int(ids[n]) == sid]
        rows = [sel[i] for i in pos]
        out[pos] = denoise_group(shape, P, obs[rows], noise[:, rows], effs[sid], clip)
    stats = bookkeeping(shape, lattices, ids, granularity, cold_policy)
    return out, stats


# ---------------------------------------------------------------------------
# integer bookkeeping (Sec. 4.1 budgets; Tables 1-3 FLOPs)
# ---------------------------------------------------------------------------
def unit_flops(shape) -> Dict[str, int]:
    """Matmul FLOPs (2 per multiply-add) of one evaluation of each unit for
    one sample; attention score and value products counted dense."""
    H, d, S, dff = shape.horizon, shape.d_model, shape.n_mem, shape.d_ff
    return {
        "SA": 2 * (4 * H * d * d + 2 * H * H * d),
        "CA": 2 * (2 * H * d * d + 2 * S * d * d + 2 * H * S * d),
        "FFN": 2 * (2 * H * d * dff),
        "always_step": 4 * H * shape.action_dim * d,
        "always_query": 2 * shape.n_obs * shape.obs_dim * d,
    }


def bookkeeping(shape, lattices: List[np.ndarray], ids: np.ndarray,
                granularity: int = GRAN_LAYER, cold_policy: int = COLD_COMPUTE) -> Dict[str, int]:
    """Requested and effective unit refreshes and FLOP counts summed over the
    batch, as Python integers."""
    F = unit_flops(shape)
    per_type = [F["SA"], F["CA"], F["FFN"]]
    T, L = shape.n_steps, shape.n_layers
    req_n, eff_n, fl_n = [], [], []
    for lt in lattices:
        u = expand_lattice(lt, granularity, L)
        e = effective_lattice(u, cold_policy)
        req_n.append(int(u.sum()))
        eff_n.append(int(e.sum()))
        fl_n.append(sum(int(e[b].sum()) * per_type[b % 3] for b in range(3 * L)))
    req = eff = fc = 0
    for n in np.asarray(ids).tolist():
        req += req_n[n]
        eff += eff_n[n]
        fc += fl_n[n]
    B = len(ids)
    always = B * (T * F["always_step"] + F["always_query"])
    full = B * T * L * sum(per_type) + always
    return {"refreshes_requested": req, "refreshes_effective": eff,
            "flops_cacheable": fc, "flops_always": always, "flops_full": full}
