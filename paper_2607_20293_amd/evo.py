"""Python binding of libevo.so (ctypes).  Argument marshalling only: every
step of the denoising loop runs in the library's HIP kernels.  torch is used
for device memory (tensors' data pointers) and streams.

If the library is not built this module raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libevo.so")

EVO_FP32, EVO_BF16 = 0, 1
GRAN_LAYER, GRAN_UNIT = 0, 1
COLD_COMPUTE, COLD_ZERO = 0, 1

CODE_EVAL, CODE_STORE, CODE_REUSE, CODE_MERGED = 1, 2, 4, 8

EXPORTED = ("evo_weight_count", "evo_check_desc", "evo_create_policy", "evo_set_schedule",
            "evo_set_schedule_pairs", "evo_denoise", "evo_get_stats", "evo_schedule_stats",
            "evo_schedule_codes", "evo_debug_read_cache", "evo_synchronize", "evo_destroy_policy",
            "evo_last_error", "evo_collect_activations", "evo_redundancy_scores", "evo_guided_probabilities",
            "evo_guided_sample")


def guided_probabilities(scores, eps: float, gamma: float) -> np.ndarray:
    """Eq. 7 (host): scores [rows][T] -> probabilities (float64)."""
    sc = np.ascontiguousarray(np.asarray(scores, np.float32))
    rows, T = sc.shape
    out = np.zeros((rows, T), np.float64)
    _check(lib().evo_guided_probabilities(sc.ctypes.data, rows, T, float(eps), float(gamma), out.ctypes.data))
    return out


def guided_sample(probs, K: int, uniforms) -> np.ndarray:
    """K distinct (row, step) positions from probs [rows][T] with the given
    uniforms (same shape, in (0, 1)); int32 [K][2] in flat order."""
    pr = np.ascontiguousarray(np.asarray(probs, np.float64))
    u = np.ascontiguousarray(np.asarray(uniforms, np.float64))
    if u.shape != pr.shape:
        raise ValueError("uniforms must have the shape of probs")
    rows, T = pr.shape
    out = np.zeros((K, 2), np.int32)
    _check(lib().evo_guided_sample(pr.ctypes.data, rows, T, int(K), u.ctypes.data, out.ctypes.data))
    return out


class EvoError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"evo error {code}: {msg}")
        self.code = code


class PolicyDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "d_ff", "horizon", "action_dim",
        "n_obs_tokens", "obs_dim", "n_steps", "dtype", "cold_policy", "clip_sample",
        "max_batch", "max_schedules")]


class Stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "refreshes_requested", "refreshes_effective", "flops_cacheable", "flops_always",
        "flops_full", "flops_kernel", "cache_bytes_read", "cache_bytes_written",
        "weight_bytes", "n_tiles", "n_workgroups")]

    def as_dict(self):
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build()")
        # torch ships its own HIP runtime; loading it first makes the library
        # bind to that same runtime (one HIP runtime per process), so torch
        # tensors and streams are valid in the library's calls.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        P, I32, U64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64
        L.evo_weight_count.argtypes = [ctypes.POINTER(PolicyDesc)]
        L.evo_weight_count.restype = ctypes.c_int64
        L.evo_check_desc.argtypes = [ctypes.POINTER(PolicyDesc)]
        L.evo_check_desc.restype = ctypes.c_int
        L.evo_create_policy.argtypes = [ctypes.POINTER(PolicyDesc), P, ctypes.c_size_t, ctypes.POINTER(P)]
        L.evo_create_policy.restype = ctypes.c_int
        L.evo_set_schedule.argtypes = [P, I32, P, I32, I32, I32]
        L.evo_set_schedule.restype = ctypes.c_int
        L.evo_set_schedule_pairs.argtypes = [P, I32, P, I32, I32]
        L.evo_set_schedule_pairs.restype = ctypes.c_int
        L.evo_denoise.argtypes = [P, I32, P, P, P, P, P]
        L.evo_denoise.restype = ctypes.c_int
        L.evo_get_stats.argtypes = [P, ctypes.POINTER(Stats)]
        L.evo_get_stats.restype = ctypes.c_int
        L.evo_schedule_stats.argtypes = [ctypes.POINTER(PolicyDesc), P, I32, I32, I32, P, I32,
                                         ctypes.POINTER(Stats)]
        L.evo_schedule_stats.restype = ctypes.c_int
        L.evo_schedule_codes.argtypes = [ctypes.POINTER(PolicyDesc), P, I32, I32, P]
        L.evo_schedule_codes.restype = ctypes.c_int
        L.evo_debug_read_cache.argtypes = [P, I32, I32, P]
        L.evo_debug_read_cache.restype = ctypes.c_int
        L.evo_collect_activations.argtypes = [P, I32, P, P, P, P, P, P]
        L.evo_collect_activations.restype = ctypes.c_int
        L.evo_redundancy_scores.argtypes = [P, I32, P, P, P]
        L.evo_redundancy_scores.restype = ctypes.c_int
        L.evo_guided_probabilities.argtypes = [P, I32, I32, ctypes.c_double, ctypes.c_double, P]
        L.evo_guided_probabilities.restype = ctypes.c_int
        L.evo_guided_sample.argtypes = [P, I32, I32, I32, P, P]
        L.evo_guided_sample.restype = ctypes.c_int
        L.evo_synchronize.argtypes = [P]
        L.evo_synchronize.restype = ctypes.c_int
        L.evo_destroy_policy.argtypes = [P]
        L.evo_destroy_policy.restype = None
        L.evo_last_error.argtypes = []
        L.evo_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc: int):
    if rc != 0:
        raise EvoError(rc, lib().evo_last_error().decode(errors="replace"))


def make_desc(shape, dtype: str = "bf16", max_batch: int = 1, max_schedules: int = 1,
              cold_policy: int = COLD_COMPUTE, clip: bool = True) -> PolicyDesc:
    return PolicyDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.d_ff, shape.horizon,
                      shape.action_dim, shape.n_obs, shape.obs_dim, shape.n_steps,
                      EVO_BF16 if dtype == "bf16" else EVO_FP32, cold_policy, 1 if clip else 0,
                      max_batch, max_schedules)


def weight_count(desc: PolicyDesc) -> int:
    n = lib().evo_weight_count(ctypes.byref(desc))
    if n < 0:
        _check(int(n))
    return int(n)


def check_desc(desc: PolicyDesc) -> int:
    return lib().evo_check_desc(ctypes.byref(desc))


def _u8(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.uint8)


def schedule_stats(desc: PolicyDesc, lattices: Sequence[np.ndarray], ids, granularity: int) -> dict:
    lats = np.ascontiguousarray(np.stack([_u8(x) for x in lattices]))
    ids = np.ascontiguousarray(np.asarray(ids, np.int32))
    st = Stats()
    _check(lib().evo_schedule_stats(ctypes.byref(desc), lats.ctypes.data, lats.shape[0], lats.shape[1],
                                    granularity, ids.ctypes.data, ids.size, ctypes.byref(st)))
    return st.as_dict()


def schedule_codes(desc: PolicyDesc, lattice: np.ndarray, granularity: int) -> np.ndarray:
    lat = _u8(lattice)
    out = np.zeros((3 * desc.n_layers, desc.n_steps), np.uint8)
    _check(lib().evo_schedule_codes(ctypes.byref(desc), lat.ctypes.data, lat.shape[0], granularity,
                                    out.ctypes.data))
    return out


def _dev_ptr(t, dtype_name: str, shape) -> int:
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("expected a HIP device tensor")
    if t.dtype != getattr(torch, dtype_name):
        raise TypeError(f"expected {dtype_name}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"expected shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


class Policy:
    """A created policy on the current HIP device (see include/evo.h)."""

    def __init__(self, shape, weights: np.ndarray, dtype: str = "bf16", max_batch: int = 1,
                 max_schedules: int = 1, cold_policy: int = COLD_COMPUTE, clip: bool = True):
        self.shape = shape
        self.desc = make_desc(shape, dtype, max_batch, max_schedules, cold_policy, clip)
        w = np.ascontiguousarray(weights, dtype=np.float32)
        h = ctypes.c_void_p()
        _check(lib().evo_create_policy(ctypes.byref(self.desc), w.ctypes.data, w.size, ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            lib().evo_destroy_policy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_schedule(self, sid: int, lattice: np.ndarray, granularity: int = GRAN_LAYER):
        lat = _u8(lattice)
        if lat.ndim != 2:
            raise ValueError("lattice must be 2-D [rows][n_steps]")
        _check(lib().evo_set_schedule(self._h, sid, lat.ctypes.data, lat.shape[0], lat.shape[1], granularity))

    def set_schedule_pairs(self, sid: int, pairs, granularity: int = GRAN_UNIT):
        pr = np.ascontiguousarray(np.asarray(pairs, np.int32).reshape(-1, 2))
        _check(lib().evo_set_schedule_pairs(self._h, sid, pr.ctypes.data, pr.shape[0], granularity))

    def denoise(self, obs, noise, ids=None, out=None, stream=None, acts=None):
        """obs: float32 [B][n_obs][obs_dim], noise: float32 [T][B][H][A]
        (HIP tensors); ids: host int32 [B] or None.  Returns out [B][H][A].
        acts (optional HIP tensor [B][3L][T][H][d]) receives the residuals of
        the evaluated units (evo_collect_activations)."""
        import torch
        s = self.shape
        B = int(obs.shape[0])
        po = _dev_ptr(obs, "float32", (B, s.n_obs, s.obs_dim))
        pn = _dev_ptr(noise, "float32", (s.n_steps, B, s.horizon, s.action_dim))
        if out is None:
            out = torch.empty((B, s.horizon, s.action_dim), dtype=torch.float32, device=obs.device)
        pout = _dev_ptr(out, "float32", (B, s.horizon, s.action_dim))
        if ids is not None:
            ids_np = np.ascontiguousarray(np.asarray(ids, np.int32))
            if ids_np.shape != (B,):
                raise ValueError("ids must have shape [B]")
            pid = ids_np.ctypes.data
        else:
            ids_np, pid = None, None
        st = torch.cuda.current_stream(obs.device) if stream is None else stream
        if acts is None:
            _check(lib().evo_denoise(self._h, B, po, pn, pid, pout, ctypes.c_void_p(st.cuda_stream)))
        else:
            pa = _dev_ptr(acts, "float32", (B, 3 * s.n_layers, s.n_steps, s.horizon, s.d_model))
            _check(lib().evo_collect_activations(self._h, B, po, pn, pid, pout, pa, ctypes.c_void_p(st.cuda_stream)))
        return out

    def collect_activations(self, obs, noise, ids=None, stream=None):
        """denoise that also records every evaluated unit's residual:
        returns (out [B][H][A], acts [B][3L][T][H][d]) as HIP tensors."""
        import torch
        s = self.shape
        B = int(obs.shape[0])
        acts = torch.zeros((B, 3 * s.n_layers, s.n_steps, s.horizon, s.d_model), dtype=torch.float32,
                           device=obs.device)
        out = self.denoise(obs, noise, ids, stream=stream, acts=acts)
        return out, acts

    def redundancy_scores(self, acts, rollouts=None, stream=None):
        """Eq. 6 scores [3L][T] (HIP tensor) from acts [R][3L][T][H][d]."""
        import torch
        s = self.shape
        R = int(acts.shape[0]) if rollouts is None else int(rollouts)
        acts = acts.reshape(acts.shape[0], 3 * s.n_layers, s.n_steps, s.horizon, s.d_model)
        pa = _dev_ptr(acts, "float32", tuple(acts.shape))
        out = torch.empty((3 * s.n_layers, s.n_steps), dtype=torch.float32, device=acts.device)
        st = torch.cuda.current_stream(acts.device) if stream is None else stream
        _check(lib().evo_redundancy_scores(self._h, R, pa, out.data_ptr(), ctypes.c_void_p(st.cuda_stream)))
        return out

    def synchronize(self):
        """Wait for the last denoise call; raise if its kernel reported a
        device-side failure (a timed-out team barrier)."""
        _check(lib().evo_synchronize(self._h))

    def stats(self) -> dict:
        st = Stats()
        _check(lib().evo_get_stats(self._h, ctypes.byref(st)))
        return st.as_dict()

    def read_cache(self, unit: int, sample: int) -> np.ndarray:
        buf = np.zeros((self.shape.horizon, self.shape.d_model), np.float32)
        _check(lib().evo_debug_read_cache(self._h, unit, sample, buf.ctypes.data))
        return buf
