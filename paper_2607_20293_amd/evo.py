"""Python binding of libevo.so (ctypes).  Argument marshalling only: every
step of the denoising loop runs in the library's HIP kernels.  torch is used
for device memory (tensors' data pointers) and streams.

If the library is not built this module raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import sys
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libevo.so")

EVO_FP32, EVO_BF16 = 0, 1
GRAN_LAYER, GRAN_UNIT = 0, 1
COLD_COMPUTE, COLD_ZERO = 0, 1

CODE_EVAL, CODE_STORE, CODE_REUSE, CODE_MERGED = 1, 2, 4, 8

EXPORTED = ("evo_weight_count", "evo_check_desc", "evo_create_policy", "evo_set_schedule",
            "evo_set_schedule_pairs", "evo_denoise", "evo_get_stats", "evo_schedule_stats",
            "evo_schedule_codes", "evo_debug_read_cache", "evo_debug_team_withhold", "evo_synchronize", "evo_destroy_policy",
            "evo_last_error", "evo_collect_activations", "evo_redundancy_scores", "evo_guided_probabilities",
            "evo_guided_sample", "evo_ga_initial_population", "evo_ga_next_generation", "evo_ga_search",
            "evo_search", "evo_encoder_weight_count", "evo_create_encoder", "evo_encode", "evo_encoder_flops",
            "evo_destroy_encoder", "evo_set_kernel_timing", "evo_kernel_time", "evo_denoise_noalloc",
            "evo_noalloc_scratch_bytes")


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


class GAConfig(ctypes.Structure):
    """evo_ga_config (Sec. 3.2 / Sec. 4.1 defaults: population 30, 10 elites,
    30 generations)."""
    _fields_ = [("K", ctypes.c_int32), ("pop_size", ctypes.c_int32), ("n_elite", ctypes.c_int32),
                ("max_generations", ctypes.c_int32), ("tournament", ctypes.c_int32),
                ("n_guided", ctypes.c_int32), ("mutation_rate", ctypes.c_double), ("seed", ctypes.c_uint64)]

    @classmethod
    def make(cls, K, pop_size=30, n_elite=10, max_generations=30, tournament=2, n_guided=15,
             mutation_rate=0.05, seed=0):
        return cls(int(K), int(pop_size), int(n_elite), int(max_generations), int(tournament), int(n_guided),
                   float(mutation_rate), int(seed))


class SearchResult(ctypes.Structure):
    _fields_ = [("generations", ctypes.c_int32), ("evaluations", ctypes.c_int32), ("memo_hits", ctypes.c_int32),
                ("formal_evaluations", ctypes.c_int32), ("accepted", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("best_quick", ctypes.c_double), ("best_formal", ctypes.c_double)]

    def as_dict(self):
        return {n: (float(getattr(self, n)) if n.startswith("best") else int(getattr(self, n)))
                for n, _ in self._fields_ if n != "reserved"}


class SearchOptions(ctypes.Structure):
    _fields_ = [("granularity", ctypes.c_int32), ("n_quick", ctypes.c_int32), ("n_formal", ctypes.c_int32),
                ("tau", ctypes.c_float), ("q_base", ctypes.c_double), ("delta_acc", ctypes.c_double)]


QUICK_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                            ctypes.POINTER(ctypes.c_double))
FORMAL_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                             ctypes.POINTER(ctypes.c_double))


def _probs_ptr(probs, rows, T):
    if probs is None:
        return None, None
    pr = np.ascontiguousarray(np.asarray(probs, np.float64))
    if pr.size != rows * T:
        raise ValueError(f"probs must have {rows} x {T} entries")
    return pr, pr.ctypes.data


def ga_initial_population(cfg: GAConfig, rows: int, T: int, probs=None) -> np.ndarray:
    """Initial population int32 [pop_size][K] (sorted flat positions)."""
    pr, pp = _probs_ptr(probs, rows, T)
    out = np.zeros((cfg.pop_size, cfg.K), np.int32)
    _check(lib().evo_ga_initial_population(ctypes.byref(cfg), rows, T, pp, out.ctypes.data))
    return out


def ga_next_generation(cfg: GAConfig, rows: int, T: int, generation: int, pop, fitness) -> np.ndarray:
    pop = np.ascontiguousarray(np.asarray(pop, np.int32).reshape(cfg.pop_size, cfg.K))
    fit = np.ascontiguousarray(np.asarray(fitness, np.float64).reshape(cfg.pop_size))
    out = np.zeros_like(pop)
    _check(lib().evo_ga_next_generation(ctypes.byref(cfg), rows, T, int(generation), pop.ctypes.data,
                                        fit.ctypes.data, out.ctypes.data))
    return out


def _search_out(cfg, res, best, ph, fh):
    d = res.as_dict()
    g = d["generations"]
    d["best"] = best
    d["populations"] = ph[:g]
    d["fitness"] = fh[:g]
    return d


def ga_search(cfg: GAConfig, rows: int, T: int, quick, formal=None, probs=None, q_base: float = 1.0,
              delta_acc: float = 0.0) -> dict:
    """The host search loop with Python fitness callbacks: quick(int32
    [n][K]) -> n floats; formal(int32 [K]) -> float."""
    pr, pp = _probs_ptr(probs, rows, T)
    K = cfg.K
    err = []

    def _quick(user, n, sch, out):
        try:
            a = np.ctypeslib.as_array(sch, shape=(n, K)).copy()
            v = np.asarray(quick(a), np.float64).reshape(n)
            for i in range(n):
                out[i] = float(v[i])
            return 0
        except Exception as e:          # reported after the call returns
            err.append(e)
            return 1

    def _formal(user, sch, out):
        try:
            out[0] = float(formal(np.ctypeslib.as_array(sch, shape=(K,)).copy()))
            return 0
        except Exception as e:
            err.append(e)
            return 1

    qf = QUICK_FN(_quick)
    ff = FORMAL_FN(_formal) if formal is not None else FORMAL_FN()
    res = SearchResult()
    best = np.zeros(K, np.int32)
    ph = np.zeros((cfg.max_generations, cfg.pop_size, K), np.int32)
    fh = np.zeros((cfg.max_generations, cfg.pop_size), np.float64)
    rc = lib().evo_ga_search(ctypes.byref(cfg), rows, T, pp, qf, ff, None, float(q_base), float(delta_acc),
                             ctypes.byref(res), best.ctypes.data, ph.ctypes.data, fh.ctypes.data)
    if err:
        raise err[0]
    _check(rc)
    return _search_out(cfg, res, best, ph, fh)


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
        L.evo_debug_team_withhold.argtypes = [P, I32]
        L.evo_debug_team_withhold.restype = ctypes.c_int
        L.evo_collect_activations.argtypes = [P, I32, P, P, P, P, P, P]
        L.evo_collect_activations.restype = ctypes.c_int
        L.evo_redundancy_scores.argtypes = [P, I32, P, P, P]
        L.evo_redundancy_scores.restype = ctypes.c_int
        L.evo_guided_probabilities.argtypes = [P, I32, I32, ctypes.c_double, ctypes.c_double, P]
        L.evo_guided_probabilities.restype = ctypes.c_int
        L.evo_guided_sample.argtypes = [P, I32, I32, I32, P, P]
        L.evo_guided_sample.restype = ctypes.c_int
        L.evo_ga_initial_population.argtypes = [ctypes.POINTER(GAConfig), I32, I32, P, P]
        L.evo_ga_initial_population.restype = ctypes.c_int
        L.evo_ga_next_generation.argtypes = [ctypes.POINTER(GAConfig), I32, I32, I32, P, P, P]
        L.evo_ga_next_generation.restype = ctypes.c_int
        L.evo_ga_search.argtypes = [ctypes.POINTER(GAConfig), I32, I32, P, QUICK_FN, FORMAL_FN, P,
                                    ctypes.c_double, ctypes.c_double, ctypes.POINTER(SearchResult), P, P, P]
        L.evo_ga_search.restype = ctypes.c_int
        L.evo_search.argtypes = [P, ctypes.POINTER(GAConfig), ctypes.POINTER(SearchOptions), P, P, P, P, P,
                                 ctypes.POINTER(SearchResult), P, P, P, P]
        L.evo_search.restype = ctypes.c_int
        L.evo_denoise_noalloc.argtypes = [P, I32, P, P, P, P, P]
        L.evo_denoise_noalloc.restype = ctypes.c_int
        L.evo_noalloc_scratch_bytes.argtypes = []
        L.evo_noalloc_scratch_bytes.restype = ctypes.c_size_t
        L.evo_set_kernel_timing.argtypes = [P, I32]
        L.evo_set_kernel_timing.restype = ctypes.c_int
        L.evo_kernel_time.argtypes = [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
        L.evo_kernel_time.restype = ctypes.c_int
        L.evo_synchronize.argtypes = [P]
        L.evo_synchronize.restype = ctypes.c_int
        L.evo_destroy_policy.argtypes = [P]
        L.evo_destroy_policy.restype = None
        L.evo_encoder_weight_count.argtypes = [ctypes.POINTER(EncoderDesc)]
        L.evo_encoder_weight_count.restype = ctypes.c_int64
        L.evo_create_encoder.argtypes = [ctypes.POINTER(EncoderDesc), P, ctypes.c_size_t, ctypes.POINTER(P)]
        L.evo_create_encoder.restype = ctypes.c_int
        L.evo_encode.argtypes = [P, I32, P, P, I32, P]
        L.evo_encode.restype = ctypes.c_int
        L.evo_encoder_flops.argtypes = [P, I32, ctypes.POINTER(U64)]
        L.evo_encoder_flops.restype = ctypes.c_int
        L.evo_destroy_encoder.argtypes = [P]
        L.evo_destroy_encoder.restype = None
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
        # at interpreter shutdown the HIP runtime may already be torn down:
        # release nothing then (the process is ending)
        if sys is None or sys.is_finalizing():
            return
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

    def denoise_noalloc(self, obs, noise, ids, out, stream=None):
        """evo_denoise_noalloc: as denoise with a caller-provided out, the
        working data in the device's fixed scratch array (nothing is
        allocated by the library)."""
        import torch
        s = self.shape
        B = int(obs.shape[0])
        po = _dev_ptr(obs, "float32", (B, s.n_obs, s.obs_dim))
        pn = _dev_ptr(noise, "float32", (s.n_steps, B, s.horizon, s.action_dim))
        pout = _dev_ptr(out, "float32", (B, s.horizon, s.action_dim))
        ids_np = None if ids is None else np.ascontiguousarray(np.asarray(ids, np.int32))
        if ids_np is not None and ids_np.shape != (B,):
            raise ValueError("ids must have shape [B]")
        st = torch.cuda.current_stream(obs.device) if stream is None else stream
        _check(lib().evo_denoise_noalloc(self._h, B, po, pn, None if ids_np is None else ids_np.ctypes.data, pout,
                                         ctypes.c_void_p(st.cuda_stream)))
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

    def search(self, cfg: GAConfig, obs_quick, noise_quick, obs_formal=None, noise_formal=None, probs=None,
               granularity: int = GRAN_UNIT, tau: float = 0.1, q_base: float = 1.0, delta_acc: float = 0.0,
               stream=None) -> dict:
        """evo_search: GA over fixed-budget schedules with the GPU fitness
        (fraction of episodes whose chunk stays within tau of the uncached
        chunk).  obs/noise: HIP tensors as for denoise with n_quick / n_formal
        episodes.  Returns the result fields, 'best' (flat positions) and the
        per-generation 'populations' and 'fitness'."""
        import torch
        s = self.shape
        nq = int(obs_quick.shape[0])
        pq = _dev_ptr(obs_quick, "float32", (nq, s.n_obs, s.obs_dim))
        pnq = _dev_ptr(noise_quick, "float32", (s.n_steps, nq, s.horizon, s.action_dim))
        nf, pf, pnf = 0, None, None
        if obs_formal is not None:
            nf = int(obs_formal.shape[0])
            pf = _dev_ptr(obs_formal, "float32", (nf, s.n_obs, s.obs_dim))
            pnf = _dev_ptr(noise_formal, "float32", (s.n_steps, nf, s.horizon, s.action_dim))
        rows = 3 * s.n_layers if granularity == GRAN_UNIT else s.n_layers
        pr, pp = _probs_ptr(probs, rows, s.n_steps)
        opt = SearchOptions(int(granularity), nq, nf, float(tau), float(q_base), float(delta_acc))
        res = SearchResult()
        K = cfg.K
        best = np.zeros(K, np.int32)
        ph = np.zeros((cfg.max_generations, cfg.pop_size, K), np.int32)
        fh = np.zeros((cfg.max_generations, cfg.pop_size), np.float64)
        st = torch.cuda.current_stream(obs_quick.device) if stream is None else stream
        _check(lib().evo_search(self._h, ctypes.byref(cfg), ctypes.byref(opt), pq, pnq, pf, pnf, pp,
                                ctypes.byref(res), best.ctypes.data, ph.ctypes.data, fh.ctypes.data,
                                ctypes.c_void_p(st.cuda_stream)))
        return _search_out(cfg, res, best, ph, fh)

    def set_kernel_timing(self, enable: bool = True):
        """Record timing events around every later denoising-kernel launch."""
        _check(lib().evo_set_kernel_timing(self._h, 1 if enable else 0))

    def kernel_time(self):
        """(summed ms, launches) of the denoising kernel since the last call."""
        ms, n = ctypes.c_double(), ctypes.c_int64()
        _check(lib().evo_kernel_time(self._h, ctypes.byref(ms), ctypes.byref(n)))
        return float(ms.value), int(n.value)

    def synchronize(self):
        """Wait for the last denoise call; raise if its kernel reported a
        device-side failure (a timed-out team barrier)."""
        _check(lib().evo_synchronize(self._h))

    def stats(self) -> dict:
        st = Stats()
        _check(lib().evo_get_stats(self._h, ctypes.byref(st)))
        return st.as_dict()

    def debug_team_withhold(self, enable: bool) -> None:
        """Test hook: team member 0 of later calls withholds its partials
        (their waits time out; outputs invalid)."""
        _check(lib().evo_debug_team_withhold(self._h, 1 if enable else 0))

    def read_cache(self, unit: int, sample: int) -> np.ndarray:
        buf = np.zeros((self.shape.horizon, self.shape.d_model), np.float32)
        _check(lib().evo_debug_read_cache(self._h, unit, sample, buf.ctypes.data))
        return buf


class EncoderDesc(ctypes.Structure):
    _fields_ = [("height", ctypes.c_int32), ("width", ctypes.c_int32), ("in_ch", ctypes.c_int32),
                ("stem_ch", ctypes.c_int32), ("n_stages", ctypes.c_int32), ("widths", ctypes.c_int32 * 4),
                ("blocks", ctypes.c_int32 * 4), ("gn_group", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("max_batch", ctypes.c_int32)]


def make_encoder_desc(e, dtype: str = "bf16", max_batch: int = 1) -> EncoderDesc:
    """e: an encoder shape with height, width, in_ch, stem_ch, widths, blocks,
    gn_group (at most 4 stages)."""
    n = len(e.widths)
    if n != len(e.blocks) or not 1 <= n <= 4:
        raise ValueError("widths and blocks must have the same length, 1 to 4")
    w = (ctypes.c_int32 * 4)(*(list(e.widths) + [0] * (4 - n)))
    b = (ctypes.c_int32 * 4)(*(list(e.blocks) + [0] * (4 - n)))
    return EncoderDesc(e.height, e.width, e.in_ch, e.stem_ch, n, w, b, e.gn_group,
                       EVO_BF16 if dtype == "bf16" else EVO_FP32, max_batch)


def encoder_weight_count(desc: EncoderDesc) -> int:
    n = lib().evo_encoder_weight_count(ctypes.byref(desc))
    if n < 0:
        _check(int(n))
    return int(n)


class Encoder:
    """A created observation encoder on the current HIP device (see
    include/evo.h)."""

    def __init__(self, e, weights: np.ndarray, dtype: str = "bf16", max_batch: int = 1):
        self.shape = e
        self.out_dim = int(e.widths[-1])
        self.desc = make_encoder_desc(e, dtype, max_batch)
        w = np.ascontiguousarray(weights, dtype=np.float32)
        h = ctypes.c_void_p()
        _check(lib().evo_create_encoder(ctypes.byref(self.desc), w.ctypes.data, w.size, ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            lib().evo_destroy_encoder(self._h)
            self._h = None

    def __del__(self):
        # at interpreter shutdown the HIP runtime may already be torn down:
        # release nothing then (the process is ending)
        if sys is None or sys.is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass

    def encode(self, images, out=None, stream=None):
        """images: float32 HIP tensor [B][height][width][in_ch].  out: None, or
        a float32 HIP tensor [B][out_dim] whose rows may be strided (e.g. a
        column slice of the policy's observation rows).  Returns out."""
        import torch
        e = self.shape
        B = int(images.shape[0])
        pi = _dev_ptr(images, "float32", (B, e.height, e.width, e.in_ch))
        if out is None:
            out = torch.empty((B, self.out_dim), dtype=torch.float32, device=images.device)
        if not isinstance(out, torch.Tensor) or not out.is_cuda or out.dtype != torch.float32:
            raise TypeError("out must be a float32 HIP tensor")
        if tuple(out.shape) != (B, self.out_dim) or out.stride(1) != 1 or (B > 1 and out.stride(0) < self.out_dim):
            raise ValueError(f"out must be [{B}][{self.out_dim}] with unit column stride")
        row = out.stride(0) if B > 1 else self.out_dim
        st = torch.cuda.current_stream(images.device) if stream is None else stream
        _check(lib().evo_encode(self._h, B, pi, out.data_ptr(), row, ctypes.c_void_p(st.cuda_stream)))
        return out

    def flops(self, batch: int) -> int:
        v = ctypes.c_uint64()
        _check(lib().evo_encoder_flops(self._h, batch, ctypes.byref(v)))
        return int(v.value)
