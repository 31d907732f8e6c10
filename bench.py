"""Benchmark of the cached denoising loop on one MI355X.

Headline: action chunks/s at batch 256 on the image-conditioned policy
(8 layers, d 256, horizon 16, action_dim 10, 2 obs tokens of 521 features,
100 DDPM steps, bf16) with one shared 12.5%-density layer lattice, plus the
p50 per-chunk latency at batch 1 on the Push-T-shaped policy with a
25%-density lattice.  A step is one evo_denoise call (the whole 100-step
cached loop for the batch), timed with inputs resident in HBM.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "action chunks/sec at batch 256 + p50 latency/chunk at batch 1, 25%-density schedule"
PEAK = {"bf16": 2500.0, "fp32": 157.3}           # dense MFMA TFLOP/s of MI355X
HBM_PEAK_GBS = 8000.0
COUNTERS = os.path.join(ROOT, "profiles", "denoise_kernel_counters.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_sha() -> str:
    h = hashlib.sha256()
    for f in ("evo_kernels.hip", "evo_kernels.hpp"):
        with open(os.path.join(ROOT, "paper_2607_20293_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


class Runner:
    def __init__(self, name, shape, weights, dtype, lattices, ids, obs, noise, gran=0):
        import torch
        from paper_2607_20293_amd import evo
        self.torch = torch
        self.name = name
        self.shape = shape
        self.B = obs.shape[0]
        self.pol = evo.Policy(shape, weights, dtype=dtype, max_batch=self.B, max_schedules=len(lattices))
        for j, lt in enumerate(lattices):
            self.pol.set_schedule(j, lt, gran)
        dev = torch.device("cuda:0")
        self.obs = torch.from_numpy(np.ascontiguousarray(obs)).to(dev)
        self.noise = torch.from_numpy(np.ascontiguousarray(noise)).to(dev)
        self.out = torch.empty((self.B, shape.horizon, shape.action_dim), dtype=torch.float32, device=dev)
        self.ids = np.ascontiguousarray(ids, np.int32)

    def call(self):
        self.pol.denoise(self.obs, self.noise, self.ids, out=self.out)

    def throughput(self, steps, warmup):
        """K back-to-back calls: wall time between two synchronisations, the
        per-call time of the call's kernels from events recorded on the launch
        stream around each call, and the mean duration of the denoising
        kernel alone from the library's events around its launch (same
        stream)."""
        torch = self.torch
        for _ in range(warmup):
            self.call()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        self.pol.set_kernel_timing(True)
        self.pol.kernel_time()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for s, e in ev:
            s.record()
            self.call()
            e.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        self.pol.synchronize()   # raises if a kernel reported a device-side failure
        kms = [s.elapsed_time(e) for s, e in ev]
        dms, dn = self.pol.kernel_time()
        self.pol.set_kernel_timing(False)
        self.den_ms = dms / max(dn, 1)
        return wall, kms

    def latency(self, n, warmup):
        """Per-call latency: enqueue, run, synchronise (what a controller sees)."""
        torch = self.torch
        for _ in range(warmup):
            self.call()
        torch.cuda.synchronize()
        lat = []
        for _ in range(n):
            t = time.perf_counter()
            self.call()
            torch.cuda.synchronize()
            lat.append((time.perf_counter() - t) * 1e3)
        self.pol.synchronize()
        return lat

    def close(self):
        """Release the policy and the device tensors (nothing is left for
        interpreter shutdown)."""
        self.torch.cuda.synchronize()
        self.pol.close()
        self.obs = self.noise = self.out = None


def host_info():
    """CPU model of the host and the BLAS library numpy calls."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas, threads = None, os.cpu_count() or 1
    try:
        from threadpoolctl import threadpool_info
        infos = [t for t in threadpool_info() if t.get("user_api") == "blas"]
        if infos:
            t = infos[0]
            blas = f"{t.get('internal_api')} {t.get('version')} ({t.get('threading_layer')} threads)"
            threads = max(int(x.get("num_threads", 1)) for x in infos)
    except Exception:
        pass
    return {"cpu_model": model, "blas": blas, "blas_threads": int(threads), "logical_cpus": os.cpu_count()}


def _oracle_time(w, inp, samples, budget_s):
    """Seconds the fp64 oracle spends on the listed samples of a workload,
    one sample per call, stopping at the budget (at least one sample)."""
    from oracle import evo_oracle as O
    from paper_2607_20293_amd import inputs as I
    P = I.split_weights(w.shape, inp.weights)
    n, t0 = 0, time.perf_counter()
    for j in samples:
        O.denoise(w.shape, P, inp.obs, inp.noise, inp.lattices, inp.ids, dtype=w.dtype, samples=[j])
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    return n, time.perf_counter() - t0


def cpu_baseline(inp, budget_s=12.0):
    """The fp64 oracle on the host cores, on a bounded sample of the headline
    workload's samples (independent by construction)."""
    info = host_info()
    w = inp.workload
    n, el = _oracle_time(w, inp, range(w.batch), budget_s)
    return {"value": n / el, "unit": "chunks/s", "cores": info["blas_threads"], "kind": "oracle",
            "sample": f"{n} of the {w.batch} samples of {w.name} (fp64 NumPy oracle, one sample per call, "
                      f"{el:.1f} s)", **info}


def cpu_baseline_configs(budget_s=6.0):
    """The oracle on the other workloads: the tiny policy and the Push-T
    policy at batch 1 in full, the Push-T batch of 64 until the budget, and
    8-sample subsets of the bimanual and population workloads (their first 8
    samples; chunks/s scales linearly, samples being independent)."""
    from paper_2607_20293_amd import inputs as I
    out = {}
    for name, cap in (("tiny_fp32_b1", None), ("pusht_bf16_b1_d25", None), ("pusht_fp32_b1_d25", None),
                      ("pusht_bf16_b64_d25", None), ("bimanual_bf16_b128_d20", 8), ("population_bf16_b512", 8)):
        w = I.WORKLOADS[name]
        inp = I.make_inputs(w)
        idx = range(w.batch if cap is None else cap)
        n, el = _oracle_time(w, inp, idx, budget_s if w.batch > 1 else 1e9)
        out[name] = {"chunks_per_s": round(n / el, 3), "latency_ms": round(el / n * 1e3, 2),
                     "samples_timed": n, "batch": w.batch, "seconds": round(el, 2)}
        log(f"[bench] oracle {name}: {out[name]}")
    return out


def bench_encoder(dev):
    """Observation encoder of the image policy (84x84 frames, ResNet-18
    topology with GroupNorm, bf16 operands) at 512 frames (256 chunks x 2
    observation steps), and the whole action query at batch 1: encode the 2
    observation frames into the observation rows, then the cached loop."""
    import torch
    from paper_2607_20293_amd import evo
    from paper_2607_20293_amd import inputs as I
    extras = {}
    e, s = I.ENC_ROBOMIMIC, I.IMAGE
    nf = 256 * s.n_obs
    enc = evo.Encoder(e, I.make_encoder_weights(e, 0), "bf16", max_batch=nf)
    imgs = torch.from_numpy(I.make_images(e, nf, 0)).to(dev)
    obs_e = torch.from_numpy(I.make_obs(s, 256, 0)).to(dev)
    feats = obs_e.view(nf, s.obs_dim)[:, :e.out_dim]
    for _ in range(3):
        enc.encode(imgs, out=feats)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    reps = 20
    ev[0].record()
    for _ in range(reps):
        enc.encode(imgs, out=feats)
    ev[1].record()
    torch.cuda.synchronize()
    enc_ms = ev[0].elapsed_time(ev[1]) / reps
    enc_tf = enc.flops(nf) / (enc_ms * 1e-3) / 1e12
    flops_frame = enc.flops(1)
    enc.close()
    # the batch-1 query runs on an encoder planned for its own batch (the
    # work split follows max_batch)
    enc = evo.Encoder(e, I.make_encoder_weights(e, 0), "bf16", max_batch=s.n_obs)
    wts = I.make_weights(s, 0)
    img1 = imgs[:s.n_obs].contiguous()
    pa = {}
    # the paper's wall-clock table rows (uncached, EVO at M = 8 and M = 10) in
    # this policy's terms: the uncached loop, the fixed-interval M = 8 and
    # M = 10 unit lattices, the printed EVO Push-T lattice (same 8 layers and
    # 100 steps; M = 10), plus the 25%-density lattice of the headline
    gold = os.path.join(ROOT, "tests", "golden", "schedules_pusht.txt")
    U = 3 * s.n_layers
    lats = {"0.25": (I.make_lattice("dirichlet", s.n_layers, s.n_steps, 0.25, 0), 0),
            "1.0": (I.make_lattice("all", s.n_layers, s.n_steps, 1.0, 0), 0),
            "fixed_interval_M8": (I.lattice_fixed_interval(U, s.n_steps, 8), 1),
            "fixed_interval_M10": (I.lattice_fixed_interval(U, s.n_steps, 10), 1),
            "printed_evo_M10": (I.printed_lattice(gold, "EVO", s.n_layers, s.n_steps), 1)}
    for name, (lt, gran) in lats.items():
        r = Runner(f"image_bf16_b1_{name}", s, wts, "bf16", [lt], np.zeros(1, np.int32),
                   I.make_obs(s, 1, 0), I.make_noise(s, 1, 0), gran=gran)
        f1 = r.obs.view(s.n_obs, s.obs_dim)[:, :e.out_dim]

        def query():
            enc.encode(img1, out=f1)
            r.call()

        for _ in range(3):
            query()
        torch.cuda.synchronize()
        ls, le = [], []
        for _ in range(30):
            t = time.perf_counter()
            query()
            torch.cuda.synchronize()
            ls.append((time.perf_counter() - t) * 1e3)
        for _ in range(30):
            t = time.perf_counter()
            enc.encode(img1, out=f1)
            torch.cuda.synchronize()
            le.append((time.perf_counter() - t) * 1e3)
        r.pol.synchronize()
        r.close()
        pa[name] = {"p50_ms": round(statistics.median(ls), 4), "encode_p50_ms": round(statistics.median(le), 4)}
    enc.close()
    extras["encoder_robomimic_bf16_b512"] = {
        "frames_per_s": round(nf / (enc_ms * 1e-3), 1), "ms": round(enc_ms, 4), "TFLOPs": round(enc_tf, 2),
        "frac_peak": round(enc_tf / PEAK["bf16"], 4), "flops_per_frame": flops_frame}
    for name in pa:
        pa[name]["speedup_vs_uncached"] = round(pa["1.0"]["p50_ms"] / pa[name]["p50_ms"], 3)
    extras["predict_action_image_bf16_b1"] = pa
    log(f"[bench] encoder_robomimic_bf16_b512: {extras['encoder_robomimic_bf16_b512']}")
    log(f"[bench] predict_action_image_bf16_b1: {pa}")
    return extras


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--only-main", action="store_true", help="headline workload only (profiling runs)")
    ap.add_argument("--workload", default="image_bf16_b256_d12",
                    help="workload timed for the main line (profiling runs of other workloads)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only-encoder", action="store_true",
                    help="observation encoder and batch-1 action query only (profiling runs)")
    ap.add_argument("--calib-copy", action="store_true", help="also run one 256 MiB device copy (counter scale)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported by this build "
              f"(samples shard across GPUs with no communication, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_20293_amd import evo
    from paper_2607_20293_amd import inputs as I
    evo.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"

    if args.only_encoder:
        print(json.dumps(bench_encoder(torch.device("cuda:0"))), flush=True)
        return

    if args.calib_copy:
        x = torch.ones(64 << 20, dtype=torch.float32, device="cuda:0")
        y = torch.empty_like(x)
        y.copy_(x)
        torch.cuda.synchronize()
        del x, y

    # ---------------- headline: batch 256, shared 12.5% lattice
    w = I.WORKLOADS[args.workload]
    inp = I.make_inputs(w)
    log(f"[bench] {w.name}: setup")
    run = Runner(w.name, w.shape, inp.weights, w.dtype, inp.lattices, inp.ids, inp.obs, inp.noise)
    wall, kms = run.throughput(args.steps, args.warmup)
    st = run.pol.stats()
    den_ms = run.den_ms
    run.close()
    K = args.steps
    value = w.batch * K / wall
    ms_per_step = wall / K * 1e3
    k_avg_ms = float(np.mean(kms))
    log(f"[bench] {w.name}: {value:.1f} chunks/s, {ms_per_step:.3f} ms/call, kernels {k_avg_ms:.3f} ms, "
        f"denoise_kernel {den_ms:.4f} ms")
    # algorithmic work of one launch: the refreshed units' FLOPs in the
    # paper's convention (every evaluated unit counted with its full
    # projections) plus the always-on products, over the denoising kernel's
    # own mean duration
    alg_flops = st["flops_cacheable"] + st["flops_always"]
    achieved = alg_flops / (den_ms * 1e-3) / 1e12
    impl = st["flops_kernel"] / (k_avg_ms * 1e-3) / 1e12
    roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK[w.dtype], "unit": "TFLOP/s",
            "frac": round(achieved / PEAK[w.dtype], 4), "traffic": None,
            "kernel": "denoise_kernel", "kernel_ms": round(den_ms, 4), "flops_per_launch": alg_flops,
            "flops_basis": "flops_cacheable + flops_always",
            "executed": {"flops_kernel": st["flops_kernel"], "kernels": "obs_fold_kernel + denoise_kernel",
                         "kernels_ms": round(k_avg_ms, 4), "achieved": round(impl, 2),
                         "frac": round(impl / PEAK[w.dtype], 4)},
            "weight_stream_GBps": round(st["weight_bytes"] / (den_ms * 1e-3) / 1e9, 1)}
    if os.path.exists(COUNTERS):
        try:
            c = json.load(open(COUNTERS))
            cw = c.get("workloads", {}).get(w.name)
            if c.get("source_sha") == kernel_source_sha() and cw:
                # HBM bytes of one denoise_kernel launch (FETCH_SIZE and
                # WRITE_SIZE scaled by a 256 MiB copy), taken while this
                # kernel source was current
                roof["traffic"] = cw["hbm_bytes_per_launch"]
                roof["traffic_GBps"] = round(cw["hbm_bytes_per_launch"] / (den_ms * 1e-3) / 1e9, 1)
                roof["mfma_util_pct_counter"] = cw.get("mfma_util_pct")
        except Exception:
            pass

    extras = {}
    lat = {}
    if not args.only_main:
        # ---------------- batch-1 latency vs density (Push-T-shaped policy)
        s = I.PUSHT
        wts = I.make_weights(s, 0)
        obs1, noise1 = I.make_obs(s, 1, 0), I.make_noise(s, 1, 0)
        for dtype in ("bf16", "fp32"):
            row = {}
            for dens in (0.125, 0.25, 0.5, 1.0):
                lt = I.make_lattice("all" if dens == 1.0 else "dirichlet", s.n_layers, s.n_steps, dens, 0)
                r = Runner(f"pusht_{dtype}_b1_{dens}", s, wts, dtype, [lt], np.zeros(1, np.int32), obs1, noise1)
                ls = r.latency(40 if dtype == "bf16" else 20, 3)
                _, kk = r.throughput(10, 2)
                r.close()
                row[str(dens)] = {"p50_ms": round(statistics.median(ls), 4),
                                  "p90_ms": round(float(np.percentile(ls, 90)), 4),
                                  "kernel_ms": round(float(np.median(kk)), 4)}
                log(f"[bench] pusht b1 {dtype} density {dens}: p50 {row[str(dens)]['p50_ms']:.3f} ms "
                    f"kernel {row[str(dens)]['kernel_ms']:.3f} ms")
            lat[dtype] = row
        # ---------------- comparison schedule families at batch 1 (Push-T-shaped, bf16):
        # fixed-interval synchronous refresh (EfficientVLA, M = 8, 10), a block-wise
        # fixed budget (M = 10 per unit) and the printed BAC / EVO Push-T schedules;
        # FLOP speed-up (full / cached-path FLOPs) next to the measured one
        gold = os.path.join(ROOT, "tests", "golden", "schedules_pusht.txt")
        U = 3 * s.n_layers
        fams = {"full": I.lattice_all(U, s.n_steps),
                "efficientvla_M8": I.lattice_fixed_interval(U, s.n_steps, 8),
                "efficientvla_M10": I.lattice_fixed_interval(U, s.n_steps, 10),
                "blockwise_M10": I.lattice_blockwise_budget(U, s.n_steps, 10, np.random.default_rng(10)),
                "printed_bac": I.printed_lattice(gold, "BAC", s.n_layers, s.n_steps),
                "printed_evo": I.printed_lattice(gold, "EVO", s.n_layers, s.n_steps)}
        fam = {}
        for fname, lt in fams.items():
            r = Runner(f"pusht_bf16_b1_{fname}", s, wts, "bf16", [lt], np.zeros(1, np.int32), obs1, noise1,
                       gran=1)
            ls = r.latency(30, 3)
            sx = r.pol.stats()
            r.close()
            fam[fname] = {"p50_ms": round(statistics.median(ls), 4),
                          "refreshes": int(sx["refreshes_effective"]),
                          "flop_speedup": round(sx["flops_full"] / (sx["flops_cacheable"] + sx["flops_always"]), 3)}
        for fname in fam:
            fam[fname]["measured_speedup"] = round(fam["full"]["p50_ms"] / fam[fname]["p50_ms"], 3)
            log(f"[bench] schedule family {fname}: {fam[fname]}")
        extras["schedule_families_pusht_bf16_b1"] = fam

        # ---------------- other workloads
        for name in ("tiny_fp32_b1", "pusht_bf16_b64_d25", "population_bf16_b512", "bimanual_bf16_b128_d20",
                     "bimanual_bf16_b128_all"):
            wl = I.WORKLOADS[name]
            ip = I.make_inputs(wl)
            r = Runner(name, wl.shape, ip.weights, wl.dtype, ip.lattices, ip.ids, ip.obs, ip.noise)
            steps = 3 if wl.shape.d_model == 768 else 10
            wl_wall, kk = r.throughput(steps, 1)
            sx = r.pol.stats()
            dms = r.den_ms
            r.close()
            kavg = float(np.mean(kk))
            tf = sx["flops_kernel"] / (kavg * 1e-3) / 1e12
            ta = (sx["flops_cacheable"] + sx["flops_always"]) / (dms * 1e-3) / 1e12
            extras[name] = {"chunks_per_s": round(wl.batch * steps / wl_wall, 2), "kernel_ms": round(kavg, 4),
                            "denoise_kernel_ms": round(dms, 4), "alg_TFLOPs": round(ta, 2),
                            "alg_frac_peak": round(ta / PEAK[wl.dtype], 4),
                            "TFLOPs": round(tf, 2), "frac_peak": round(tf / PEAK[wl.dtype], 4),
                            "density_eff": round(sx["refreshes_effective"] / (wl.batch * 3 * wl.shape.n_layers
                                                                              * wl.shape.n_steps), 4)}
            log(f"[bench] {name}: {extras[name]}")
            del ip

        # ---------------- redundancy statistics (Sec. 3.3): 8 uncached queries of the
        # Push-T-shaped policy, activations recorded, Eq. 6 scores on the GPU
        s = I.PUSHT
        R = 8
        pol = evo.Policy(s, I.make_weights(s, 0), dtype="fp32", max_batch=R, max_schedules=1)
        pol.set_schedule(0, np.ones((3 * s.n_layers, s.n_steps), np.uint8), evo.GRAN_UNIT)
        dev = torch.device("cuda:0")
        obs_r = torch.from_numpy(I.make_obs(s, R, 0)).to(dev)
        noise_r = torch.from_numpy(I.make_noise(s, R, 0)).to(dev)
        _, acts = pol.collect_activations(obs_r, noise_r)
        sc = pol.redundancy_scores(acts)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        reps = 5
        ev[0].record()
        for _ in range(reps):
            pol.denoise(obs_r, noise_r, acts=acts)
        ev[1].record()
        for _ in range(reps):
            sc = pol.redundancy_scores(acts)
        ev[2].record()
        torch.cuda.synchronize()
        pol.synchronize()
        pol.close()
        collect_ms = ev[0].elapsed_time(ev[1]) / reps
        scores_ms = ev[1].elapsed_time(ev[2]) / reps
        U, T, V = 3 * s.n_layers, s.n_steps, s.horizon * s.d_model
        gram_flops = 2.0 * R * U * T * T * V
        extras["redundancy_pusht_fp32_r8"] = {
            "collect_ms": round(collect_ms, 4), "scores_ms": round(scores_ms, 4),
            "gram_TFLOPs": round(gram_flops / (scores_ms * 1e-3) / 1e12, 2),
            "frac_fp32_peak": round(gram_flops / (scores_ms * 1e-3) / 1e12 / PEAK["fp32"], 4)}
        log(f"[bench] redundancy_pusht_fp32_r8: {extras['redundancy_pusht_fp32_r8']}")
        del acts

        # ---------------- schedule search (Sec. 3.2, Sec. 4.1 settings): K = 240 on the
        # Push-T-shaped policy in bf16, population 30, 10 elites, 30 generations, 16 quick
        # episodes per schedule (one batched call of up to 480 episodes per generation),
        # guided individuals from the Eq. 6 scores above, synthetic success fitness
        s = I.PUSHT
        rows, T = 3 * s.n_layers, s.n_steps
        probs = evo.guided_probabilities(sc.cpu().numpy(), 0.05, 2.0)
        nq, P = 16, 30
        pol = evo.Policy(s, I.make_weights(s, 0), dtype="bf16", max_batch=P * nq, max_schedules=P)
        obs_q = torch.from_numpy(I.make_obs(s, nq, 91)).to(dev)
        noise_q = torch.from_numpy(I.make_noise(s, nq, 91)).to(dev)
        obs_f = torch.from_numpy(I.make_obs(s, 64, 92)).to(dev)
        noise_f = torch.from_numpy(I.make_noise(s, 64, 92)).to(dev)
        cfg = evo.GAConfig.make(240, pop_size=P, n_elite=10, max_generations=30, n_guided=15, seed=0)
        t0 = time.perf_counter()
        res = pol.search(cfg, obs_q, noise_q, obs_f, noise_f, probs=probs, tau=0.4, q_base=1.0, delta_acc=0.125)
        wall = time.perf_counter() - t0
        pol.close()
        fits = res["fitness"]
        extras["search_pusht_bf16_K240"] = {
            "seconds": round(wall, 3), "generations": res["generations"], "evaluations": res["evaluations"],
            "formal_evaluations": res["formal_evaluations"], "accepted": res["accepted"],
            "ms_per_generation": round(wall / res["generations"] * 1e3, 2),
            "episodes_per_s": round((res["evaluations"] * nq + res["formal_evaluations"] * 64) / wall, 1),
            "best_quick_initial": float(np.max(fits[0])), "best_quick": res["best_quick"],
            "mean_quick_initial": round(float(np.mean(fits[0])), 4),
            "mean_quick_last": round(float(np.mean(fits[-1])), 4)}
        log(f"[bench] search_pusht_bf16_K240: {extras['search_pusht_bf16_K240']}")

        extras.update(bench_encoder(dev))

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] oracle CPU baseline ...")
        cpu = cpu_baseline(inp)
        log(f"[bench] oracle: {cpu}")
        if not args.only_main:
            cpu["configs"] = cpu_baseline_configs()

    res = {
        "metric": METRIC, "value": round(value, 2), "unit": "chunks/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "density": w.density, "n_layers": w.shape.n_layers,
                   "d_model": w.shape.d_model, "horizon": w.shape.horizon, "action_dim": w.shape.action_dim,
                   "n_steps": w.shape.n_steps, "parallelism": "none (one GPU)"},
        "latency_b1_p50_ms": lat.get("bf16", {}).get("0.25", {}).get("p50_ms"),
        "latency_b1": lat or None,
        "workloads": extras or None,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    # everything the run created on the device is released before the
    # interpreter shuts down
    import gc
    gc.collect()
    torch.cuda.synchronize()


if __name__ == "__main__":
    main()
