"""Throughput of the batched sliding-window anomaly scorer on one MI355X.

One step is one pass of the whole detection path over one batch of synthetic streams
already resident in HBM: window enumeration (host helper + offsets upload), reference
statistics, scoring of every window (normalise -> encoder -> KL score -> decoder MD),
the peaks-over-threshold threshold over the calibration windows, and the flags of every
window. Prints one JSON line.

    python bench.py [--gpus 1] [--steps 10] [--warmup 3] [--config c5]

With --mode stream it measures the streaming path instead: the config's detector shape over
its number of streams, every push appending one step to each stream, scoring each stream's
newest window and updating each stream's SPOT threshold (one push is one step).

With --mode train it measures one semi-supervised ELBO training step of the config's detector
shape (Eq. (9): forward, PI-controlled KL weight, backward, Adam) on a batch of --batch labelled
windows resident in HBM (one step is one training step).

With --mode variants it measures the detector-output variants on the config's workload: every
window normalised against itself (--norm window, default) or its reference prefix, with its KL
score, md, per-metric md vector and reconstruction error (one step is one call).

With --mode config it measures the configuration scans (Section IV-A, Eqs. (4)-(6)) over 1024
services x 16384 one-minute steps of the Table II metrics: every window's OLS fits and t-test,
then each service's KDE limits and configuration (one step is both calls).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "metric-windows scored/sec at 1 MI355X; % of HBM/MFMA roofline"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}     # dense MFMA peaks of the MI355X datasheet
HBM_PEAK_GBS = 8000.0
# CPU-baseline sample per config: (streams per timed group, windows per stream)
CPU_SAMPLE = {"c1": (1, None), "c2": (2, 8192), "c3": (8, 1024), "c4": (16, 128), "c5": (24, 16384)}
KERNEL_SRC = os.path.join(ROOT, "paper_2407_09486_amd", "csrc", "k_score_mfma.hip")


def flops_per_window(cfg) -> int:
    """Algorithmic flops of one window: encoder layer 2HD, posterior heads 4LH, decoder 2LH + 2H."""
    H, L, D = cfg.hidden, cfg.latent, cfg.d
    return 2 * H * D + 4 * L * H + 2 * L * H + 2 * H


def score_kernel_name(cfg) -> str:
    """The library's scoring kernel for a workload: bf16 detectors with 193..256 hidden units take
    the ring kernel, every other matrix-core shape the general one."""
    return "k_score_ring" if cfg.dtype == "bf16" and 192 < cfg.hidden <= 256 else "k_score_mfma"


def kernel_source_hash(kernel="k_score_mfma") -> str:
    """Hash of the sources one scoring kernel is built from (a counter summary taken on other
    sources no longer describes it)."""
    h = hashlib.sha256()
    for name in (f"{kernel}.hip", "mfma_common.h", "internal.h"):
        with open(os.path.join(ROOT, "paper_2407_09486_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(cfg, kernel=None):
    """HBM bytes per launch of a workload's kernel (default: its scoring kernel) from the committed
    rocprofv3 counter summary (profiles/<kernel>_<workload>_counters.txt, read from a file, not
    measured in this run), if it still describes the current kernel source (else None)."""
    kernel = kernel or score_kernel_name(cfg)
    path = os.path.join(ROOT, "profiles", f"{kernel[2:]}_{cfg.name}_counters.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.strip().split("=", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha") != kernel_source_hash(kernel):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    """The host CPU's model name (first processor of /proc/cpuinfo), or the platform's guess."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(cfg, weights, budget_s=10.0):
    """The oracle (all host cores) on groups of leading streams, each capped at a number of windows
    per stream, until about budget_s seconds of work have been timed."""
    import numpy as np

    import oracle
    from paper_2407_09486_amd import workloads as wl
    group, max_w = CPU_SAMPLE.get(cfg.name, (4, 4096))
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    n_done, s0, dt, threads = 0, 0, 0.0, 1
    while dt < budget_s and s0 < cfg.n_streams:
        streams = np.arange(s0, min(s0 + group, cfg.n_streams))
        w = wl.generate(cfg, streams=streams)
        x = w.values_f64()
        t0 = time.perf_counter()
        sc, md, info = oracle.score(x, w.stream_offsets, window=cfg.window, stride=cfg.stride,
                                    weights=weights.as_f64(), act=cfg.act, ref_frac=cfg.ref_frac,
                                    bf16=cfg.dtype == "bf16", max_windows=max_w, threads=cores,
                                    return_stats=True)
        dt += time.perf_counter() - t0
        n_done += int(np.isfinite(sc).sum())
        threads = int(info["threads"])
        s0 = int(streams[-1]) + 1
    # the same oracle on one thread, over the first stream's sampled windows
    w1 = wl.generate(cfg, streams=np.arange(0, 1))
    t0 = time.perf_counter()
    sc1 = oracle.score(w1.values_f64(), w1.stream_offsets, window=cfg.window, stride=cfg.stride,
                       weights=weights.as_f64(), act=cfg.act, ref_frac=cfg.ref_frac,
                       bf16=cfg.dtype == "bf16", max_windows=max_w, threads=1, return_stats=True)[0]
    dt1 = time.perf_counter() - t0
    n1 = int(np.isfinite(sc1).sum())
    sample = (f"{cfg.name}: streams 0..{s0 - 1}, "
              + (f"first {max_w} windows each" if max_w else "all windows")
              + f" ({n_done} windows, {dt:.1f} s of fp64 oracle incl. reference statistics); "
              + f"on 1 thread {n1 / dt1:.4g} windows/s (stream 0, {n1} windows, {dt1:.1f} s)")
    return {"value": n_done / dt, "unit": "windows/s", "cores": threads, "cpu_model": cpu_model(),
            "kind": "oracle", "sample": sample}


def secondary_leg(name, launches=5, warmup=2):
    """Kernel-only timing of the scorer on a second workload (after the headline's timed region,
    not part of ms_per_step): the bf16 matrix-core path of the 16384-stream workload by default."""
    import numpy as np
    import torch

    from paper_2407_09486_amd import binding
    from paper_2407_09486_amd import workloads as wl
    cfg = wl.CONFIGS[name]
    t0 = time.perf_counter()
    w = wl.generate(cfg)
    weights = wl.make_weights(cfg)
    print(f"[bench] secondary {cfg.name}: generated in {time.perf_counter() - t0:.1f} s", file=sys.stderr,
          flush=True)
    dev = torch.device("cuda", 0)
    x = torch.from_numpy(w.x_bits.view(np.int16) if cfg.dtype == "bf16" else w.x).to(dev)
    so = torch.from_numpy(w.stream_offsets).to(dev)
    so_h = w.stream_offsets
    del w
    det = binding.Detector(cfg.metrics, cfg.window, cfg.stride, cfg.hidden,
                           binding.weights_for_library(weights, cfg.dtype), latent=cfg.latent,
                           dtype=cfg.dtype, act=cfg.act, ref_frac=cfg.ref_frac)
    binding.enova_detect_set_timing(det.handle, True)
    woff_h = det.window_offsets(so_h)
    N = int(woff_h[-1])
    wo = torch.from_numpy(woff_h).to(dev)
    scores = torch.empty(N, dtype=torch.float32, device=dev)
    md = torch.empty(N, dtype=torch.float32, device=dev)
    ks = []
    for i in range(warmup + launches):
        binding.enova_detect_score(det.handle, x, so, wo, len(so_h) - 1, N, None, None, math.nan, scores, md, None)
        torch.cuda.synchronize()
        if i >= warmup:
            ks.append(binding.enova_detect_kernel_times(det.handle)[0])
    det.close()
    k_ms = float(np.median(ks))
    fpw = flops_per_window(cfg)
    achieved = fpw * N / (k_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[cfg.dtype]
    return {"workload": f"{cfg.name}: {cfg.description}", "dtype": cfg.dtype, "windows": N,
            "kernel": score_kernel_name(cfg), "kernel_ms": round(k_ms, 4), "launches": launches,
            "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
            "traffic": load_traffic(cfg),
            "traffic_source": f"profiles/{score_kernel_name(cfg)[2:]}_{cfg.name}_counters.txt (rocprofv3 FETCH_SIZE + "
                              "WRITE_SIZE, read from the file when its kernel source hash matches; null otherwise)",
            "note": "kernel-only (library HIP events, median of the launches); not part of ms_per_step"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c5")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe-gib", type=float, default=0.0,
                    help="also run a plain device copy of this size (counter calibration)")
    ap.add_argument("--mode", choices=["batch", "stream", "train", "config", "variants"], default="batch")
    ap.add_argument("--norm", choices=["window", "reference"], default="window",
                    help="normalisation of --mode variants")
    ap.add_argument("--batch", type=int, default=8192, help="windows per training step (--mode train)")
    ap.add_argument("--secondary", default="auto",
                    help="second workload timed kernel-only after the headline (auto: c4 when the headline "
                         "is c5; none: skip)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the detector shards by stream with no collectives, "
              "and the bench measures the single-GPU kernel (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2407_09486_amd import binding
    from paper_2407_09486_amd import workloads as wl

    cfg = wl.CONFIGS[args.config]
    if args.mode == "stream":
        stream_main(args, cfg)
        return
    if args.mode == "train":
        train_main(args, cfg)
        return
    if args.mode == "config":
        config_main(args)
        return
    if args.mode == "variants":
        variants_main(args, cfg)
        return
    t_gen = time.perf_counter()
    w = wl.generate(cfg)
    weights = wl.make_weights(cfg)
    t_gen = time.perf_counter() - t_gen
    print(f"[bench] {cfg.name}: generated {w.n_streams} streams, {int(w.stream_offsets[-1])} steps "
          f"in {t_gen:.1f} s", file=sys.stderr, flush=True)

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    x = torch.from_numpy(w.x_bits.view(np.int16) if cfg.dtype == "bf16" else w.x).to(dev)
    so = torch.from_numpy(w.stream_offsets).to(dev)
    so_h = w.stream_offsets
    del w
    det = binding.Detector(cfg.metrics, cfg.window, cfg.stride, cfg.hidden,
                           binding.weights_for_library(weights, cfg.dtype), latent=cfg.latent,
                           dtype=cfg.dtype, act=cfg.act, ref_frac=cfg.ref_frac)
    binding.enova_detect_set_timing(det.handle, True)
    woff_h = det.window_offsets(so_h)
    N = int(woff_h[-1])
    woff_pin = torch.from_numpy(woff_h).pin_memory()
    wo = torch.empty_like(woff_pin, device=dev)
    scores = torch.empty(N, dtype=torch.float32, device=dev)
    md = torch.empty(N, dtype=torch.float32, device=dev)
    flags = torch.empty(N, dtype=torch.uint8, device=dev)
    n_streams = len(so_h) - 1
    stream = torch.cuda.current_stream()
    kernel_ms = []
    stats_ms = []
    thr_hist = []

    def step(record):
        wh = det.window_offsets(so_h)                                   # window enumeration
        woff_pin.numpy()[:] = wh
        wo.copy_(woff_pin, non_blocking=True)
        binding.enova_detect_score(det.handle, x, so, wo, n_streams, N, None, None, math.nan,
                                   scores, md, None, stream)            # stats + score + md
        if record:
            a, b = binding.enova_detect_kernel_times(det.handle)
            kernel_ms.append(a)
            stats_ms.append(b)
        thr, _ = binding.enova_detect_threshold(det.handle, scores, so, wo, n_streams, N, 0.98, 1e-3,
                                                flags, stream)          # POT threshold + flags
        thr_hist.append(thr)

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(True)
        print(f"[bench] step {i + 1}/{args.steps} kernel {kernel_ms[-1]:.2f} ms", file=sys.stderr,
              flush=True)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = ev0.elapsed_time(ev1) / args.steps
    value = N * args.steps / (wall if wall > 0 else float("nan"))
    value_ev = N / (ms_step / 1e3)

    if args.copy_probe_gib > 0:
        nbytes = int(args.copy_probe_gib * (1 << 30))
        a = torch.empty(nbytes // 4, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    k_ms = float(np.mean(kernel_ms))
    fpw = flops_per_window(cfg)
    achieved = fpw * N / (k_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[cfg.dtype]
    traffic = load_traffic(cfg)
    roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4), "traffic": traffic,
            "traffic_source": f"profiles/{score_kernel_name(cfg)[2:]}_{cfg.name}_counters.txt (rocprofv3 FETCH_SIZE "
                              "+ WRITE_SIZE, read from the file when its kernel source hash matches; null otherwise)",
            "kernel": score_kernel_name(cfg), "kernel_ms": round(k_ms, 4),
            "flops_per_window": fpw, "windows_per_launch": N,
            "stats_kernel_ms": round(float(np.mean(stats_ms)), 4)}
    out = {
        "metric": METRIC, "value": round(value_ev, 1), "unit": "windows/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic (seeded generators standing in for the paper's industrial series)",
        "config": {"workload": f"{cfg.name}: {cfg.description}", "streams": n_streams, "windows": N,
                   "metrics": cfg.metrics, "window": cfg.window, "stride": cfg.stride,
                   "hidden": cfg.hidden, "latent": cfg.latent, "act": cfg.act,
                   "data_seed": cfg.data_seed, "weight_seed": cfg.weight_seed,
                   "wall_windows_per_s": round(value, 1), "threshold": thr_hist[-1]},
        "roofline": roof,
    }
    det.close()
    sec = args.secondary
    if sec == "auto":
        sec = "c4" if cfg.name == "c5" else "none"
    if sec != "none":
        del x, so, scores, md, flags
        torch.cuda.empty_cache()
        out["secondary"] = secondary_leg(sec)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, weights)
    print(json.dumps(out), flush=True)


STREAM_REF_STEPS = 2048      # reference history per stream: statistics and SPOT calibration


def stream_cpu_baseline(cfg, weights, x_ref, x_live, n_streams, pushes):
    """The oracle on a bounded sample of the streaming work: the newest windows of the first
    streams scored window by window, then their SPOT steps."""
    import numpy as np

    import oracle
    k = min(512, n_streams)
    W, S, M = cfg.window, cfg.stride, cfg.metrics
    steps = W - 1 + pushes
    xs = np.concatenate([x_live[s, :steps] for s in range(k)]).astype(np.float64)
    offs = np.arange(k + 1, dtype=np.int64) * steps
    mean = np.array([x_ref[s].mean(axis=0) for s in range(k)])
    std = np.array([x_ref[s].std(axis=0) for s in range(k)])
    std[std <= 1e-6] = 1.0
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    t0 = time.perf_counter()
    sc, _, info = oracle.score(xs, offs, window=W, stride=S, weights=weights.as_f64(), act=cfg.act,
                               bf16=cfg.dtype == "bf16", ref_mean=mean, ref_std=std, threads=cores,
                               return_stats=True)
    sc = sc.reshape(k, -1)
    for s in range(k):
        sp = oracle.Spot(np.random.default_rng(s).gamma(2.0, 1.0, 500))
        for v in sc[s]:
            sp.step(float(v))
    dt = time.perf_counter() - t0
    n = sc.size
    return {"value": n / dt, "unit": "windows/s", "cores": int(info["threads"]), "cpu_model": cpu_model(), "kind": "oracle",
            "sample": f"streams 0..{k - 1}, {sc.shape[1]} pushes each ({n} windows + SPOT steps, {dt:.1f} s)"}


def stream_main(args, cfg):
    import numpy as np
    import torch

    from paper_2407_09486_amd import binding
    from paper_2407_09486_amd import workloads as wl

    n = cfg.n_streams
    W, S, M = cfg.window, cfg.stride, cfg.metrics
    extra = max(3, min(args.steps, 10))        # pushes after the timed region, for the kernels' own times
    live_steps = W - 1 + (args.warmup + args.steps + extra) * S
    scfg = cfg.replace(kind="ragged_mix") if cfg.kind == "ragged_mix" else cfg
    t_gen = time.perf_counter()
    w = wl.generate(scfg, lengths=[STREAM_REF_STEPS + live_steps] * n)
    weights = wl.make_weights(cfg)
    v = w.values_f32().reshape(n, STREAM_REF_STEPS + live_steps, M)
    x_ref, x_live = v[:, :STREAM_REF_STEPS], v[:, STREAM_REF_STEPS:]
    del w
    print(f"[bench] stream {cfg.name}: {n} streams, {STREAM_REF_STEPS} reference + {live_steps} live steps "
          f"generated in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)

    def to_dev(a):
        a = np.ascontiguousarray(a, np.float32)
        if cfg.dtype == "bf16":
            return torch.from_numpy(wl.to_bf16_bits(a).view(np.int16)).to(dev)
        return torch.from_numpy(a).to(dev)

    det = binding.Detector(M, W, S, cfg.hidden, binding.weights_for_library(weights, cfg.dtype),
                           latent=cfg.latent, dtype=cfg.dtype, act=cfg.act, ref_frac=1.0)
    so_h = np.arange(n + 1, dtype=np.int64) * STREAM_REF_STEPS
    xr = to_dev(x_ref.reshape(-1, M))
    so = torch.from_numpy(so_h).to(dev)
    mean = torch.empty(n * M, dtype=torch.float32, device=dev)
    std = torch.empty(n * M, dtype=torch.float32, device=dev)
    binding.enova_detect_ref_stats(det.handle, xr, so, n, mean, std)
    woff = det.window_offsets(so_h)
    sc_ref, _, _ = det.score(xr, so, torch.from_numpy(woff).to(dev), int(woff[-1]), ref_mean=mean,
                             ref_std=std, md=False)
    t_c = time.perf_counter()
    ss = binding.StreamSet(det, mean, std, sc_ref, woff, level=0.98, q=1e-3, peak_cap=4096)
    t_c = time.perf_counter() - t_c
    del xr, sc_ref
    steps = to_dev(np.ascontiguousarray(x_live.transpose(1, 0, 2)))   # [step][n][M]
    scores = torch.empty(n, dtype=torch.float32, device=dev)
    md = torch.empty(n, dtype=torch.float32, device=dev)
    flags = torch.empty(n, dtype=torch.uint8, device=dev)
    binding.enova_detect_set_timing(det.handle, True)
    t = 0
    for _ in range(W - 1):                                  # fill the rings: no window is due yet
        ss.push(steps[t], scores, md, flags)
        t += 1

    def push_window():
        # one scoring push (and the S - 1 non-scoring pushes before it when S > 1)
        nonlocal t
        due = 0
        while not due:
            due = ss.push(steps[t], scores, md, flags)
            t += 1
    for _ in range(args.warmup):
        push_window()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        push_window()
    ss.state()          # waits for the last push's refit (it runs on the set's own stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_push = ev0.elapsed_time(ev1) / args.steps
    # the kernels' own times: further pushes, each waited for, after the timed region
    score_ms, spot_ms = [], []
    for _ in range(extra):
        push_window()
        a, b = ss.kernel_times()
        score_ms.append(a)
        spot_ms.append(b)
    k_ms = float(np.mean(score_ms))
    fpw = flops_per_window(cfg)
    achieved = fpw * n / (k_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[cfg.dtype]
    t_s, z_s, n_s, k_s = ss.state()
    out = {
        "metric": "streaming windows scored/sec (newest window of every stream per push, per-stream SPOT)",
        "value": round(n / (ms_push / 1e3), 1), "unit": "windows/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_push, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
        "data": "synthetic (seeded generators standing in for the paper's industrial series)",
        "config": {"workload": f"stream {cfg.name} shape: {n} streams x {M} metrics, W={W} S={S}, "
                               f"H={cfg.hidden}, {cfg.dtype}; one step per stream per push",
                   "streams": n, "reference_steps": STREAM_REF_STEPS, "pushes_per_step": S,
                   "wall_windows_per_s": round(n * args.steps / wall, 1),
                   "create_s": round(t_c, 3), "peaks_stored": int(k_s.sum())},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None, "kernel": "k_stream_score",
                     "kernel_ms": round(k_ms, 4), "spot_kernels_ms": round(float(np.mean(spot_ms)), 4),
                     "flops_per_window": fpw, "windows_per_launch": n},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = stream_cpu_baseline(cfg, weights, x_ref, x_live, n, args.steps)
    ss.close()
    det.close()
    print(json.dumps(out), flush=True)


def train_flops_per_window(cfg) -> int:
    """Matrix-product flops of one window in a training step: the forward products
    (encoder 2HD, heads 4LH, decoder 2LH + 2DH) and the backward ones (weight and input gradients
    of the same layers, the encoder's input gradient excluded): 2 (5HD + 9HL)."""
    H, L, D = cfg.hidden, cfg.latent, cfg.d
    return 2 * (5 * H * D + 9 * H * L)


def train_cpu_baseline(cfg, p0, batch, margin, budget_s=10.0):
    """The oracle's training step on the same batch, repeated for about budget_s seconds."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import elbo
    p = {k: v.astype(np.float64) for k, v in p0.items()}
    m = {k: np.zeros_like(v) for k, v in p.items()}
    v = {k: np.zeros_like(x) for k, x in p.items()}
    V, lab, eps = (batch.V.astype(np.float64), batch.labels.astype(np.float64), batch.eps.astype(np.float64))
    integ, k = 0.0, 0
    t0 = time.perf_counter()
    while True:
        k += 1
        p, m, v, integ, _ = elbo.train_step(p, m, v, k, integ, V, lab, eps, act=cfg.act, margin=margin)
        dt = time.perf_counter() - t0
        if dt >= budget_s:
            break
    threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    B = V.shape[0]
    return {"value": round(k * B / dt, 1), "unit": "windows/s", "cores": int(threads), "cpu_model": cpu_model(), "kind": "oracle",
            "sample": f"{k} fp64 oracle steps on the same {B}-window batch ({dt:.1f} s, numpy BLAS threads)"}


def train_main(args, cfg):
    import numpy as np
    import torch

    from paper_2407_09486_amd import binding
    from paper_2407_09486_amd import workloads as wl

    B = args.batch
    w = wl.make_weights(cfg.replace(dtype="f32"), bias_scale=0.1)
    p0 = {k: np.asarray(getattr(w, k), np.float32)
          for k in ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")}
    batch = wl.training_batch(cfg, B, seed=cfg.data_seed)
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    V = torch.from_numpy(batch.V).to(dev)
    lab = torch.from_numpy(batch.labels).to(dev)
    eps = torch.from_numpy(batch.eps).to(dev)
    info = torch.zeros(4, dtype=torch.float32, device=dev)
    margin = float(cfg.d)      # anomalous windows are pushed up to a reconstruction error of D
    tr = binding.Trainer(cfg.d, cfg.hidden, cfg.latent, p0, act=cfg.act, margin=margin)
    for _ in range(args.warmup):
        tr.step(V, lab, eps, info)          # the first step captures the step's graph
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    # timed region: K graph replays back to back, as a training loop runs them
    ev0.record(stream)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        tr.step(V, lab, eps, info)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    # the products' own time: further steps with timing on (launched one by one, events around
    # each product kernel), after the timed region
    tr.set_timing(True)
    gemm_ms, step_ms = [], []
    for _ in range(max(3, min(args.steps, 10))):
        tr.step(V, lab, eps, info)
        a, b = tr.kernel_times()
        gemm_ms.append(a)
        step_ms.append(b)
    tr.set_timing(False)
    g_ms = float(np.mean(gemm_ms))
    fpw = train_flops_per_window(cfg)
    achieved = fpw * B / (g_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS["f32"]
    inf = info.cpu().numpy()
    out = {
        "metric": "windows trained/sec (one semi-supervised ELBO step: forward, backward, Adam)",
        "value": round(B / (ms / 1e3), 1), "unit": "windows/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded labelled AR(1) windows with injected level shifts)",
        "config": {"workload": f"train {cfg.name} detector shape: D={cfg.d} (W={cfg.window} x M={cfg.metrics}), "
                               f"H={cfg.hidden}, L={cfg.latent}, {cfg.act}, batch {B} windows (10% anomalous), "
                               f"anomaly margin {margin:g}",
                   "batch": B, "wall_windows_per_s": round(B * args.steps / wall, 1),
                   "eager_step_ms": round(float(np.mean(step_ms)), 4),
                   "last_loss": float(inf[0]), "last_beta": float(inf[3])},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None,
                     "kernel": "k_gemm_rs + k_gemm (the 11 matrix products of a step)",
                     "kernel_ms": round(g_ms, 4), "flops_per_window": fpw, "windows_per_launch": B},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = train_cpu_baseline(cfg, p0, batch, margin)
    tr.close()
    print(json.dumps(out), flush=True)


def variants_flops_per_window(cfg) -> int:
    """Matrix-product flops of one window's variants: encoder 2HD, heads 4LH, decoder hidden 2LH,
    decoder output 2DH."""
    H, L, D = cfg.hidden, cfg.latent, cfg.d
    return 4 * H * D + 6 * L * H


def variants_cpu_baseline(cfg, w, work, norm, budget_s=10.0):
    import numpy as np

    from oracle import variants as ov
    wts = {k: np.asarray(getattr(w, k), np.float64) for k in
           ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")}
    import oracle
    x = work.values_f64()
    offs = work.stream_offsets
    nw = oracle.window_count(np.diff(offs), cfg.window, cfg.stride)
    n, t0 = 0, time.perf_counter()
    k = 0
    while time.perf_counter() - t0 < budget_s and k < int(nw.max()):
        pairs = [(s, k) for s in range(min(64, work.n_streams)) if k < nw[s]]
        r = ov.score_ext(x, offs, window=cfg.window, stride=cfg.stride, weights=wts, act=cfg.act, norm=norm,
                         ref_frac=cfg.ref_frac, bf16=cfg.dtype == "bf16", pairs=pairs)
        n += len(r["score"])
        k += 1
    dt = time.perf_counter() - t0
    return {"value": round(n / dt, 1), "unit": "windows/s", "cores": 1, "cpu_model": cpu_model(), "kind": "oracle",
            "sample": f"windows 0..{k - 1} of streams 0..63 ({n} windows, {dt:.1f} s, fp64, one core)"}


def variants_main(args, cfg):
    import numpy as np
    import torch

    from paper_2407_09486_amd import binding
    from paper_2407_09486_amd import workloads as wl

    t_gen = time.perf_counter()
    work = wl.generate(cfg)
    w = wl.make_weights(cfg)
    print(f"[bench] variants {cfg.name}: generated in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr,
          flush=True)
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    det = binding.Detector(cfg.metrics, cfg.window, cfg.stride, cfg.hidden, binding.weights_for_library(w, cfg.dtype),
                           latent=cfg.latent, dtype=cfg.dtype, act=cfg.act, ref_frac=cfg.ref_frac)
    if cfg.dtype == "bf16":
        x = torch.from_numpy(work.x_bits.view(np.int16)).to(dev)
    else:
        x = torch.from_numpy(work.x).to(dev)
    so = torch.from_numpy(work.stream_offsets).to(dev)
    woff = det.window_offsets(work.stream_offsets)
    wo = torch.from_numpy(woff).to(dev)
    N = int(woff[-1])
    M = cfg.metrics
    sc = torch.empty(N, dtype=torch.float32, device=dev)
    md = torch.empty(N, dtype=torch.float32, device=dev)
    mdm = torch.empty((N, M), dtype=torch.float32, device=dev)
    rec = torch.empty(N, dtype=torch.float32, device=dev)
    norm = {"window": binding.ENOVA_NORM_WINDOW, "reference": binding.ENOVA_NORM_REFERENCE}[args.norm]

    def step():
        binding.enova_detect_score_ext(det.handle, x, so, wo, work.n_streams, N, None, None, norm, sc, md, mdm, rec)
    kernel = "k_ext_fused" if det.ext_fused() else "chunked"
    for _ in range(args.warmup):
        step()
    binding.enova_detect_set_timing(det.handle, True)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    k_ms = []
    ev0.record(stream)
    for _ in range(args.steps):
        step()
        k_ms.append(binding.enova_detect_ext_time(det.handle))
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    if args.copy_probe_gib > 0:
        # a device copy of known size, the scale of the HBM byte counters
        a = torch.empty(int(args.copy_probe_gib * (1 << 30)) // 4, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    km = float(np.mean(k_ms))
    fpw = variants_flops_per_window(cfg)
    achieved = fpw * N / (km / 1e3) / 1e12
    fused = kernel == "k_ext_fused"
    out = {
        "metric": "windows evaluated/sec (KL score, md, per-metric md vector, reconstruction error)",
        "value": round(N / (ms / 1e3), 1), "unit": "windows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded generators standing in for the paper's industrial series)",
        "config": {"workload": f"variants on {cfg.name}: {work.n_streams} streams x {M} metrics, W={cfg.window} "
                               f"S={cfg.stride}, H={cfg.hidden}, {cfg.dtype} ({N} windows), {args.norm} normalisation",
                   "windows": N},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_TFLOPS["f32"], "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_TFLOPS["f32"], 4),
                     "traffic": load_traffic(cfg, kernel) if fused else None,
                     "traffic_source": (f"profiles/{kernel[2:]}_{cfg.name}_counters.txt (rocprofv3 FETCH_SIZE + "
                                        "WRITE_SIZE, read from the file when its kernel source hash matches; null "
                                        "otherwise)") if fused else None,
                     "kernel": (kernel + " (one launch: staging, per-window statistics, encoder, heads, decoder, "
                                "reductions; timed with its tile scan and map)") if fused else
                               "the chunked variant pass (staging, 4 products, latent, reductions)",
                     "kernel_ms": round(km, 4), "flops_per_window": fpw, "windows_per_launch": N},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = variants_cpu_baseline(cfg, w, work, args.norm)
    det.close()
    print(json.dumps(out), flush=True)


CONFIG_STREAMS, CONFIG_STEPS, CONFIG_W = 1024, 16384, 64


def config_flops_per_window(W: int) -> int:
    """fp64 operations of one window's two-pass fits: means (3W adds), then centred sums
    (3W subtractions and 4W fused multiply-adds, 2 flops each)."""
    return 14 * W


def config_cpu_baseline(x, offs, W, budget_s=10.0):
    """The oracle's window scan on the first streams, for about budget_s seconds."""
    import numpy as np

    from oracle import config_scan as cs
    n, T = 0, int(offs[1] - offs[0])
    t0 = time.perf_counter()
    s = 0
    while time.perf_counter() - t0 < budget_s and s < len(offs) - 1:
        rows = min(T, 2048)
        r = cs.window_scan(x[offs[s]:offs[s] + rows].astype(np.float64), np.array([0, rows]), window=W, stride=1,
                           col_f=0, col_r=1, col_m=5)
        n += len(r["b"])
        s += 1
    dt = time.perf_counter() - t0
    return {"value": round(n / dt, 1), "unit": "windows/s", "cores": 1, "cpu_model": cpu_model(), "kind": "oracle",
            "sample": f"first 2048 steps of streams 0..{s - 1} ({n} windows, {dt:.1f} s, fp64 Python loops)"}


def config_main(args):
    import numpy as np
    import torch

    from paper_2407_09486_amd import binding
    from paper_2407_09486_amd import workloads as wl

    t_gen = time.perf_counter()
    w = wl.config_series(CONFIG_STREAMS, CONFIG_STEPS, seed=20240712)
    print(f"[bench] config: {CONFIG_STREAMS} services x {CONFIG_STEPS} steps generated in "
          f"{time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    W = CONFIG_W
    M = len(wl.CONFIG_METRICS)
    sc = binding.ConfigScanner(M, W, 1, col_finished=0, col_running=1, col_exec_time=4, col_mem_util=5)
    x = torch.from_numpy(w.x).to(dev)
    so = torch.from_numpy(w.stream_offsets).to(dev)
    woff_h = sc.window_offsets(w.stream_offsets)
    wo = torch.from_numpy(woff_h).to(dev)
    N = int(woff_h[-1])

    def step():
        sc.scan(x, so, wo, N)
        sc.recommend(x, so)
    for _ in range(args.warmup):
        step()
    sc.set_timing(True)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    k_ms = []
    ev0.record(stream)
    for _ in range(args.steps):
        step()
        k_ms.append(sc.kernel_time())
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    km = float(np.mean(k_ms))
    fpw = config_flops_per_window(W)
    achieved = fpw * N / (km / 1e3) / 1e12
    out = {
        "metric": "windows scanned/sec (per-window OLS fits and t-test, then per-service KDE limits)",
        "value": round(N / (ms / 1e3), 1), "unit": "windows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64",
        "data": "synthetic (seeded serving metrics of Table II, half the services saturating)",
        "config": {"workload": f"config scans: {CONFIG_STREAMS} services x {CONFIG_STEPS} one-minute steps x {M} "
                               f"metrics, W={W} S=1 ({N} windows)", "windows": N},
        "roofline": {"bound": "alu", "achieved": round(achieved, 3), "peak": 78.6, "unit": "TFLOP/s",
                     "frac": round(achieved / 78.6, 4), "traffic": None, "kernel": "k_cfg_scan",
                     "kernel_ms": round(km, 4), "flops_per_window": fpw, "windows_per_launch": N},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = config_cpu_baseline(w.x, w.stream_offsets, W)
    sc.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
