"""Seeded synthetic monitoring streams and detector weights.

This module only *draws inputs*. It holds none of the detector's arithmetic
(no window enumeration, normalisation, scoring or thresholding), so the HIP
path and the CPU oracle can both consume what it produces without sharing any
of the method.

The paper's detection dataset (an industrial chatbot service: 8 LLMs x 2
replicas, 1-minute sampling, Section VI RQ2 setup) is not available; the five
workloads below stand in for it. Each is shaped like the monitoring metrics of
Table II (arrivals, running and pending requests, execution time, GPU memory and
GPU utilisation, sequence lengths) observed as sliding windows, with anomalies
injected only after the reference (training) prefix, mirroring the paper's
train-on-the-first-half / test-on-the-second-half split.

Every stream has its own child seed (``SeedSequence(data_seed).spawn``), so any
subset of streams can be regenerated bit-identically on its own.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np
from scipy.signal import lfilter

PHI = 0.8                                   # AR(1) coefficient of every workload
SIGMA_MARG = 1.0 / math.sqrt(1.0 - PHI * PHI)   # stationary std of the AR(1) with unit innovations


@dataclass(frozen=True)
class Config:
    """One workload: stream shapes, window geometry and detector sizes."""
    name: str
    n_streams: int
    metrics: int
    t_len: int            # fixed stream length (ragged configs: 0)
    t_min: int            # ragged stream length bounds (inclusive)
    t_max: int
    window: int
    stride: int
    hidden: int
    latent: int
    dtype: str            # "f32" or "bf16" (storage/MFMA type of x and W1)
    act: str              # "relu" or "tanh"
    ref_frac: float
    kind: str
    data_seed: int
    weight_seed: int
    description: str = ""

    @property
    def d(self) -> int:
        return self.window * self.metrics

    def replace(self, **kw) -> "Config":
        vals = {f: getattr(self, f) for f in self.__dataclass_fields__}
        vals.update(kw)
        return Config(**vals)


def _cfg(i, **kw):
    base = dict(latent=16, act="relu", ref_frac=0.5, t_min=0, t_max=0,
                data_seed=20240712 + i, weight_seed=7 + i)
    base.update(kw)
    return Config(name=f"c{i}", **base)


CONFIGS = {
    "c1": _cfg(1, n_streams=1, metrics=8, t_len=2048, window=32, stride=1, hidden=32,
               dtype="f32", kind="ar1_spikes",
               description="1 service x 8 metrics x 2048 steps, W=32 S=1, H=32; AR(1) + 4 spikes"),
    "c2": _cfg(2, n_streams=64, metrics=8, t_len=16384, window=64, stride=1, hidden=64,
               dtype="f32", kind="llm_service",
               description="64 services x 8 metrics x 16384 steps, W=64 S=1, H=64; diurnal LLM load + 2 level shifts"),
    "c3": _cfg(3, n_streams=1024, metrics=16, t_len=8192, window=128, stride=4, hidden=128,
               dtype="f32", kind="diurnal_corr",
               description="1024 services x 16 metrics x 8192 steps, W=128 S=4, H=128; diurnal + correlated AR(1) + spikes/drops"),
    "c4": _cfg(4, n_streams=16384, metrics=32, t_len=4096, window=256, stride=8, hidden=256,
               dtype="bf16", kind="ar1_bursts",
               description="16384 streams x 32 metrics x 4096 steps, W=256 S=8, H=256, bf16 x and W1; AR(1) + Poisson bursts"),
    "c5": _cfg(5, n_streams=4096, metrics=16, t_len=0, t_min=512, t_max=65536, window=64, stride=1,
               hidden=128, dtype="f32", kind="ragged_mix",
               description="4096 ragged streams (T ~ U{512..65536}) x 16 metrics, W=64 S=1, H=128; steady/bursty/drifting"),
}


# ----------------------------------------------------------------------------- bf16 helpers
def to_bf16_bits(a) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even); return the bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u >> 16) & 1) + 0x7FFF
    return ((u + r) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ----------------------------------------------------------------------------- containers
@dataclass
class Workload:
    cfg: Config
    stream_offsets: np.ndarray          # int64 [n+1], CSR row offsets into x
    x: np.ndarray | None                # float32 [sum T, M] (f32 configs)
    x_bits: np.ndarray | None           # uint16 [sum T, M] bf16 patterns (bf16 configs)
    labels: np.ndarray                  # uint8 [sum T]: 1 where an anomaly was injected
    streams: np.ndarray                 # int64 ids (within the config) of the generated streams
    seeds: dict = field(default_factory=dict)

    @property
    def n_streams(self) -> int:
        return len(self.stream_offsets) - 1

    def values_f32(self) -> np.ndarray:
        """The input values as float32 (exact for bf16 storage)."""
        if self.x is not None:
            return self.x
        return bf16_bits_to_f32(self.x_bits)

    def values_f64(self) -> np.ndarray:
        return self.values_f32().astype(np.float64)


@dataclass
class Weights:
    w1: np.ndarray          # float32 [H, D] (bf16-exact values for bf16 configs)
    w1_bits: np.ndarray | None
    b1: np.ndarray          # [H]
    wmu: np.ndarray         # [L, H]
    bmu: np.ndarray         # [L]
    wlv: np.ndarray         # [L, H]
    blv: np.ndarray         # [L]
    wd1: np.ndarray         # [H, L]
    bd1: np.ndarray         # [H]
    wd2: np.ndarray         # [D, H]
    bd2: np.ndarray         # [D]

    def as_f64(self) -> dict:
        return {k: getattr(self, k).astype(np.float64)
                for k in ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")}


# ----------------------------------------------------------------------------- weights
def make_weights(cfg: Config, seed: int | None = None, bias_scale: float = 0.0) -> Weights:
    """Xavier-uniform weights U(+-sqrt(6/(fan_in+fan_out))) drawn in the order W1, Wmu, Wlv, Wd1, Wd2.

    Biases are zero unless ``bias_scale`` > 0 (then U(+-bias_scale), drawn after the weights).
    Every array is rounded to float32 once here; for bf16 configs W1 is rounded to bf16 (RNE).
    """
    rng = np.random.default_rng(cfg.weight_seed if seed is None else seed)
    H, L, D = cfg.hidden, cfg.latent, cfg.d

    def xavier(fan_out, fan_in):
        b = math.sqrt(6.0 / (fan_in + fan_out))
        return rng.uniform(-b, b, size=(fan_out, fan_in)).astype(np.float32)

    w1 = xavier(H, D)
    wmu = xavier(L, H)
    wlv = xavier(L, H)
    wd1 = xavier(H, L)
    wd2 = xavier(D, H)

    def bias(n):
        if bias_scale <= 0.0:
            return np.zeros(n, np.float32)
        return rng.uniform(-bias_scale, bias_scale, size=n).astype(np.float32)

    b1, bmu, blv, bd1, bd2 = bias(H), bias(L), bias(L), bias(H), bias(D)
    w1_bits = None
    if cfg.dtype == "bf16":
        w1_bits = to_bf16_bits(w1)
        w1 = bf16_bits_to_f32(w1_bits).reshape(H, D)
    return Weights(w1=w1, w1_bits=w1_bits, b1=b1, wmu=wmu, bmu=bmu, wlv=wlv, blv=blv,
                   wd1=wd1, bd1=bd1, wd2=wd2, bd2=bd2)


# ----------------------------------------------------------------------------- streams
def _ar1(rng, T, M):
    """Stationary Gaussian AR(1), phi=0.8, unit innovations; shape [T, M]."""
    e = rng.standard_normal((T, M))
    e[0] *= SIGMA_MARG
    return lfilter([1.0], [1.0, -PHI], e, axis=0)


def _logistic(z):
    return 1.0 / (1.0 + np.exp(-z))


def _ref_len(cfg, T):
    # first step of the test half (the reference prefix is the first ref_frac of a stream)
    return int(math.floor(float(np.float32(cfg.ref_frac)) * T))


def _gen_ar1_spikes(cfg, rng, T, s):
    M = cfg.metrics
    x = _ar1(rng, T, M)
    lab = np.zeros(T, np.uint8)
    R = _ref_len(cfg, T)
    pos = rng.choice(np.arange(R, T), size=min(4, T - R), replace=False)
    x[pos, :] += 6.0 * SIGMA_MARG
    lab[pos] = 1
    return x, lab


def _gen_llm_service(cfg, rng, T, s):
    """Eight load-linked LLM-serving metrics driven by a diurnal arrival rate."""
    M, W = cfg.metrics, cfg.window
    t = np.arange(T, dtype=np.float64)
    phase = rng.uniform(0.0, 1440.0)
    lam = 50.0 + 30.0 * np.sin(2.0 * np.pi * (t + phase) / 1440.0)
    lab = np.zeros(T, np.uint8)
    R = _ref_len(cfg, T)
    for _ in range(2):                      # two level shifts of the load in the test half
        dur = int(rng.integers(W, 8 * W + 1))
        st = int(rng.integers(R, max(R + 1, T - dur + 1)))
        lam[st:st + dur] += 40.0
        lab[st:st + dur] = 1
    x = np.empty((T, M), np.float64)
    arrivals = rng.poisson(lam)                                            # n^a per step
    in_len = rng.lognormal(6.0, 1.0, T)                                    # mean input length
    out_len = rng.lognormal(6.0, 1.0, T)                                   # mean output length
    util = np.clip(_logistic(6.0 * (lam / 80.0 - 0.6)) + rng.normal(0, 0.02, T), 0, 1)   # g^u
    kv = np.clip(_logistic(5.0 * (lam / 80.0 - 0.7)) + rng.normal(0, 0.02, T), 0, 1)     # m^u
    latency = (0.5 + 1.5 * kv) * rng.lognormal(0.0, 0.1, T)                # t^r (s)
    running = rng.poisson(lam * latency)                                   # n^r (Little's law)
    pending = rng.poisson(20.0 * np.maximum(0.0, lam / 80.0 - 0.8))        # n^p (queue beyond capacity)
    cols = [arrivals, in_len, out_len, util, kv, latency, running, pending]
    for m in range(M):
        x[:, m] = cols[m % len(cols)]
    return x, lab


_CMIX_CACHE = {}


def _gen_diurnal_corr(cfg, rng, T, s):
    M, W = cfg.metrics, cfg.window
    if M not in _CMIX_CACHE:
        _CMIX_CACHE[M] = np.linalg.cholesky(0.4 * np.eye(M) + 0.6 * np.ones((M, M)))
    cm = _CMIX_CACHE[M]
    amp = rng.uniform(1.0, 3.0, M)
    phase = rng.uniform(0.0, 1440.0, M)
    noise = _ar1(rng, T, M) @ cm.T          # cross-metric correlation 0.6, marginal std SIGMA_MARG
    t = np.arange(T, dtype=np.float64)[:, None]
    x = amp * np.sin(2.0 * np.pi * (t + phase) / 1440.0) + noise
    lab = np.zeros(T, np.uint8)
    R = _ref_len(cfg, T)
    n_ev = int(rng.poisson(0.01 * T / W))   # about 1% of windows contain an event
    for _ in range(n_ev):
        t0 = int(rng.integers(R, T))
        sign = 1.0 if rng.random() < 0.5 else -1.0
        x[t0, :] += sign * 6.0 * SIGMA_MARG
        lab[t0] = 1
    return x, lab


def _gen_ar1_bursts(cfg, rng, T, s):
    M = cfg.metrics
    x = _ar1(rng, T, M)
    lab = np.zeros(T, np.uint8)
    starts = np.nonzero(rng.random(T) < 1.0 / 512.0)[0]
    for st in starts:
        dur = int(rng.geometric(1.0 / 16.0))
        x[st:st + dur, :] += 3.0 * SIGMA_MARG
        lab[st:st + dur] = 1
    return x, lab


def _gen_ragged_mix(cfg, rng, T, s):
    """Steady (AR(1)), bursty (Pareto(1.5) renewal arrivals + load-linked metrics) or drifting."""
    M = cfg.metrics
    kind = s % 3
    lab = np.zeros(T, np.uint8)
    if kind == 0:
        return _ar1(rng, T, M), lab
    if kind == 2:
        x = _ar1(rng, T, M)
        x += (0.5 * SIGMA_MARG / 1000.0) * np.arange(T, dtype=np.float64)[:, None]
        return x, lab
    # bursty: a renewal process with Pareto(alpha=1.5, x_m=0.2) inter-arrival gaps
    xm, alpha = 0.2, 1.5
    times = []
    tot, last = 0, 0.0
    while last < T:
        g = (rng.pareto(alpha, size=max(1024, int(2 * T / 0.6))) + 1.0) * xm
        c = last + np.cumsum(g)
        times.append(c)
        last = c[-1]
    times = np.concatenate(times)
    times = times[times < T]
    counts = np.bincount(times.astype(np.int64), minlength=T)[:T].astype(np.float64)
    ema = lfilter([0.05], [1.0, -0.95], counts)
    x = np.empty((T, M), np.float64)
    x[:, 0] = counts
    x[:, 1] = ema
    beta = rng.uniform(0.5, 2.0, M)
    noise = _ar1(rng, T, M)
    for m in range(2, M):
        x[:, m] = beta[m] * ema + noise[:, m]
    return x, lab


_GEN = {
    "ar1_spikes": _gen_ar1_spikes,
    "llm_service": _gen_llm_service,
    "diurnal_corr": _gen_diurnal_corr,
    "ar1_bursts": _gen_ar1_bursts,
    "ragged_mix": _gen_ragged_mix,
}


def _seed_tree(cfg: Config):
    root = np.random.SeedSequence(cfg.data_seed)
    return root.spawn(cfg.n_streams + 1)


def stream_lengths(cfg: Config, kids=None) -> np.ndarray:
    """Length T_s of every stream of the config (int64 [n_streams])."""
    if cfg.t_len > 0:
        return np.full(cfg.n_streams, cfg.t_len, np.int64)
    kids = kids if kids is not None else _seed_tree(cfg)
    rng = np.random.default_rng(kids[0])
    return rng.integers(cfg.t_min, cfg.t_max + 1, size=cfg.n_streams).astype(np.int64)


def _default_threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def generate(cfg: Config, streams=None, threads: int | None = None, lengths=None) -> Workload:
    """Generate the config's streams (all, or the given subset of stream ids, in that order).

    ``lengths`` overrides the stream lengths (used by edge-case tests; every listed
    stream then gets that length instead of the config's).
    """
    kids = _seed_tree(cfg)
    all_T = stream_lengths(cfg, kids)
    ids = np.arange(cfg.n_streams, dtype=np.int64) if streams is None else np.asarray(streams, np.int64)
    Ts = all_T[ids] if lengths is None else np.asarray(lengths, np.int64)
    offs = np.zeros(len(ids) + 1, np.int64)
    np.cumsum(Ts, out=offs[1:])
    M = cfg.metrics
    total = int(offs[-1])
    bf16 = cfg.dtype == "bf16"
    x = None if bf16 else np.empty((total, M), np.float32)
    xb = np.empty((total, M), np.uint16) if bf16 else None
    labels = np.zeros(total, np.uint8)
    gen = _GEN[cfg.kind]

    def one(i):
        s = int(ids[i])
        T = int(Ts[i])
        if T == 0:
            return
        rng = np.random.default_rng(kids[1 + s])
        xv, lab = gen(cfg, rng, T, s)
        a, b = int(offs[i]), int(offs[i + 1])
        if bf16:
            xb[a:b] = to_bf16_bits(xv.astype(np.float32))
        else:
            x[a:b] = xv
        labels[a:b] = lab

    nthr = threads or _default_threads()
    if nthr <= 1 or len(ids) <= 1:
        for i in range(len(ids)):
            one(i)
    else:
        with ThreadPoolExecutor(nthr) as ex:
            list(ex.map(one, range(len(ids))))
    return Workload(cfg=cfg, stream_offsets=offs, x=x, x_bits=xb, labels=labels, streams=ids,
                    seeds={"data_seed": cfg.data_seed, "weight_seed": cfg.weight_seed})


def constant_streams(cfg: Config, lengths, values) -> Workload:
    """Streams whose every metric is the given constant (one value per stream)."""
    Ts = np.asarray(lengths, np.int64)
    offs = np.zeros(len(Ts) + 1, np.int64)
    np.cumsum(Ts, out=offs[1:])
    x = np.empty((int(offs[-1]), cfg.metrics), np.float32)
    for i, v in enumerate(values):
        x[offs[i]:offs[i + 1]] = v
    bits = None
    if cfg.dtype == "bf16":
        bits = to_bf16_bits(x)
        x = None
    return Workload(cfg=cfg, stream_offsets=offs, x=x, x_bits=bits,
                    labels=np.zeros(int(offs[-1]), np.uint8), streams=np.arange(len(Ts)))


def from_arrays(cfg: Config, x, stream_offsets) -> Workload:
    """Wrap caller-made float arrays (rounded to bf16 for bf16 configs)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    offs = np.asarray(stream_offsets, np.int64)
    bits = None
    if cfg.dtype == "bf16":
        bits = to_bf16_bits(x)
        x = None
    return Workload(cfg=cfg, stream_offsets=offs, x=x, x_bits=bits,
                    labels=np.zeros(int(offs[-1]), np.uint8), streams=np.arange(len(offs) - 1))


# ----------------------------------------------------------------------------- training batches
@dataclass
class TrainBatch:
    """One labelled batch for a training step: V [B, D] float32 (rows flattened j = t*M + m),
    labels [B] float32 (+1 normal, -1 anomalous), eps [B, L] float32 (reparameterisation noise)."""
    V: np.ndarray
    labels: np.ndarray
    eps: np.ndarray


def training_batch(cfg: Config, batch: int, seed: int = 0, anomaly_frac: float = 0.1) -> TrainBatch:
    """Windows of W steps of M unit-variance AR(1) metrics (the scale of z-scored metrics).

    A fraction ``anomaly_frac`` of the rows (drawn per row) are anomalous: one random metric takes
    a level shift of U(3, 6) standard deviations, of random sign, from a random step to the end of
    the window. eps is standard normal. Every draw comes from ``default_rng(seed)``.
    """
    rng = np.random.default_rng(seed)
    W, M, L = cfg.window, cfg.metrics, cfg.latent
    e = rng.standard_normal((batch, W, M))
    e[:, 0] *= SIGMA_MARG
    x = lfilter([1.0], [1.0, -PHI], e, axis=1) / SIGMA_MARG
    anomalous = rng.random(batch) < anomaly_frac
    idx = np.flatnonzero(anomalous)
    metric = rng.integers(0, M, size=idx.size)
    start = rng.integers(0, W, size=idx.size)
    shift = rng.uniform(3.0, 6.0, size=idx.size) * rng.choice([-1.0, 1.0], size=idx.size)
    for r, m, t0, a in zip(idx, metric, start, shift):
        x[r, t0:, m] += a
    labels = np.where(anomalous, -1.0, 1.0).astype(np.float32)
    eps = rng.standard_normal((batch, L)).astype(np.float32)
    return TrainBatch(V=np.ascontiguousarray(x.reshape(batch, W * M), dtype=np.float32), labels=labels, eps=eps)


# ----------------------------------------------------------------------------- configuration series
CONFIG_METRICS = ("n_f", "n_r", "n_a", "n_p", "t_r", "m_u", "g_u")   # Table II order


def config_series(n_streams: int, T: int, seed: int = 0) -> Workload:
    """Serving metrics of n_streams services over T steps (one step = one minute), Table II order.

    Arrivals n^a ~ Poisson(lambda_t), lambda_t = base (1 + 0.5 sin(2 pi (t + phase) / 1440)).
    Even streams have capacity C = 3 base (never saturated), odd streams C = 0.8 base (saturated
    around the daily peak). Execution time t^r = t0 (1 + 0.5 min(lambda_t / C, 1.5)) LogNormal(0, 0.05).
    Below capacity the running requests n^r ~ Poisson(lambda_t t^r) and the finished rate follows
    them (Little's law), n^f = n^r / t^r + N(0, 0.02 base); at capacity n^r ~ Poisson(C t^r)
    fluctuates around the concurrency limit and n^f = C + N(0, 0.05 C) does not follow it.
    Pending n^p ~ Poisson(5 max(0, lambda_t - C)); GPU memory use
    m^u = 0.05 + 0.9 min(1, n^r / R) + N(0, 0.005) with R = 2 C t0; GPU use
    g^u = logistic(4 (lambda_t / C - 0.7)) + N(0, 0.02), clipped to [0, 1].
    """
    rng = np.random.default_rng(seed)
    x = np.empty((n_streams * T, len(CONFIG_METRICS)), np.float32)
    t = np.arange(T, dtype=np.float64)
    for s in range(n_streams):
        base = rng.uniform(20.0, 80.0)
        phase = rng.uniform(0.0, 1440.0)
        cap = base * (3.0 if s % 2 == 0 else 0.8)
        t0 = rng.uniform(1.0, 4.0)
        lam = base * (1.0 + 0.5 * np.sin(2.0 * math.pi * (t + phase) / 1440.0))
        sat = lam >= cap
        n_a = rng.poisson(lam)
        t_r = t0 * (1.0 + 0.5 * np.minimum(lam / cap, 1.5)) * rng.lognormal(0.0, 0.05, T)
        n_r = rng.poisson(np.minimum(lam, cap) * t_r).astype(np.float64)
        n_f = np.where(sat, cap + rng.normal(0.0, 0.05 * cap, T), n_r / t_r + rng.normal(0.0, 0.02 * base, T))
        n_p = rng.poisson(5.0 * np.maximum(0.0, lam - cap))
        m_u = 0.05 + 0.9 * np.minimum(1.0, n_r / (2.0 * cap * t0)) + rng.normal(0.0, 0.005, T)
        g_u = np.clip(1.0 / (1.0 + np.exp(-4.0 * (lam / cap - 0.7))) + rng.normal(0.0, 0.02, T), 0.0, 1.0)
        x[s * T:(s + 1) * T] = np.stack([n_f, n_r, n_a, n_p, t_r, m_u, g_u], axis=1)
    offs = np.arange(n_streams + 1, dtype=np.int64) * T
    cfg = Config(name="config", n_streams=n_streams, metrics=len(CONFIG_METRICS), t_len=T, t_min=0, t_max=0,
                 window=64, stride=1, hidden=1, latent=1, dtype="f32", act="relu", ref_frac=0.5,
                 kind="config_series", data_seed=seed, weight_seed=0)
    return Workload(cfg=cfg, stream_offsets=offs, x=x, x_bits=None,
                    labels=np.zeros(n_streams * T, np.uint8), streams=np.arange(n_streams))
