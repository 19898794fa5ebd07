"""Oracle for the ENOVA detection path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct CPU implementation of what the detector of
Section IV-B ("Performance Detection Module") computes, in fp64:

* window enumeration over each stream (Table II observation windows);
* reference statistics and normalisation (inputs are normalised before the VAE);
* the VAE encoder, the KL-divergence score of the posterior from the prior and
  the Mean-Difference direction from the reconstruction (``core.c``);
* the peaks-over-threshold threshold (the method of Siffer et al. cited in
  Section IV-B) fitted by maximum likelihood with Grimshaw's reduction, and the
  "score exceeds threshold" flag;
* its streaming form (SPOT, ``Spot``): per-stream thresholds updated score by score.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg
may import this package. It shares no code with the HIP library and never
imports it. Every function below states the passage it follows; the pins that
tie it to the paper and to the mathematics live in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "core.c")
_BUILD = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD, "liboracle.so")
_lib = None

ACT = {"relu": 0, "tanh": 1}


def build(force: bool = True) -> str:
    """Compile core.c with gcc (fp64, no FMA contraction, OpenMP over windows)."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    os.makedirs(_BUILD, exist_ok=True)
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC",
           _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    I = ctypes.c_int
    lib.oracle_ref_stats.argtypes = [P, I64, I, P, P]
    lib.oracle_ref_stats.restype = None
    lib.oracle_window_debug.argtypes = [P, I, I, I, I64, I, I, I] + [P] * 10 + [P, P, I, P, P, P]
    lib.oracle_window_debug.restype = None
    lib.oracle_score_batch.argtypes = ([P, P, I, I, I, I, I, I, I, P] + [P] * 10 +
                                       [I, P, P, P, P, P, P, P, P, P, I])
    lib.oracle_score_batch.restype = I
    lib.oracle_score_pairs.argtypes = ([P, P, I, I, I, I, I, I, I, P] + [P] * 10 +
                                       [I, P, P, P, P, I64, P, P, P, I])
    lib.oracle_score_pairs.restype = I
    lib.oracle_bf16_round_array.argtypes = [P, P, I64]
    lib.oracle_bf16_round_array.restype = None
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------- windows
def window_count(T, W, S):
    """Windows of a stream of length T: k*S + W <= T for k = 0, 1, ... (partial tail dropped).

    Table II observes each metric over a window of consecutive steps; windows
    start at step 0 and advance by the stride.
    """
    T = np.asarray(T, np.int64)
    return np.where(T >= W, (T - W) // S + 1, 0).astype(np.int64)


def window_offsets(stream_offsets, W, S):
    T = np.diff(np.asarray(stream_offsets, np.int64))
    off = np.zeros(len(T) + 1, np.int64)
    np.cumsum(window_count(T, W, S), out=off[1:])
    return off


def ref_len(T, ref_frac):
    """Reference-prefix length R = floor(ref_frac * T) (the training half of Section VI's split)."""
    rf = float(np.float32(ref_frac))
    T = np.asarray(T, np.int64)
    return np.floor(rf * T.astype(np.float64)).astype(np.int64)


def calibration_count(T, W, S, ref_frac):
    """Windows lying wholly inside the reference prefix: k*S + W <= R."""
    return window_count(ref_len(T, ref_frac), W, S)


def bf16_round(a):
    """Nearest bfloat16 value of each fp64 entry, ties to even, rounded once from fp64.

    The bf16 workload stores the normalised inputs as bfloat16; step 3 of the window
    evaluation applies this to v = (x - mean) / std computed in fp64.
    """
    lib = _load()
    a = _f64(a)
    out = np.empty_like(a)
    if a.size:
        lib.oracle_bf16_round_array(_ptr(a), _ptr(out), a.size)
    return out


# ----------------------------------------------------------------------------- statistics
def ref_stats(x, stream_offsets, ref_frac):
    """Per-stream, per-metric mean and population std over the reference prefix (fp64)."""
    lib = _load()
    x = _f64(x)
    offs = np.asarray(stream_offsets, np.int64)
    n, M = len(offs) - 1, x.shape[1]
    R = ref_len(np.diff(offs), ref_frac)
    mean = np.empty((n, M))
    std = np.empty((n, M))
    for s in range(n):
        lib.oracle_ref_stats(_ptr(x[offs[s]:]) if offs[s] < len(x) else _ptr(x), int(R[s]), M,
                             _ptr(mean[s]), _ptr(std[s]))
    return mean, std


# ----------------------------------------------------------------------------- scoring
def score(x, stream_offsets, *, window, stride, weights, act="relu", ref_frac=0.5,
          bf16=False, ref_mean=None, ref_std=None, max_windows=None, threads=0,
          return_stats=False):
    """Scores and MD of every window (fp64), laid out like the library's output.

    ``weights`` is a dict of arrays w1 [H,D], b1, wmu [L,H], bmu, wlv, blv, wd1 [H,L],
    bd1, wd2 [D,H], bd2. ``max_windows`` scores only the first that many windows of
    each stream (the rest are NaN). Returns (scores, md) or (scores, md, info).
    """
    lib = _load()
    x = _f64(x)
    offs = np.ascontiguousarray(stream_offsets, np.int64)
    n = len(offs) - 1
    M = x.shape[1] if x.ndim == 2 else 1
    W, S = int(window), int(stride)
    w = {k: _f64(v) for k, v in weights.items()}
    H, D = w["w1"].shape
    L = w["wmu"].shape[0]
    assert D == W * M, "W1 must have W*M columns"
    T = np.diff(offs)
    nwin = window_count(T, W, S)
    woff = np.zeros(n + 1, np.int64)
    np.cumsum(nwin, out=woff[1:])
    cnt = nwin if max_windows is None else np.minimum(nwin, int(max_windows))
    R = ref_len(T, ref_frac)
    N = int(woff[-1])
    sc = np.full(N, np.nan)
    md = np.full(N, np.nan)
    mds = np.full(N, np.nan)
    mean_o = np.empty((max(n, 1), M))
    std_o = np.empty((max(n, 1), M))
    em = es = None
    if ref_mean is not None:
        em = _f64(np.asarray(ref_mean).reshape(n, M))
        es = _f64(np.asarray(ref_std).reshape(n, M))
    if x.size == 0:
        x = np.zeros((1, M))
    used = 0
    if n > 0:
        used = lib.oracle_score_batch(
            _ptr(x), _ptr(offs), n, M, W, S, H, L, ACT[act], _ptr(R),
            _ptr(w["w1"]), _ptr(w["b1"]), _ptr(w["wmu"]), _ptr(w["bmu"]), _ptr(w["wlv"]),
            _ptr(w["blv"]), _ptr(w["wd1"]), _ptr(w["bd1"]), _ptr(w["wd2"]), _ptr(w["bd2"]),
            1 if bf16 else 0, _ptr(em), _ptr(es), _ptr(woff), _ptr(cnt),
            _ptr(sc), _ptr(md), _ptr(mds), _ptr(mean_o), _ptr(std_o), int(threads))
    if return_stats:
        return sc, md, {"window_offsets": woff, "mean": mean_o[:n], "std": std_o[:n],
                        "threads": used, "ref_len": R, "md_scale": mds}
    return sc, md


def score_pairs(x, stream_offsets, streams, ks, *, window, stride, weights, act="relu",
                ref_frac=0.5, bf16=False, ref_mean=None, ref_std=None, threads=0):
    """Scores, MD and MD scale (mean|v| + mean|m'|) of window ks[i] of stream streams[i]."""
    lib = _load()
    x = _f64(x)
    offs = np.ascontiguousarray(stream_offsets, np.int64)
    n = len(offs) - 1
    M = x.shape[1]
    w = {k: _f64(v) for k, v in weights.items()}
    H, D = w["w1"].shape
    L = w["wmu"].shape[0]
    assert D == window * M
    ps = np.ascontiguousarray(streams, np.int32)
    pk = np.ascontiguousarray(ks, np.int64)
    nwin = window_count(np.diff(offs), window, stride)
    assert np.all(pk >= 0) and np.all(pk < nwin[ps]), "window index out of range"
    R = ref_len(np.diff(offs), ref_frac)
    em = es = None
    if ref_mean is not None:
        em = _f64(np.asarray(ref_mean).reshape(n, M))
        es = _f64(np.asarray(ref_std).reshape(n, M))
    npairs = len(ps)
    sc, md, mds = np.empty(npairs), np.empty(npairs), np.empty(npairs)
    if npairs:
        lib.oracle_score_pairs(
            _ptr(x), _ptr(offs), n, M, int(window), int(stride), H, L, ACT[act], _ptr(R),
            _ptr(w["w1"]), _ptr(w["b1"]), _ptr(w["wmu"]), _ptr(w["bmu"]), _ptr(w["wlv"]),
            _ptr(w["blv"]), _ptr(w["wd1"]), _ptr(w["bd1"]), _ptr(w["wd2"]), _ptr(w["bd2"]),
            1 if bf16 else 0, _ptr(em), _ptr(es), _ptr(ps), _ptr(pk), npairs,
            _ptr(sc), _ptr(md), _ptr(mds), int(threads))
    return sc, md, mds


def window_debug(x_stream, k, *, window, stride, weights, mean, std, act="relu", bf16=False):
    """One window with every intermediate: dict(v, h, mu, lv, hd, mrec, score, md)."""
    lib = _load()
    xs = _f64(x_stream)
    M = xs.shape[1]
    w = {kk: _f64(v) for kk, v in weights.items()}
    H, D = w["w1"].shape
    L = w["wmu"].shape[0]
    dbg = np.empty(2 * D + 2 * H + 2 * L)
    sc = ctypes.c_double()
    md = ctypes.c_double()
    lib.oracle_window_debug(_ptr(xs), M, int(window), int(stride), int(k), H, L, ACT[act],
                            _ptr(w["w1"]), _ptr(w["b1"]), _ptr(w["wmu"]), _ptr(w["bmu"]),
                            _ptr(w["wlv"]), _ptr(w["blv"]), _ptr(w["wd1"]), _ptr(w["bd1"]),
                            _ptr(w["wd2"]), _ptr(w["bd2"]), _ptr(_f64(mean)), _ptr(_f64(std)),
                            1 if bf16 else 0, ctypes.byref(sc), ctypes.byref(md), _ptr(dbg))
    o = 0
    out = {}
    for name, size in (("v", D), ("h", H), ("mu", L), ("lv", L), ("hd", H), ("mrec", D)):
        out[name] = dbg[o:o + size].copy()
        o += size
    out["score"] = sc.value
    out["md"] = md.value
    return out


# ----------------------------------------------------------------------------- POT
GRID = 512          # grid points per admissible interval for the roots of u(x) v(x) = 1
BISECT_ITERS = 200  # bisection steps (stops earlier once the bracket cannot shrink)


def _gpd_loglik(Y, gamma, sigma):
    """GPD log-likelihood of excesses Y (gamma = 0 is the exponential)."""
    N = len(Y)
    if sigma <= 0:
        return -math.inf
    if gamma == 0.0:
        return -N * math.log(sigma) - float(np.sum(Y)) / sigma
    r = gamma * Y / sigma
    if np.any(r <= -1.0):
        return -math.inf
    return -N * math.log(sigma) - (1.0 + 1.0 / gamma) * float(np.sum(np.log1p(r)))


def gpd_grid(ymean, ymin, ymax):
    """Evaluation grid of Grimshaw's equation over both admissible intervals of x = gamma/sigma.

    Right interval (0, B], B = 2 (mean - min) / min^2: GRID points geometric from
    eps = 1e-8/mean to B. Left interval (-1/Y_max, 0): x = -f/Y_max with f the logistic of
    GRID points linear in z from logit(eps*Y_max) to 30, i.e. geometric towards both 0 and the
    endpoint -1/Y_max. Returns a list of increasing-index arrays, one per interval.
    """
    eps = 1e-8 / ymean
    out = []
    f0 = eps * ymax
    if f0 < 0.5:
        zlo = math.log(f0 / (1.0 - f0))
        zhi = 30.0
        xs = []
        for i in range(GRID):
            z = zlo + (zhi - zlo) * i / (GRID - 1)
            xs.append(-(1.0 / (1.0 + math.exp(-z))) / ymax)
        out.append(xs)
    right = 2.0 * (ymean - ymin) / (ymin * ymin)
    if right > 2.0 * eps:
        ratio = right / eps
        out.append([eps * ratio ** (i / (GRID - 1)) for i in range(GRID)])
    return out


def grimshaw(Y):
    """Maximum-likelihood GPD fit of excesses Y by Grimshaw's reduction.

    With x = gamma / sigma the likelihood equations reduce to u(x) v(x) = 1 with
    u(x) = mean 1/(1 + x Y) and v(x) = 1 + mean log(1 + x Y); a root gives
    gamma = v(x) - 1 and sigma = gamma / x. The equation is evaluated without cancellation
    as w = b - a - a b, a = mean(xY/(1+xY)) = 1 - u, b = mean log1p(xY) = v - 1. Roots are
    bracketed on the geometric grids of ``gpd_grid`` and bisected; the exponential
    (gamma = 0, sigma = mean) is always a candidate; the candidate of largest
    log-likelihood wins (ties: smaller |gamma|). Returns (gamma, sigma, loglik).
    """
    Y = np.asarray(Y, np.float64)
    ymax, ymin, ymean = float(Y.max()), float(Y.min()), float(Y.mean())

    def w(xv):
        xy = xv * Y
        a = float(np.mean(xy / (1.0 + xy)))
        b = float(np.mean(np.log1p(xy)))
        return b - a - a * b

    roots = []
    for xs in gpd_grid(ymean, ymin, ymax):
        ws = [w(xv) for xv in xs]
        for i in range(len(xs) - 1):
            if ws[i] == 0.0:
                roots.append(xs[i])
                continue
            if ws[i] * ws[i + 1] < 0.0:
                lo, hi, wlo = xs[i], xs[i + 1], ws[i]
                for _ in range(BISECT_ITERS):
                    mid = 0.5 * (lo + hi)
                    if mid == lo or mid == hi:
                        break
                    wm = w(mid)
                    if wm == 0.0:
                        lo = hi = mid
                        break
                    if (wm < 0.0) == (wlo < 0.0):
                        lo, wlo = mid, wm
                    else:
                        hi = mid
                roots.append(0.5 * (lo + hi))
        if ws[-1] == 0.0:
            roots.append(xs[-1])
    best = (0.0, ymean, _gpd_loglik(Y, 0.0, ymean))
    for xr in roots:
        gamma = float(np.mean(np.log1p(xr * Y)))
        if gamma == 0.0:
            continue
        sigma = gamma / xr
        ll = _gpd_loglik(Y, gamma, sigma)
        if ll > best[2] or (ll == best[2] and abs(gamma) < abs(best[0])):
            best = (gamma, sigma, ll)
    return best


def pot_fit(t, n, Y, q=1e-3):
    """z_q from the excesses Y over t among n observations (the tail model of Siffer et al.,
    the peaks-over-threshold method Section IV-B cites).

    The tail above t is a generalised Pareto distribution GPD(gamma, sigma) and
        z_q = t + sigma/gamma * ((q n / N_t)^(-gamma) - 1)   (gamma != 0)
        z_q = t - sigma * log(q n / N_t)                      (gamma = 0).
    N_t >= 10: maximum likelihood (``grimshaw``); 2 <= N_t < 10: method of moments with the
    unbiased sample variance; N_t <= 1 (or zero variance): z_q = t. Returns (z_q, info dict).
    """
    Y = np.asarray(Y, np.float64)
    Nt = int(Y.size)
    info = {"t": t, "n": n, "n_peaks": Nt, "gamma": None, "sigma": None, "method": None}
    if Nt >= 10:
        gamma, sigma, _ = grimshaw(Y)
        info["method"] = "mle"
    elif Nt >= 2:
        m = float(Y.mean())
        s2 = float(Y.var(ddof=1))
        if s2 <= 0.0:
            info["method"] = "t"
            return t, info
        gamma = 0.5 * (1.0 - m * m / s2)
        sigma = 0.5 * m * (1.0 + m * m / s2)
        info["method"] = "moments"
    else:
        info["method"] = "t"
        return t, info
    info["gamma"], info["sigma"] = gamma, sigma
    r = q * n / Nt
    if abs(gamma) < 1e-9:
        z = t - sigma * math.log(r)
    else:
        z = t + sigma / gamma * (r ** (-gamma) - 1.0)
    return float(z), info


def pot_threshold(calib_scores, level=0.98, q=1e-3):
    """Peaks-over-threshold anomaly threshold z_q over calibration scores.

    t = the level-quantile (order statistic at ceil(level*n) - 1 of the sorted scores),
    excesses Y = {c - t : c > t}, z_q from ``pot_fit``. Returns (z_q, info dict).
    """
    C = np.sort(np.asarray(calib_scores, np.float64).ravel())
    n = C.size
    if n == 0:
        raise ValueError("no calibration scores")
    idx = max(int(math.ceil(level * n)) - 1, 0)
    t = float(C[idx])
    return pot_fit(t, n, C[C > t] - t, q)


class Spot:
    """Streaming peaks-over-threshold of one stream: SPOT of Siffer et al. (the POT method that
    Section IV-B cites; Section V runs the detector inside a stream-computing job).

    Start: ``pot_threshold`` over the stream's calibration scores gives t, the peaks Y and z_q,
    with n = the number of calibration scores (no calibration score: t = z_q = +inf and the
    model never changes, so the stream never flags). Then each new score s, in time order:
      s > z_q          an alarm (flag 1); the model is left as it is;
      t < s <= z_q     s - t joins the peaks, n += 1, and z_q is refitted (``pot_fit``) on all
                       peaks with the new n;
      s <= t           n += 1 only (z_q changes at the next peak);
      s is NaN         flag 0, nothing changes.
    Readings taken here (the paper is silent): once ``peak_cap`` peaks are stored the model is frozen (later
    scores are only compared); a stream's level and q are those of the batch threshold.
    """

    def __init__(self, calib_scores, level=0.98, q=1e-3, peak_cap=None):
        C = np.sort(np.asarray(calib_scores, np.float64).ravel())
        self.q = q
        self.cap = peak_cap
        if C.size == 0:
            self.t = self.z = math.inf
            self.n = 0
            self.Y = []
            return
        idx = max(int(math.ceil(level * C.size)) - 1, 0)
        self.t = float(C[idx])
        self.Y = [float(v) for v in C[C > self.t] - self.t]
        self.n = int(C.size)
        if self.cap is not None and len(self.Y) > self.cap:
            raise ValueError("more calibration peaks than the peak capacity")
        self.z, _ = pot_fit(self.t, self.n, self.Y, q)

    def frozen(self):
        return math.isinf(self.t) or (self.cap is not None and len(self.Y) >= self.cap)

    def step(self, s):
        """Process one score; returns its flag (0/1)."""
        if math.isnan(s):
            return 0
        if s > self.z:
            return 1
        if self.frozen():
            return 0
        self.n += 1
        if s > self.t:
            self.Y.append(s - self.t)
            self.z, _ = pot_fit(self.t, self.n, self.Y, self.q)
        return 0


def calibration_scores(scores, stream_offsets, *, window, stride, ref_frac=0.5):
    """Scores of the windows that lie wholly in each stream's reference prefix."""
    offs = np.asarray(stream_offsets, np.int64)
    T = np.diff(offs)
    nwin = window_count(T, window, stride)
    woff = np.zeros(len(T) + 1, np.int64)
    np.cumsum(nwin, out=woff[1:])
    ncal = np.minimum(calibration_count(T, window, stride, ref_frac), nwin)
    parts = [np.asarray(scores)[woff[s]:woff[s] + ncal[s]] for s in range(len(T))]
    return np.concatenate(parts) if parts else np.zeros(0)


def flags(scores, threshold):
    """An anomaly is a window whose score strictly exceeds the threshold."""
    return (np.asarray(scores, np.float64) > threshold).astype(np.uint8)
