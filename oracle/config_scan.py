"""Oracle of the configuration module's scans (Section IV-A, Eqs. (4)-(6), Table II) -- TEST
INFRASTRUCTURE ONLY, plain fp64 Python/numpy.

Section IV-A sets max_num_seqs ~ n_limit * t^r_limit (Eq. (4)) from the monitoring series of a
service: it first asks whether the finished-request rate n^f still depends on the number of
running requests n^r, by an ordinary-least-squares fit n^f = f(n^r) (Eq. (5)) and a t-test of its slope.
A significant relation means n^f has not yet reached its limit, so n_limit and t^r_limit are
taken from the extreme values of the observed window; no relation means n^f sits at its limit
and they come from the centre of a normal-like distribution. Both are read off a kernel density
estimate of the window's observations. The GPU memory is then g(max_num_seqs) for an OLS fit
m^u = g(n^r) (Eq. (6)).

Readings taken here (the paper fixes none of them):

* windows are the detector's: W steps, stride S, from step 0 of every stream (Table II);
* the t-test is two-sided at level alpha on the slope, with W - 2 degrees of freedom:
  t = b / sqrt(RSS / ((W - 2) Sxx)), significant iff |t| > t_{1 - alpha/2, W-2};
  a window whose n^r is constant (Sxx = 0) has no relation (b = 0, a = mean of n^f, t = 0);
  RSS = 0 with b != 0 gives |t| = inf (significant);
* the KDE is Gaussian with Silverman's rule of thumb, h = 0.9 min(sd, IQR / 1.34) W^(-1/5)
  (sd with W - 1 in the denominator, IQR from linearly interpolated sample quantiles); IQR = 0
  falls back to sd, and h = 0 (a constant window) makes the estimate a point mass;
* n_limit and t^r_limit are the KDE quantiles at level q_extreme (significant relation) or 0.5
  (no relation) of the stream's last window of n^f and of t^r; the quantile is found by bisection
  on the KDE's distribution function;
* max_num_seqs = n_limit * t^r_limit; gpu_memory = g0 + g1 * max_num_seqs with (g0, g1) the OLS
  fit of m^u on n^r over the same last window.
"""
from __future__ import annotations

import math

import numpy as np
from scipy import stats

from . import window_count


def t_critical(alpha: float, dof: int) -> float:
    """Two-sided critical value t_{1 - alpha/2, dof} of Student's t distribution."""
    return float(stats.t.ppf(1.0 - alpha / 2.0, dof))


def ols(x, y):
    """Ordinary least squares y = a + b x by the centred closed form, with the slope's t statistic.

    Returns dict(a, b, t, sxx, sxy, syy, rss). Degenerate cases as in the module docstring."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    n = x.size
    xm = x.sum() / n
    ym = y.sum() / n
    dx = x - xm
    dy = y - ym
    sxx = float(np.dot(dx, dx))
    sxy = float(np.dot(dx, dy))
    syy = float(np.dot(dy, dy))
    if sxx == 0.0:
        return dict(a=ym, b=0.0, t=0.0, sxx=sxx, sxy=sxy, syy=syy, rss=syy)
    b = sxy / sxx
    a = ym - b * xm
    rss = max(syy - b * sxy, 0.0)
    if b == 0.0:
        t = 0.0
    elif rss == 0.0:
        t = math.copysign(math.inf, b)
    else:
        t = b * math.sqrt((n - 2) * sxx / rss)
    return dict(a=a, b=b, t=t, sxx=sxx, sxy=sxy, syy=syy, rss=rss)


def window_scan(x, stream_offsets, *, window, stride, col_f, col_r, col_m, alpha=0.05):
    """Every window of every stream: the OLS of n^f on n^r (a, b, t, significant) and of m^u on n^r
    (g0, g1). x: [sum T, M] float; returns a dict of arrays of length N (window order = stream
    order, then window index)."""
    x = np.asarray(x, np.float64)
    tc = t_critical(alpha, window - 2)
    out = {k: [] for k in ("a", "b", "t", "sig", "g0", "g1")}
    offs = np.asarray(stream_offsets, np.int64)
    for s in range(len(offs) - 1):
        T = int(offs[s + 1] - offs[s])
        seg = x[offs[s]:offs[s + 1]]
        for k in range(window_count(T, window, stride)):
            w = seg[k * stride:k * stride + window]
            f = ols(w[:, col_r], w[:, col_f])
            g = ols(w[:, col_r], w[:, col_m])
            out["a"].append(f["a"])
            out["b"].append(f["b"])
            out["t"].append(f["t"])
            out["sig"].append(1 if abs(f["t"]) > tc else 0)
            out["g0"].append(g["a"])
            out["g1"].append(g["b"])
    return {k: np.asarray(v, np.float64 if k != "sig" else np.uint8) for k, v in out.items()}


def sample_quantile(v, p):
    """Linearly interpolated sample quantile: sorted v at position (n - 1) p."""
    s = np.sort(np.asarray(v, np.float64))
    h = (s.size - 1) * p
    lo = int(math.floor(h))
    hi = min(lo + 1, s.size - 1)
    return float(s[lo] + (h - lo) * (s[hi] - s[lo]))


def silverman_bandwidth(v):
    """h = 0.9 min(sd, IQR/1.34) n^(-1/5); IQR = 0 falls back to sd."""
    v = np.asarray(v, np.float64)
    n = v.size
    m = v.sum() / n
    sd = math.sqrt(float(np.dot(v - m, v - m)) / (n - 1)) if n > 1 else 0.0
    iqr = sample_quantile(v, 0.75) - sample_quantile(v, 0.25)
    a = min(sd, iqr / 1.34) if iqr > 0.0 else sd
    return 0.9 * a * n ** (-0.2)


def kde_cdf(v, h, x):
    """Distribution function of the Gaussian KDE with bandwidth h > 0 at x."""
    v = np.asarray(v, np.float64)
    return float(np.mean([0.5 * math.erfc(-(x - vi) / (h * math.sqrt(2.0))) for vi in v]))


def kde_quantile(v, q):
    """Quantile at level q of the Gaussian KDE of v (Silverman bandwidth), by bisection."""
    v = np.asarray(v, np.float64)
    h = silverman_bandwidth(v)
    if h == 0.0:
        return float(v[0])
    lo, hi = float(v.min()) - 10.0 * h, float(v.max()) + 10.0 * h
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if mid <= lo or mid >= hi:
            break
        if kde_cdf(v, h, mid) < q:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def stream_config(x, stream_offsets, *, window, stride, col_f, col_r, col_t, col_m, alpha=0.05,
                  q_extreme=0.99):
    """The configuration read off each stream's last window (Eqs. (4)-(6)). Returns dict of arrays
    [n_streams]: sig, n_limit, t_limit, max_num_seqs, gpu_memory (NaN for a stream without a
    window)."""
    x = np.asarray(x, np.float64)
    tc = t_critical(alpha, window - 2)
    offs = np.asarray(stream_offsets, np.int64)
    n = len(offs) - 1
    out = {k: np.full(n, np.nan) for k in ("n_limit", "t_limit", "max_num_seqs", "gpu_memory")}
    out["sig"] = np.zeros(n, np.uint8)
    for s in range(n):
        T = int(offs[s + 1] - offs[s])
        nw = window_count(T, window, stride)
        if nw == 0:
            continue
        k = nw - 1
        w = x[offs[s] + k * stride:offs[s] + k * stride + window]
        f = ols(w[:, col_r], w[:, col_f])
        g = ols(w[:, col_r], w[:, col_m])
        sig = abs(f["t"]) > tc
        q = q_extreme if sig else 0.5
        nl = kde_quantile(w[:, col_f], q)
        tl = kde_quantile(w[:, col_t], q)
        out["sig"][s] = 1 if sig else 0
        out["n_limit"][s] = nl
        out["t_limit"][s] = tl
        out["max_num_seqs"][s] = nl * tl
        out["gpu_memory"][s] = g["a"] + g["b"] * nl * tl
    return out
