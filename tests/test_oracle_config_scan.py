"""Pins of the configuration-scan oracle (Section IV-A, Eqs. (4)-(6)): OLS against least squares
and scipy's linregress, the t-test decision against the p-value, critical values against printed
table values, Silverman's bandwidth on a hand example, the KDE against scipy's gaussian_kde, the
quantile by its defining equation, and the regime logic on series built to have or lack a
relation between n^f and n^r."""
import math

import numpy as np
import pytest
from scipy import stats

import oracle
from oracle import config_scan as cs


def test_ols_matches_least_squares_and_linregress():
    rng = np.random.default_rng(0)
    for trial in range(20):
        n = int(rng.integers(3, 200))
        x = rng.normal(5, 2, n)
        y = 1.5 - 0.7 * x + rng.normal(0, 1 + trial % 3, n)
        r = cs.ols(x, y)
        A = np.stack([np.ones(n), x], axis=1)
        (a, b), *_ = np.linalg.lstsq(A, y, rcond=None)
        assert r["a"] == pytest.approx(a, rel=1e-10, abs=1e-12)
        assert r["b"] == pytest.approx(b, rel=1e-10, abs=1e-12)
        lr = stats.linregress(x, y)
        assert r["t"] == pytest.approx(lr.slope / lr.stderr, rel=1e-9)


def test_t_test_decision_is_the_p_value_decision():
    rng = np.random.default_rng(1)
    for alpha in (0.05, 0.01):
        for n in (5, 32, 64):
            tc = cs.t_critical(alpha, n - 2)
            for _ in range(50):
                x = rng.normal(0, 1, n)
                y = 0.3 * x + rng.normal(0, 1, n)
                r = cs.ols(x, y)
                p = stats.linregress(x, y).pvalue
                if abs(p - alpha) > 1e-9:
                    assert (abs(r["t"]) > tc) == (p < alpha)


def test_critical_values_against_printed_tables():
    # two-sided 5% and 1% critical values of Student's t (standard printed tables)
    assert cs.t_critical(0.05, 10) == pytest.approx(2.228, abs=5e-4)
    assert cs.t_critical(0.05, 30) == pytest.approx(2.042, abs=5e-4)
    assert cs.t_critical(0.01, 20) == pytest.approx(2.845, abs=5e-4)
    assert cs.t_critical(0.05, 10 ** 7) == pytest.approx(1.960, abs=5e-4)


def test_ols_degenerate_cases():
    x = np.full(10, 3.0)
    y = np.arange(10.0)
    r = cs.ols(x, y)
    assert r["b"] == 0.0 and r["t"] == 0.0 and r["a"] == pytest.approx(4.5)
    x = np.arange(10.0)
    r = cs.ols(x, 2.0 + 0.5 * x)
    assert r["b"] == pytest.approx(0.5) and math.isinf(r["t"]) and r["t"] > 0
    r = cs.ols(x, np.full(10, 7.0))
    assert r["b"] == 0.0 and r["t"] == 0.0 and r["a"] == 7.0


def test_silverman_bandwidth_hand_example():
    v = np.array([1.0, 2.0, 3.0, 4.0, 5.0, 6.0, 7.0, 8.0])
    sd = math.sqrt(42.0 / 7.0)                  # sum of squared deviations 42, n - 1 = 7
    iqr = 6.25 - 2.75                           # quantiles at positions 5.25 and 1.75
    assert cs.silverman_bandwidth(v) == pytest.approx(0.9 * min(sd, iqr / 1.34) * 8 ** -0.2)
    # IQR = 0 but spread: falls back to sd
    w = np.array([0.0] * 10 + [5.0])
    sd_w = float(np.std(w, ddof=1))
    assert cs.silverman_bandwidth(w) == pytest.approx(0.9 * sd_w * 11 ** -0.2)
    assert cs.silverman_bandwidth(np.full(6, 2.5)) == 0.0


def test_kde_cdf_matches_scipy_gaussian_kde():
    rng = np.random.default_rng(2)
    v = rng.gamma(2.0, 3.0, 64)
    h = cs.silverman_bandwidth(v)
    kde = stats.gaussian_kde(v, bw_method=h / np.std(v, ddof=1))
    for xq in (-5.0, 1.0, 4.0, 9.0, 30.0):
        assert cs.kde_cdf(v, h, xq) == pytest.approx(kde.integrate_box_1d(-np.inf, xq), abs=1e-10)


def test_kde_quantile_solves_its_equation():
    rng = np.random.default_rng(3)
    v = rng.normal(10, 2, 64)
    h = cs.silverman_bandwidth(v)
    for q in (0.01, 0.5, 0.99):
        xq = cs.kde_quantile(v, q)
        assert cs.kde_cdf(v, h, xq) == pytest.approx(q, abs=1e-12)
    assert cs.kde_quantile(np.full(8, 3.25), 0.99) == 3.25
    # symmetric sample: the median of its KDE is the centre
    sym = np.array([-3.0, -1.0, -0.5, 0.5, 1.0, 3.0])
    assert cs.kde_quantile(sym, 0.5) == pytest.approx(0.0, abs=1e-12)


def _stream(rng, T, related):
    nr = rng.poisson(40, T).astype(np.float64)
    if related:
        nf = 0.5 * nr + rng.normal(0, 1.0, T)          # still tracks the running requests
    else:
        nf = 20.0 + rng.normal(0, 1.0, T)              # saturated: independent of them
    tr = 2.0 + 0.05 * nr + rng.normal(0, 0.1, T)
    mu = 0.1 + 0.002 * nr
    return np.stack([nf, nr, tr, mu], axis=1)


def test_regimes_and_configuration():
    rng = np.random.default_rng(4)
    T, W = 300, 64
    x = np.concatenate([_stream(rng, T, True), _stream(rng, T, False)])
    offs = np.array([0, T, 2 * T])
    out = cs.stream_config(x, offs, window=W, stride=1, col_f=0, col_r=1, col_t=2, col_m=3)
    assert out["sig"][0] == 1 and out["sig"][1] == 0
    last = [x[T - W:T], x[2 * T - W:2 * T]]
    # related: n_limit is an upper-tail value; saturated: the centre of the window
    assert out["n_limit"][0] > np.quantile(last[0][:, 0], 0.95)
    assert abs(out["n_limit"][1] - np.median(last[1][:, 0])) < 0.5
    assert out["max_num_seqs"][1] == pytest.approx(out["n_limit"][1] * out["t_limit"][1])
    # m^u is exactly linear in n^r, so gpu_memory is that line at max_num_seqs
    for s in (0, 1):
        assert out["gpu_memory"][s] == pytest.approx(0.1 + 0.002 * out["max_num_seqs"][s], rel=1e-9)


def test_window_scan_order_and_short_streams():
    rng = np.random.default_rng(5)
    lens = [10, 3, 0, 25]
    x = np.concatenate([_stream(rng, T, True) for T in lens]) if sum(lens) else np.zeros((0, 4))
    offs = np.concatenate([[0], np.cumsum(lens)])
    W, S = 5, 2
    r = cs.window_scan(x, offs, window=W, stride=S, col_f=0, col_r=1, col_m=3)
    woff = oracle.window_offsets(offs, W, S)
    assert len(r["b"]) == woff[-1]
    # window k of stream 3
    k = 4
    w = x[offs[3] + k * S:offs[3] + k * S + W]
    f = cs.ols(w[:, 1], w[:, 0])
    assert r["b"][woff[3] + k] == f["b"] and r["t"][woff[3] + k] == f["t"]
