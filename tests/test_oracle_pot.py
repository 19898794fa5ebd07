"""Pins of the oracle's peaks-over-threshold threshold (CPU only)."""
import math

import numpy as np
import pytest
import scipy.stats as st

import oracle


@pytest.mark.parametrize("gamma0", [0.2, -0.2, 0.0, 0.5])
def test_grimshaw_matches_scipy_mle(gamma0):
    rng = np.random.default_rng(11)
    Y = st.genpareto.rvs(gamma0, scale=2.0, size=3000, random_state=rng)
    g, s, ll = oracle.grimshaw(Y)
    c, _, sc = st.genpareto.fit(Y, floc=0)
    ll_sp = float(st.genpareto.logpdf(Y, c, 0, sc).sum())
    # the grid+bisection root is at least as good as scipy's optimiser
    assert ll >= ll_sp - 1e-6 * abs(ll_sp)
    assert g == pytest.approx(c, abs=5e-3)
    assert s == pytest.approx(sc, rel=5e-3)
    # and our log-likelihood is the library's log-density summed
    assert ll == pytest.approx(float(st.genpareto.logpdf(Y, g, 0, s).sum()), rel=1e-10)


def test_grimshaw_recovers_parameters_within_3se():
    gamma, sigma, n = 0.2, 1.0, 20000
    rng = np.random.default_rng(12)
    Y = st.genpareto.rvs(gamma, scale=sigma, size=n, random_state=rng)
    g, s, _ = oracle.grimshaw(Y)
    se_g = (1 + gamma) / math.sqrt(n)
    se_s = sigma * math.sqrt(2 * (1 + gamma) / n)
    assert abs(g - gamma) < 3 * se_g
    assert abs(s - sigma) < 3 * se_s


def test_grimshaw_many_peaks_heavy_tail():
    """With many excesses Y_min is tiny, so the right admissible interval (0, 2(mean-min)/min^2]
    spans many decades; the root near gamma/sigma must still be bracketed (a linear grid puts it
    inside its first cell, where the sign of the equation at the left end is rounding noise)."""
    gamma, sigma, n = 0.1, 20.0, 100_000
    Y = st.genpareto.rvs(gamma, scale=sigma, size=n, random_state=np.random.default_rng(21))
    g, s, ll = oracle.grimshaw(Y)
    assert abs(g - gamma) < 3 * (1 + gamma) / math.sqrt(n)
    assert abs(s - sigma) < 3 * sigma * math.sqrt(2 * (1 + gamma) / n)
    assert ll > oracle._gpd_loglik(Y, 0.0, float(Y.mean()))
    # the same excesses in another order give the same fit
    g2, s2, _ = oracle.grimshaw(Y[::-1].copy())
    assert g2 == pytest.approx(g, rel=1e-9) and s2 == pytest.approx(s, rel=1e-9)


def test_exponential_tail_threshold_closed_form():
    """Exp(lam) scores: P(X > z) = e^(-lam z), so the q-quantile of the tail is -ln(q)/lam."""
    lam, q = 0.5, 1e-3
    zs = []
    for seed in range(5):
        C = np.random.default_rng(100 + seed).exponential(1.0 / lam, size=400_000)
        z, info = oracle.pot_threshold(C, level=0.98, q=q)
        assert info["method"] == "mle"
        zs.append(z)
    truth = -math.log(q) / lam
    assert abs(np.mean(zs) - truth) < 0.03 * truth


def test_quantile_index_and_strict_peaks():
    """t is the sorted value at ceil(level*n) - 1; values equal to t are not peaks."""
    C = np.arange(1, 101, dtype=float)          # 1..100
    z, info = oracle.pot_threshold(C, level=0.98, q=1e-3)
    assert info["t"] == 98.0 and info["n_peaks"] == 2 and info["method"] == "moments"
    # method of moments on excesses {1, 2}: mean 1.5, unbiased variance 0.5
    m, s2 = 1.5, 0.5
    g = 0.5 * (1 - m * m / s2)
    s = 0.5 * m * (1 + m * m / s2)
    assert info["gamma"] == pytest.approx(g) and info["sigma"] == pytest.approx(s)
    assert z == pytest.approx(98 + s / g * ((1e-3 * 100 / 2) ** (-g) - 1))
    C2 = np.concatenate([np.full(99, 5.0), [7.0]])
    z2, info2 = oracle.pot_threshold(C2)
    assert info2["t"] == 5.0 and info2["n_peaks"] == 1 and z2 == 5.0


def test_method_of_moments_inverts_gpd_moments():
    """GPD mean sigma/(1-g) and variance sigma^2/((1-g)^2 (1-2g)) give back (g, sigma)."""
    g0, s0 = -0.5, 2.0           # coefficient of variation 1/sqrt(1-2g) keeps every excess > 0
    mean = s0 / (1 - g0)
    var = s0 ** 2 / ((1 - g0) ** 2 * (1 - 2 * g0))
    base = np.array([-1.0, -0.5, 0.0, 0.5, 1.0])
    Y = mean + base / base.std(ddof=1) * math.sqrt(var)
    t = 10.0
    C = np.concatenate([np.full(300, t - 1.0), np.full(45, t), t + Y])
    z, info = oracle.pot_threshold(C, level=0.98)
    assert info["n_peaks"] == 5 and info["t"] == t
    assert info["gamma"] == pytest.approx(g0, rel=1e-9) and info["sigma"] == pytest.approx(s0, rel=1e-9)


def test_all_equal_scores_give_no_flags():
    C = np.full(1000, 2.5)
    z, info = oracle.pot_threshold(C)
    assert z == 2.5 and info["n_peaks"] == 0
    assert oracle.flags(C, z).sum() == 0


def test_flags_are_strict():
    assert list(oracle.flags([1.0, 2.0, 3.0, np.nan], 2.0)) == [0, 0, 1, 0]
