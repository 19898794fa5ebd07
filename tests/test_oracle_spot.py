"""Pins of the oracle's streaming peaks-over-threshold (SPOT) against its definition: the start
is the batch POT, alarms never enter the model, normal scores only count, a peak refits the tail
on every stored peak, and the bookkeeping matches a hand-worked example."""
import math

import numpy as np
import pytest

import oracle


def _calib(seed=3, n=4000):
    return np.random.default_rng(seed).gamma(2.0, 1.0, n)


def test_start_is_the_batch_threshold():
    c = _calib()
    sp = oracle.Spot(c, level=0.98, q=1e-3)
    z, info = oracle.pot_threshold(c, level=0.98, q=1e-3)
    assert sp.z == z and sp.t == info["t"] and sp.n == c.size and len(sp.Y) == info["n_peaks"]


def test_alarms_leave_the_model_alone():
    sp = oracle.Spot(_calib())
    state = (sp.t, sp.z, sp.n, list(sp.Y))
    for s in (sp.z * 1.0001 + 1e-9, sp.z + 10.0, 1e30, math.inf):
        assert sp.step(s) == 1
    assert (sp.t, sp.z, sp.n, sp.Y) == state


def test_normal_scores_only_count_and_nan_is_ignored():
    sp = oracle.Spot(_calib())
    z0, n0, y0 = sp.z, sp.n, list(sp.Y)
    for s in np.linspace(-5.0, sp.t, 50):
        assert sp.step(float(s)) == 0
    assert sp.step(float("nan")) == 0
    assert sp.z == z0 and sp.Y == y0 and sp.n == n0 + 50


def test_a_peak_refits_on_all_stored_peaks():
    rng = np.random.default_rng(11)
    c = _calib(5, 3000)
    sp = oracle.Spot(c)
    peaks, n = list(sp.Y), sp.n
    for s in np.concatenate([rng.gamma(2.0, 1.0, 400), [sp.t + 0.5 * (sp.z - sp.t)]]):
        s = float(s)
        alarm = s > sp.z
        assert sp.step(s) == int(alarm)
        if not alarm:
            n += 1
            if s > sp.t:
                peaks.append(s - sp.t)
    assert sp.n == n and sp.Y == peaks
    # the last score was a peak: the threshold is the tail refitted on every stored peak
    z, _ = oracle.pot_fit(sp.t, n, np.array(peaks), 1e-3)
    assert sp.z == z


def test_hand_worked_moments_example():
    # calibration 1..100: t = the 98th order statistic = 98, peaks {1, 2}, n = 100
    sp = oracle.Spot(np.arange(1.0, 101.0), level=0.98, q=1e-3)
    assert sp.t == 98.0 and sorted(sp.Y) == [1.0, 2.0] and sp.n == 100
    # moments: mean 1.5, unbiased variance 0.5 -> gamma = (1 - 4.5)/2, sigma = 1.5 (1 + 4.5)/2
    g, s = -1.75, 4.125
    assert sp.z == pytest.approx(98.0 + s / g * ((1e-3 * 100 / 2) ** (-g) - 1.0), rel=1e-14)
    # a score between t and z_q joins the peaks: {1, 2, 1.5}, n = 101, variance 0.25
    assert sp.step(99.5) == 0
    g, s = 0.5 * (1 - 1.5 ** 2 / 0.25), 0.5 * 1.5 * (1 + 1.5 ** 2 / 0.25)
    assert sp.n == 101 and sp.z == pytest.approx(98.0 + s / g * ((1e-3 * 101 / 3) ** (-g) - 1.0), rel=1e-14)
    assert sp.step(100.0) == 1          # above z_q = 99.875 -> alarm


def test_single_peak_means_every_exceedance_is_an_alarm():
    sp = oracle.Spot(np.arange(1.0, 51.0), level=0.98)   # t = 49, one peak -> z_q = t
    assert sp.z == sp.t == 49.0
    assert sp.step(49.5) == 1 and sp.n == 50 and len(sp.Y) == 1
    assert sp.step(49.0) == 0 and sp.n == 51


def test_empty_calibration_never_flags():
    sp = oracle.Spot([])
    assert sp.z == math.inf and sp.step(1e30) == 0 and sp.n == 0 and sp.Y == []


def test_frozen_at_the_peak_capacity():
    c = _calib(7, 1000)
    sp = oracle.Spot(c, peak_cap=25)
    assert len(sp.Y) == 20
    added = 0
    rng = np.random.default_rng(2)
    while len(sp.Y) < 25:
        s = float(sp.t + rng.uniform(0, 0.5) * (sp.z - sp.t))
        sp.step(s)
        added += 1
    state = (sp.z, sp.n, list(sp.Y))
    assert sp.step(sp.t + 0.1 * (sp.z - sp.t)) == 0 and sp.step(sp.t - 1.0) == 0
    assert (sp.z, sp.n, sp.Y) == state
    assert sp.step(sp.z + 1.0) == 1
