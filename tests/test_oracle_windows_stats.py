"""Pins of the oracle's window enumeration and reference statistics (CPU only)."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2407_09486_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_windows(T, W, S):
    """Every start k with the whole window [k*S, k*S+W) inside [0, T)."""
    out = []
    k = 0
    while k * S + W <= T:
        out.append(k)
        k += 1
    return out


@pytest.mark.parametrize("W,S", [(1, 1), (3, 1), (4, 2), (5, 3), (2, 5), (7, 7), (8, 3)])
def test_window_count_matches_brute_force(W, S):
    for T in list(range(0, 40)) + [W - 1, W, W + 1, 3 * W + S]:
        if T < 0:
            continue
        assert oracle.window_count(T, W, S) == len(brute_windows(T, W, S)), (T, W, S)


def test_window_offsets_ragged_tiny():
    T = np.array([0, 3, 4, 5, 9, 1, 12])
    offs = np.concatenate([[0], np.cumsum(T)])
    W, S = 4, 2
    woff = oracle.window_offsets(offs, W, S)
    expect = np.concatenate([[0], np.cumsum([len(brute_windows(t, W, S)) for t in T])])
    assert np.array_equal(woff, expect)


def test_points_accounting_stride_one():
    """At stride 1 a stream of T >= W points yields one score per point after the first W-1.

    The golden fixture records the paper's test-set size (Section VI): 1440 points a
    day for 14 days over 8 LLMs x 2 replicas. A test stream that keeps W-1 points of
    history therefore yields exactly that many windows.
    """
    g = json.load(open(os.path.join(GOLDEN, "points_accounting.json")))
    per_stream = g["points_per_day"] * g["test_days"]
    n_inst = g["llms"] * g["replicas"]
    assert per_stream * n_inst == g["test_points"]
    W = 64
    T = np.full(n_inst, per_stream + W - 1)
    offs = np.concatenate([[0], np.cumsum(T)])
    assert oracle.window_offsets(offs, W, 1)[-1] == g["test_points"]


def test_ref_len_and_calibration_count():
    T = np.array([0, 1, 63, 64, 127, 128, 1000, 16384])
    R = oracle.ref_len(T, 0.5)
    assert np.array_equal(R, T // 2)
    c = oracle.calibration_count(T, 64, 1, 0.5)
    assert np.array_equal(c, [len(brute_windows(r, 64, 1)) for r in T // 2])


def test_ref_stats_match_numpy_population_std():
    rng = np.random.default_rng(3)
    T = np.array([7, 1, 2, 40, 0, 5])
    offs = np.concatenate([[0], np.cumsum(T)])
    x = rng.normal(3.0, 2.0, size=(offs[-1], 3)) * rng.uniform(0.1, 10, size=3)
    mean, std = oracle.ref_stats(x, offs, 0.5)
    for s in range(len(T)):
        R = int(T[s]) // 2
        seg = x[offs[s]:offs[s] + R]
        if R == 0:
            assert np.array_equal(mean[s], np.zeros(3)) and np.array_equal(std[s], np.ones(3))
            continue
        np.testing.assert_allclose(mean[s], seg.mean(axis=0), rtol=1e-13, atol=1e-13)
        sd = seg.std(axis=0, ddof=0)
        sd = np.where(sd <= 1e-6 * np.maximum(1.0, np.abs(seg.mean(axis=0))), 1.0, sd)
        np.testing.assert_allclose(std[s], sd, rtol=1e-12)


def test_ref_stats_constant_guard():
    x = np.full((10, 2), 1000.0)
    x[:, 1] = -2.5
    mean, std = oracle.ref_stats(x, np.array([0, 10]), 0.5)
    assert np.array_equal(mean[0], [1000.0, -2.5])
    assert np.array_equal(std[0], [1.0, 1.0])


def _score(cfg, w, W, **kw):
    return oracle.score(w.values_f64(), w.stream_offsets, window=cfg.window, stride=cfg.stride,
                        weights=W.as_f64(), act=cfg.act, **kw)


def test_affine_invariance_of_scores():
    """x -> a*x + b per (stream, metric), a > 0, leaves the normalised windows unchanged."""
    cfg = wl.CONFIGS["c1"].replace(n_streams=3, t_len=300, window=16, hidden=24)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg, bias_scale=0.1)
    s0, m0 = _score(cfg, w, Wt)
    rng = np.random.default_rng(9)
    x = w.values_f64().copy()
    for s in range(w.n_streams):
        a0, a1 = w.stream_offsets[s], w.stream_offsets[s + 1]
        x[a0:a1] = x[a0:a1] * rng.uniform(0.01, 100.0, cfg.metrics) + rng.uniform(-1e3, 1e3, cfg.metrics)
    s1, m1 = oracle.score(x, w.stream_offsets, window=cfg.window, stride=cfg.stride, weights=Wt.as_f64())
    np.testing.assert_allclose(s1, s0, rtol=1e-8, atol=1e-10)
    np.testing.assert_allclose(m1, m0, rtol=1e-8, atol=1e-10)
