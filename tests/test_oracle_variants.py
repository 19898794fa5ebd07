"""Pins of the detector-output variants oracle: the reference-normalised variants reproduce the
batch oracle's score and md; per-window normalisation is blind to per-window affine changes of a
metric (and the reference normalisation is not); closed forms of the standardised window
(mean 0, variance 1 per metric) for a decoder whose output is a constant; zero error when the
decoder reproduces the window; the md identity md = mean_m md_m."""
import numpy as np
import pytest

import oracle
from oracle import variants as ov
from paper_2407_09486_amd import workloads as wl


def _setup(seed=0, M=3, W=6, H=5, L=2, lengths=(40, 25)):
    cfg = wl.CONFIGS["c1"].replace(metrics=M, window=W, hidden=H, latent=L)
    w = wl.make_weights(cfg, seed=seed, bias_scale=0.2)
    weights = {k: np.asarray(getattr(w, k), np.float64) for k in
               ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")}
    rng = np.random.default_rng(seed)
    x = rng.normal(0, 1, (sum(lengths), M)) * rng.uniform(0.5, 3, M) + rng.uniform(-5, 5, M)
    offs = np.concatenate([[0], np.cumsum(lengths)])
    return cfg, weights, x, offs


def test_reference_variants_match_the_batch_oracle():
    cfg, wts, x, offs = _setup()
    r = ov.score_ext(x, offs, window=cfg.window, stride=2, weights=wts, act="tanh")
    sc, md = oracle.score(x, offs, window=cfg.window, stride=2, weights=wts, act="tanh")
    np.testing.assert_allclose(r["score"], sc, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(r["md"], md, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(r["md_metric"].mean(axis=1), r["md"], rtol=1e-12, atol=1e-14)
    assert np.all(r["recon"] >= 0.0)


def test_window_normalisation_ignores_per_window_affine_changes():
    cfg, wts, x, offs = _setup(1, lengths=(60,))
    W = cfg.window
    y = x.copy()
    y[30:, 1] = 4.0 * y[30:, 1] + 100.0        # a level and scale change from step 30 on
    a = ov.score_ext(x, offs, window=W, stride=1, weights=wts, norm="window")
    b = ov.score_ext(y, offs, window=W, stride=1, weights=wts, norm="window")
    after = slice(30, 60 - W + 1)              # windows wholly after the change
    for key in ("score", "md", "recon"):
        np.testing.assert_allclose(b[key][after], a[key][after], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(b["md_metric"][after], a["md_metric"][after], rtol=1e-9, atol=1e-12)
    ra = ov.score_ext(x, offs, window=W, stride=1, weights=wts)
    rb = ov.score_ext(y, offs, window=W, stride=1, weights=wts)
    assert np.max(np.abs(rb["score"][after] - ra["score"][after])) > 1e-3


def test_standardised_window_closed_forms():
    """Wd2 = 0 and bd2 = gamma: m' = gamma everywhere. Each metric of a per-window standardised
    window has mean 0 and mean square 1, so md_m = -gamma and the error is 1 + gamma^2."""
    cfg, wts, x, offs = _setup(2, lengths=(50,))
    gamma = 0.75
    w2 = dict(wts, wd2=np.zeros_like(wts["wd2"]), bd2=np.full(cfg.d, gamma))
    r = ov.score_ext(x, offs, window=cfg.window, stride=3, weights=w2, norm="window")
    np.testing.assert_allclose(r["md_metric"], -gamma, atol=1e-12)
    np.testing.assert_allclose(r["recon"], 1.0 + gamma * gamma, rtol=1e-12)
    # a constant metric is guarded to std 1 and normalises to 0 there: its md_m is -gamma and
    # it contributes gamma^2 instead of 1 + gamma^2
    xc = x.copy()
    xc[:, 2] = 7.0
    r = ov.score_ext(xc, offs, window=cfg.window, stride=3, weights=w2, norm="window")
    np.testing.assert_allclose(r["md_metric"][:, 2], -gamma, atol=1e-12)
    np.testing.assert_allclose(r["recon"], (2 * (1 + gamma ** 2) + gamma ** 2) / 3, rtol=1e-12)


def test_exact_reconstruction_has_zero_error():
    cfg, wts, x, offs = _setup(3, lengths=(30,))
    W, M = cfg.window, cfg.metrics
    k = 4
    mean, sd = oracle.ref_stats(x, offs, 0.5)
    v = ((x[k:k + W] - mean[0]) / sd[0]).reshape(-1)
    w2 = dict(wts, wd2=np.zeros_like(wts["wd2"]), bd2=v)
    r = ov.score_ext(x, offs, window=W, stride=1, weights=w2, pairs=[(0, k)])
    assert abs(r["recon"][0]) < 1e-24 and abs(r["md"][0]) < 1e-12
    np.testing.assert_allclose(r["md_metric"][0], 0.0, atol=1e-12)
