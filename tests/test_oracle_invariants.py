"""Whole-score invariants of the oracle (CPU only)."""
import numpy as np
import pytest

import oracle
from paper_2407_09486_amd import workloads as wl


def _run(cfg, w, Wt, **kw):
    return oracle.score(w.values_f64(), w.stream_offsets, window=cfg.window, stride=cfg.stride,
                        weights=Wt.as_f64(), act=cfg.act, **kw)


def test_stride_subsampling():
    """Window k at stride S is window k*S at stride 1 (reference statistics do not depend on S)."""
    base = wl.CONFIGS["c3"].replace(n_streams=3, t_len=257, window=12, hidden=16, metrics=3)
    w = wl.generate(base)
    Wt = wl.make_weights(base, bias_scale=0.2)
    s1, m1 = _run(base.replace(stride=1), w, Wt)
    woff1 = oracle.window_offsets(w.stream_offsets, 12, 1)
    for S in (2, 3, 5):
        sS, mS = _run(base.replace(stride=S), w, Wt)
        woffS = oracle.window_offsets(w.stream_offsets, 12, S)
        for s in range(3):
            a = s1[woff1[s]:woff1[s + 1]][::S]
            assert np.array_equal(sS[woffS[s]:woffS[s + 1]], a)
            assert np.array_equal(mS[woffS[s]:woffS[s + 1]], m1[woff1[s]:woff1[s + 1]][::S])


def test_stream_permutation_and_batch_composition():
    cfg = wl.CONFIGS["c5"].replace(n_streams=6, window=10, hidden=16, metrics=4, t_min=5, t_max=90)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg, bias_scale=0.1)
    sc, md = _run(cfg, w, Wt)
    woff = oracle.window_offsets(w.stream_offsets, 10, 1)
    perm = np.array([4, 0, 5, 2, 1, 3])
    wp = wl.generate(cfg, streams=perm)
    scp, mdp = _run(cfg, wp, Wt)
    woffp = oracle.window_offsets(wp.stream_offsets, 10, 1)
    for i, s in enumerate(perm):
        assert np.array_equal(scp[woffp[i]:woffp[i + 1]], sc[woff[s]:woff[s + 1]])
        alone = wl.generate(cfg, streams=[s])
        sa, ma = _run(cfg, alone, Wt)
        assert np.array_equal(sa, sc[woff[s]:woff[s + 1]])
        assert np.array_equal(ma, md[woff[s]:woff[s + 1]])


def test_relu_homogeneity():
    """ReLU with zero biases: scaling v by c >= 0 scales h, mu and lv by c, so md scales by c and
    the score 1/2 sum(c^2 mu^2 + g(c lv)) with convex g >= 0, g(0) = 0 is non-decreasing in c."""
    cfg = wl.CONFIGS["c2"].replace(n_streams=2, t_len=300, window=16, hidden=24)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg)
    x = w.values_f64()
    mean, std = oracle.ref_stats(x, w.stream_offsets, 0.5)
    prev = None
    md1 = None
    for c in (0.0, 0.25, 0.5, 1.0, 2.0, 4.0):
        sc, md = oracle.score(x, w.stream_offsets, window=16, stride=1, weights=Wt.as_f64(),
                              ref_mean=mean, ref_std=std / c if c > 0 else std * np.inf)
        if c == 0.0:
            assert np.all(sc == 0.0) and np.all(md == 0.0)
        if c == 1.0:
            md1 = md
        if md1 is not None and c > 1.0:
            np.testing.assert_allclose(md, c * md1, rtol=1e-9, atol=1e-12)
        if prev is not None:
            assert np.all(sc >= prev - 1e-12 * np.abs(prev))
        prev = sc


@pytest.mark.parametrize("value", [0.0, 3.0, -1024.5, 0.375])
def test_constant_stream_scores_zero(value):
    """A stream constant at its reference mean normalises to v = 0; with zero biases
    h = act(0) = 0, mu = lv = 0 and the reconstruction m' = 0 = v: score = md = 0 exactly."""
    for act in ("relu", "tanh"):
        cfg = wl.CONFIGS["c1"].replace(window=8, hidden=16, act=act)
        w = wl.constant_streams(cfg, [50, 8, 7], [value, value, value])
        Wt = wl.make_weights(cfg)
        sc, md = _run(cfg, w, Wt)
        assert len(sc) == 43 + 1
        assert np.all(sc == 0.0) and np.all(md == 0.0)


def test_zero_length_and_short_streams_produce_nothing():
    cfg = wl.CONFIGS["c1"].replace(window=8, hidden=8)
    w = wl.generate(cfg.replace(n_streams=4, t_len=0, t_min=0, t_max=0), lengths=[0, 7, 8, 0])
    Wt = wl.make_weights(cfg)
    sc, md = _run(cfg, w, Wt)
    assert len(sc) == 1 and np.isfinite(sc[0])
