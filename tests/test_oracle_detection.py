"""Detection sanity of the whole oracle (normalise -> VAE -> KL -> POT -> flag), CPU only.

The weights are random (seeded), so the paper's Table IV quality is not reproducible
(its data and trained weights are absent). What is checked: injected events are hit,
point-adjusted (Section VI, RQ2: a detected segment counts if any point in it is an
anomaly), significantly more often than chance.
"""
import math

import numpy as np
from scipy.stats import binomtest

import oracle
from paper_2407_09486_amd import workloads as wl


def _hits(cfg, seed, event_windows):
    c = cfg.replace(data_seed=cfg.data_seed + 1000 * seed, weight_seed=cfg.weight_seed + seed)
    w = wl.generate(c)
    Wt = wl.make_weights(c)
    sc, md = oracle.score(w.values_f64(), w.stream_offsets, window=c.window, stride=c.stride,
                          weights=Wt.as_f64(), act=c.act)
    cal = oracle.calibration_scores(sc, w.stream_offsets, window=c.window, stride=c.stride)
    thr, _ = oracle.pot_threshold(cal)
    fl = oracle.flags(sc, thr)
    return event_windows(c, w, fl, md)


def _spike_windows(c, w, fl, md):
    """(hit events, covering windows per event, false positives, clean test windows)."""
    W, S = c.window, c.stride
    T = int(w.stream_offsets[1])
    lab = np.nonzero(w.labels)[0]
    R = T // 2
    cover = np.zeros(len(fl), bool)
    hits = 0
    for p in lab:
        ks = np.arange(max(0, p - W + 1), min(p, len(fl) - 1) + 1)
        cover[ks] = True
        hits += int(fl[ks].any())
    test_k = np.arange(len(fl)) * S >= R
    clean = test_k & ~cover
    return hits, len(lab), int(fl[clean].sum()), int(clean.sum()), W


def test_spikes_detected_above_chance():
    cfg = wl.CONFIGS["c1"]
    hits = n_ev = fp = n_clean = 0
    for seed in range(32):
        h, n, f, nc, W = _hits(cfg, seed, _spike_windows)
        hits, n_ev, fp, n_clean = hits + h, n_ev + n, fp + f, n_clean + nc
    fp_rate = fp / n_clean
    chance = 1 - (1 - fp_rate) ** W
    res = binomtest(hits, n_ev, chance, alternative="greater")
    assert hits / n_ev > 0.5, (hits, n_ev, fp_rate)
    assert res.pvalue < 1e-6, (hits, n_ev, chance)


def _shift_windows(c, w, fl, md):
    W, S = c.window, c.stride
    T = int(w.stream_offsets[1])
    lab = w.labels[:T].astype(bool)
    # segments of consecutive labelled steps
    edges = np.flatnonzero(np.diff(np.concatenate([[0], lab.astype(int), [0]])))
    segs = list(zip(edges[::2], edges[1::2]))
    cover = np.zeros(len(fl), bool)
    hits = 0
    up = 0
    for a, b in segs:
        ks = np.arange(max(0, a - W + 1), min(b - 1, len(fl) - 1) + 1)
        cover[ks] = True
        hit = fl[ks].any()
        hits += int(hit)
        if hit:
            up += int(md[ks][fl[ks] == 1].mean() > 0)
    test_k = np.arange(len(fl)) * S >= T // 2
    clean = test_k & ~cover
    return hits, len(segs), int(fl[clean].sum()), int(clean.sum()), W, up


def test_level_shifts_detected_and_md_points_up():
    """Load level shifts (+40 req/step) are hit above chance, and the MD of the flagged
    windows is positive (overload -> scale up) for most hits."""
    cfg = wl.CONFIGS["c2"].replace(n_streams=1, t_len=4096)
    hits = n_ev = fp = n_clean = ups = 0
    for seed in range(32):
        h, n, f, nc, W, up = _hits(cfg, seed, _shift_windows)
        hits, n_ev, fp, n_clean, ups = hits + h, n_ev + n, fp + f, n_clean + nc, ups + up
    fp_rate = fp / max(n_clean, 1)
    # a shifted segment is covered by >= 2W windows
    chance = 1 - (1 - fp_rate) ** (2 * W)
    res = binomtest(hits, n_ev, chance, alternative="greater")
    assert res.pvalue < 1e-6, (hits, n_ev, chance)
    assert ups >= 0.8 * hits, (ups, hits)
