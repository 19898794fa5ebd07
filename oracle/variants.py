"""Oracle of the detector-output variants (Section IV-B) -- TEST INFRASTRUCTURE ONLY, fp64.

Section IV-B normalises the metrics before the VAE and reads the anomaly direction from the mean
difference between the window m and its reconstruction m'. The variants computed here, per window:

* the normalisation either against the stream's reference prefix (as the batch path) or against
  the window itself: per metric, the window's own mean and population standard deviation, with
  the reference path's guard (std <= 1e-6 max(1, |mean|) counts as constant and becomes 1) --
  the literal "per-window normalisation" reading;
* the KL score and the scalar mean difference md = mean_j (v_j - m'_j), as the batch path;
* the per-metric mean difference md_m = mean_t (v_{t,m} - m'_{t,m}) (so md = mean_m md_m);
* the reconstruction error mean_j (v_j - m'_j)^2, which needs the decoder's full output
  m' = Wd2 act(Wd1 mu + bd1) + bd2 (z = mu at inference).

Every window goes through the oracle's own window evaluation (``oracle.window_debug``), which
returns v and m'; this module only forms the statistics the variants need from them.
"""
from __future__ import annotations

import numpy as np

from . import ref_stats, window_count, window_debug


def window_stats(xw):
    """Per-metric mean and population std of one window [W, M] (fp64), with the guard."""
    xw = np.asarray(xw, np.float64)
    W, M = xw.shape
    mean = xw.sum(axis=0) / W
    sd = np.sqrt(((xw - mean) ** 2).sum(axis=0) / W)
    sd = np.where(sd <= 1e-6 * np.maximum(1.0, np.abs(mean)), 1.0, sd)
    return mean, sd


def score_ext(x, stream_offsets, *, window, stride, weights, act="relu", norm="reference", ref_frac=0.5,
              bf16=False, ref_mean=None, ref_std=None, pairs=None):
    """Variants of every window (or of the (stream, k) pairs given). Returns dict of arrays:
    score, md, md_metric [., M], recon, and scale = mean|v| + mean|m'| (the magnitude the mean
    differences are measured against); window order = stream order, then window index."""
    x = np.asarray(x, np.float64)
    offs = np.asarray(stream_offsets, np.int64)
    n = len(offs) - 1
    M = x.shape[1]
    W, S = int(window), int(stride)
    if norm == "reference":
        if ref_mean is None:
            rm, rs = ref_stats(x, offs, ref_frac)
        else:
            rm = np.asarray(ref_mean, np.float64).reshape(n, M)
            rs = np.asarray(ref_std, np.float64).reshape(n, M)
    if pairs is None:
        pairs = [(s, k) for s in range(n) for k in range(int(window_count(int(offs[s + 1] - offs[s]), W, S)))]
    out = {"score": [], "md": [], "md_metric": [], "recon": [], "scale": []}
    for s, k in pairs:
        xs = x[offs[s]:offs[s + 1]]
        if norm == "window":
            mean, sd = window_stats(xs[k * S:k * S + W])
        else:
            mean, sd = rm[s], rs[s]
        dbg = window_debug(xs, k, window=W, stride=S, weights=weights, mean=mean, std=sd, act=act, bf16=bf16)
        d = dbg["v"] - dbg["mrec"]
        out["score"].append(dbg["score"])
        out["md"].append(d.mean())
        out["md_metric"].append(d.reshape(W, M).mean(axis=0))
        out["recon"].append((d * d).mean())
        out["scale"].append(np.abs(dbg["v"]).mean() + np.abs(dbg["mrec"]).mean())
    res = {k: np.asarray(v, np.float64) for k, v in out.items()}
    if res["md_metric"].size == 0:
        res["md_metric"] = np.zeros((0, M))
    return res
