"""Shared helpers of the GPU tests: run the library through the C ABI and compare with the oracle."""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle
from paper_2407_09486_amd import binding
from paper_2407_09486_amd import workloads as wl

# Tolerances of the scores (relative + absolute floor) and of md (relative to mean|v| + mean|m'|).
TOL = {"f32": (1e-4, 1e-6), "bf16": (1e-2, 1e-4)}


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def detector(cfg: wl.Config, weights: wl.Weights, kernel="auto"):
    return binding.Detector(cfg.metrics, cfg.window, cfg.stride, cfg.hidden,
                            binding.weights_for_library(weights, cfg.dtype), latent=cfg.latent,
                            dtype=cfg.dtype, act=cfg.act, kernel=kernel, ref_frac=cfg.ref_frac)


def upload(w: wl.Workload, device="cuda"):
    import torch
    if w.cfg.dtype == "bf16":
        x = torch.from_numpy(w.x_bits.view(np.int16)).to(device)
    else:
        x = torch.from_numpy(w.x).to(device)
    so = torch.from_numpy(w.stream_offsets).to(device)
    return x, so


def gpu_score(det, w: wl.Workload, threshold=math.nan, flags=False, ref=None, pad=0):
    """Score a workload on the GPU; returns numpy (scores, md, flags|None, window_offsets).

    With pad > 0 the outputs live inside larger buffers filled with a canary, and the test
    checks that nothing outside [0, N) was written.
    """
    import torch
    x, so = upload(w)
    woff_h = det.window_offsets(w.stream_offsets)
    N = int(woff_h[-1])
    wo = torch.from_numpy(woff_h).cuda()
    canary = -12345.0
    sc_buf = torch.full((N + 2 * pad,), canary, dtype=torch.float32, device="cuda")
    md_buf = torch.full((N + 2 * pad,), canary, dtype=torch.float32, device="cuda")
    fl_buf = torch.full((N + 2 * pad,), 77, dtype=torch.uint8, device="cuda")
    sc = sc_buf[pad:pad + N]
    md = md_buf[pad:pad + N]
    fl = fl_buf[pad:pad + N] if flags else None
    rm = rs = None
    if ref is not None:
        rm = torch.from_numpy(np.ascontiguousarray(ref[0], np.float32)).cuda()
        rs = torch.from_numpy(np.ascontiguousarray(ref[1], np.float32)).cuda()
    binding.enova_detect_score(det.handle, x, so, wo, w.n_streams, N, rm, rs, threshold, sc, md, fl)
    torch.cuda.synchronize()
    if pad:
        for buf, val in ((sc_buf, canary), (md_buf, canary)):
            h = buf.cpu().numpy()
            assert np.all(h[:pad] == val) and np.all(h[pad + N:] == val), "write outside [0, N)"
        if flags:
            h = fl_buf.cpu().numpy()
            assert np.all(h[:pad] == 77) and np.all(h[pad + N:] == 77), "flag write outside [0, N)"
    return (sc.cpu().numpy(), md.cpu().numpy(), fl.cpu().numpy() if flags else None, woff_h)


def oracle_score(cfg: wl.Config, w: wl.Workload, weights: wl.Weights, ref=None, threads=0):
    return oracle.score(w.values_f64(), w.stream_offsets, window=cfg.window, stride=cfg.stride,
                        weights=weights.as_f64(), act=cfg.act, ref_frac=cfg.ref_frac,
                        bf16=cfg.dtype == "bf16",
                        ref_mean=None if ref is None else ref[0], ref_std=None if ref is None else ref[1],
                        threads=threads, return_stats=True)


def check_scores(g, o, dtype, what=""):
    rel, ab = TOL[dtype]
    g = np.asarray(g, np.float64)
    err = np.abs(g - o)
    lim = rel * np.abs(o) + ab
    bad = ~(err <= lim)
    if bad.any():
        i = np.flatnonzero(bad)[:10]
        raise AssertionError(f"{what}: {bad.sum()} of {len(o)} scores out of tolerance; "
                             f"idx {i.tolist()} gpu {g[i].tolist()} oracle {o[i].tolist()}")
    return float(np.max(err / np.maximum(lim, 1e-30))) if len(o) else 0.0


def check_md(g, o, scale, dtype, what=""):
    rel, _ = TOL[dtype]
    g = np.asarray(g, np.float64)
    err = np.abs(g - o)
    lim = rel * scale
    bad = ~(err <= lim)
    if bad.any():
        i = np.flatnonzero(bad)[:10]
        raise AssertionError(f"{what}: {bad.sum()} of {len(o)} md out of tolerance; "
                             f"idx {i.tolist()} gpu {g[i].tolist()} oracle {o[i].tolist()} "
                             f"scale {scale[i].tolist()}")


def check_flags(gf, o_scores, thr_o, thr_g, dtype, what=""):
    """Flags bit-exact except windows whose oracle score lies within tolerance of the threshold."""
    rel, _ = TOL[dtype]
    of = (o_scores > thr_o).astype(np.uint8)
    near = np.abs(o_scores - thr_o) <= rel * abs(thr_o) + abs(thr_g - thr_o)
    bad = (gf != of) & ~near
    assert not bad.any(), f"{what}: {bad.sum()} flags differ away from the threshold"
