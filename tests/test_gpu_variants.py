"""GPU parity of the detector-output variants (Section IV-B) through the C ABI: KL score, md, the
per-metric md vector and the reconstruction error of every window, for both normalisations,
against the fp64 oracle ``oracle/variants.py``.

Tolerances: the scores as the batch path (1e-4 relative in fp32, 1e-2 for the bf16 detector);
md and every md_m within that fraction of the window's scale mean|v| + mean|m'|; the
reconstruction error within that fraction of (error + scale^2), since it is a mean of squared
differences of quantities of that scale.
"""
import numpy as np
import pytest

from harness import TOL, check_scores, detector, log, upload
from oracle import variants as ov
from paper_2407_09486_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _weights_f64(w):
    return {k: np.asarray(getattr(w, k), np.float64) for k in
            ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")}


def _run(cfg, w, work, norm):
    import torch
    det = detector(cfg, w, "mfma")
    x, so = upload(work)
    woff = det.window_offsets(work.stream_offsets)
    N = int(woff[-1])
    out = det.score_ext(x, so, torch.from_numpy(woff).cuda(), N, norm=norm)
    torch.cuda.synchronize()
    res = [o.cpu().numpy() for o in out]
    det.close()
    return res, woff


def _check(g, ref, dtype, what, idx=None):
    sc, md, mdm, rec = g
    if idx is not None:
        sc, md, mdm, rec = sc[idx], md[idx], mdm[idx], rec[idx]
    rel, _ = TOL[dtype]
    check_scores(sc, ref["score"], dtype, what + " score")
    scale = ref["scale"]
    assert np.all(np.abs(md - ref["md"]) <= rel * scale), what + " md"
    assert np.all(np.abs(mdm - ref["md_metric"]) <= rel * scale[:, None]), what + " md_metric"
    assert np.all(np.abs(rec - ref["recon"]) <= rel * (ref["recon"] + scale ** 2)), what + " recon"


@pytest.mark.parametrize("norm", ["reference", "window"])
@pytest.mark.parametrize("shape", [dict(metrics=8, window=32, stride=1, hidden=32, latent=16, act="relu"),
                                   dict(metrics=5, window=7, stride=3, hidden=40, latent=3, act="tanh"),
                                   # power-of-two M: the decoder-output product reduces in its
                                   # epilogue; D = 28 (one partial column slot), M = 1, M = 32
                                   dict(metrics=4, window=7, stride=2, hidden=40, latent=3, act="tanh"),
                                   dict(metrics=1, window=50, stride=1, hidden=64, latent=8, act="relu",
                                        kind="ar1_spikes"),
                                   dict(metrics=32, window=5, stride=1, hidden=48, latent=16, act="relu"),
                                   # the detector's c5 window shape (M = 16, D = 1024)
                                   dict(metrics=16, window=64, stride=1, hidden=32, latent=16, act="relu"),
                                   # fused single-launch shapes with strides above one: 128 hidden
                                   # units with tanh and 8 metrics; a partial last super-row
                                   # (W = 14, S = 3); 4 metrics (both lane halves on one chunk)
                                   dict(metrics=8, window=16, stride=2, hidden=100, latent=10, act="tanh"),
                                   dict(metrics=16, window=14, stride=3, hidden=64, latent=16, act="relu"),
                                   dict(metrics=4, window=24, stride=3, hidden=128, latent=8, act="relu")])
def test_variants_match_oracle(norm, shape):
    cfg = wl.CONFIGS["c1"].replace(n_streams=5, t_len=0, t_min=20, t_max=900, **{"kind": "ragged_mix", **shape})
    w = wl.make_weights(cfg, bias_scale=0.1)
    work = wl.generate(cfg, lengths=[900, 5, 40, 333, 700])
    log(f"variants {norm} {shape}")
    g, woff = _run(cfg, w, work, norm)
    ref = ov.score_ext(work.values_f64(), work.stream_offsets, window=cfg.window, stride=cfg.stride,
                       weights=_weights_f64(w), act=cfg.act, norm=norm, ref_frac=cfg.ref_frac)
    assert len(ref["score"]) == woff[-1]
    _check(g, ref, "f32", f"{norm} {shape}")


@pytest.mark.parametrize("name,over,fused", [
    ("c5", {}, True),                                            # M = 16, H = 128, ReLU
    ("c2", {}, True),                                            # M = 8, H = 64
    ("c1", dict(metrics=8, window=16, stride=2, hidden=100, latent=10, act="tanh"), True),
    ("c1", dict(metrics=16, window=16, hidden=100, act="tanh"), False),   # tanh, 128 units, 16 metrics
    ("c1", dict(metrics=5, window=32), False),                  # 5 metrics
    ("c3", {}, False),                                           # a 256-window tile exceeds half the LDS
    ("c4", {}, False),                                           # bf16 detector
])
def test_variant_evaluation_mode(name, over, fused):
    """Which shapes take the fused single launch (the rest are evaluated in chunks); both kinds are
    checked against the oracle above."""
    cfg = wl.CONFIGS[name].replace(**over)
    det = detector(cfg, wl.make_weights(cfg), "mfma")
    try:
        assert det.ext_fused() == fused
    finally:
        det.close()


@pytest.mark.parametrize("window", [16, 32])
@pytest.mark.parametrize("norm", ["reference", "window"])
def test_variants_bf16_detector(norm, window):
    cfg = wl.CONFIGS["c4"].replace(n_streams=3, t_len=300, metrics=8, window=window, stride=2, hidden=64)
    w = wl.make_weights(cfg, bias_scale=0.1)
    work = wl.generate(cfg)
    log(f"variants bf16 {norm} W={window}")
    g, woff = _run(cfg, w, work, norm)
    ref = ov.score_ext(work.values_f64(), work.stream_offsets, window=cfg.window, stride=cfg.stride,
                       weights=_weights_f64(w), act=cfg.act, norm=norm, ref_frac=cfg.ref_frac, bf16=True)
    _check(g, ref, "bf16", f"bf16 {norm}")


def test_reference_variants_agree_with_the_batch_path():
    import torch
    cfg = wl.CONFIGS["c2"].replace(n_streams=4, t_len=3000)
    w = wl.make_weights(cfg)
    work = wl.generate(cfg)
    det = detector(cfg, w, "mfma")
    x, so = upload(work)
    woff = det.window_offsets(work.stream_offsets)
    N = int(woff[-1])
    wo = torch.from_numpy(woff).cuda()
    sc, md, _ = det.score(x, so, wo, N)
    sc2, md2, _, _ = det.score_ext(x, so, wo, N)
    torch.cuda.synchronize()
    a, b = sc.cpu().numpy().astype(np.float64), sc2.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(a - b) <= 2e-4 * np.abs(a) + 1e-6)
    det.close()


@pytest.mark.parametrize("hidden,fused", [(32, True), (200, False)])
def test_windows_across_chunks_and_constant_metrics(hidden, fused):
    """More windows than one chunk of the chunked evaluation (2^28 / D = 65536 windows for
    D = 512 x 8; 200 hidden units keep the detector off the fused kernel): windows on both sides
    of every chunk boundary, and a metric that is constant inside some windows (the per-window
    guard), on both evaluations."""
    cfg = wl.CONFIGS["c1"].replace(n_streams=3, t_len=30000, window=512, hidden=hidden)
    w = wl.make_weights(cfg, bias_scale=0.1)
    work = wl.generate(cfg)
    xv = work.x.copy()
    xv[1000:1700, 3] = 2.5                           # constant inside windows 1000..1188 of stream 0
    work = wl.from_arrays(cfg, xv, work.stream_offsets)
    det = detector(cfg, w, "mfma")
    assert det.ext_fused() == fused
    det.close()
    for norm in ("window", "reference"):
        g, woff = _run(cfg, w, work, norm)
        N = int(woff[-1])
        assert N > 65536
        glob = sorted({0, 1000, 1030, 65535, 65536, 65537, N - 1} | set(range(1040, 1060)))
        pairs = []
        for gi in glob:
            s = int(np.searchsorted(woff, gi, side="right") - 1)
            pairs.append((s, gi - int(woff[s])))
        ref = ov.score_ext(work.values_f64(), work.stream_offsets, window=cfg.window, stride=cfg.stride,
                           weights=_weights_f64(w), act=cfg.act, norm=norm, ref_frac=cfg.ref_frac, pairs=pairs)
        _check(g, ref, "f32", f"chunks {norm}", idx=np.asarray(glob))


def test_short_last_chunk_splits_its_products():
    """65536 + 300 windows of D = 512 x 8 (chunks of 65536) on the chunked evaluation (200 hidden
    units): the last chunk's encoder product has few output tiles and splits its reduction; its
    windows must match the oracle like the others."""
    cfg = wl.CONFIGS["c1"].replace(n_streams=1, t_len=65536 + 300 + 511, window=512, hidden=200)
    w = wl.make_weights(cfg, bias_scale=0.1)
    work = wl.generate(cfg)
    det = detector(cfg, w, "mfma")
    assert not det.ext_fused()
    det.close()
    g, woff = _run(cfg, w, work, "window")
    N = int(woff[-1])
    assert N == 65536 + 300
    glob = [0, 65535] + list(range(65536, N, 7)) + [N - 1]
    ref = ov.score_ext(work.values_f64(), work.stream_offsets, window=cfg.window, stride=cfg.stride,
                       weights=_weights_f64(w), act=cfg.act, norm="window", ref_frac=cfg.ref_frac,
                       pairs=[(0, k) for k in glob])
    _check(g, ref, "f32", "short last chunk", idx=np.asarray(glob))


@pytest.mark.parametrize("hidden", [64, 200])
def test_scores_only_skip_the_decoder(hidden):
    """With md, md_m and the error all NULL the decoder is skipped (fused kernel with 64 hidden
    units, chunked evaluation with 200); the scores are the same kernels' output, so they match a
    full call bit for bit. No windows: nothing to do."""
    import torch
    cfg = wl.CONFIGS["c2"].replace(n_streams=3, t_len=2000, hidden=hidden)
    w = wl.make_weights(cfg, bias_scale=0.1)
    work = wl.generate(cfg)
    det = detector(cfg, w, "mfma")
    x, so = upload(work)
    woff = det.window_offsets(work.stream_offsets)
    N = int(woff[-1])
    wo = torch.from_numpy(woff).cuda()
    log("variants scores only")
    full = det.score_ext(x, so, wo, N, norm="window")[0]
    only, md, mdm, rec = det.score_ext(x, so, wo, N, norm="window", scores_only=True)
    assert md is None and mdm is None and rec is None
    empty = det.score_ext(x, so, wo, 0, norm="window")
    torch.cuda.synchronize()
    assert np.array_equal(full.cpu().numpy(), only.cpu().numpy())
    assert all(t.numel() == 0 for t in empty)
    det.close()


def test_variants_full_size_sampled():
    """The benchmarked workload (c5, per-window normalisation, every output) at its real size,
    launched as bench.py launches it (one fused launch); sampled windows (random ones, stream
    edges, tile edges of the chunked evaluation's chunks) against the oracle."""
    import torch
    from test_gpu_fullsize import _sample, _sub_workload
    cfg = wl.CONFIGS["c5"]
    w = wl.make_weights(cfg)
    work = wl.generate(cfg)
    det = detector(cfg, w, "mfma")
    x, so = upload(work)
    woff = det.window_offsets(work.stream_offsets)
    N = int(woff[-1])
    log(f"variants full size: {N} windows")
    sc, md, mdm, rec = det.score_ext(x, so, torch.from_numpy(woff).cuda(), N, norm="window")
    g, s, k = _sample(woff, 128, np.random.default_rng(7), n_random=500, n_streams=20)
    chunk = (1 << 28) // cfg.d                       # windows per chunk of the chunked evaluation
    edges = [e for c in range(chunk, N, chunk) for e in (c - 1, c)]
    g = np.array(sorted(set(g.tolist()) | set(edges)), np.int64)
    s = np.searchsorted(woff, g, side="right") - 1
    k = g - woff[s]
    gi = torch.from_numpy(g).cuda()
    got = [t[gi].cpu().numpy() for t in (sc, md, mdm, rec)]
    streams = np.unique(s)
    xs, offs = _sub_workload(work, streams)
    sub = np.searchsorted(streams, s)
    ref = ov.score_ext(xs, offs, window=cfg.window, stride=cfg.stride, weights=_weights_f64(w), act=cfg.act,
                       norm="window", ref_frac=cfg.ref_frac, pairs=list(zip(sub.tolist(), k.tolist())))
    _check(got, ref, "f32", "variants full size")
    det.close()
