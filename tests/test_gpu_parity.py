"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small sizes are compared window by window; the configs' full sizes are run exactly as the
benchmark launches them and checked on sampled windows (tests/test_gpu_fullsize.py).
"""
import math

import numpy as np
import pytest

import oracle
from harness import (TOL, check_flags, check_md, check_scores, detector, gpu_score, log,
                     oracle_score)
from paper_2407_09486_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _subset(name, n):
    cfg = wl.CONFIGS[name]
    streams = np.random.default_rng(1234).choice(cfg.n_streams, size=min(n, cfg.n_streams), replace=False)
    return cfg, wl.generate(cfg, streams=np.sort(streams))


# (config, streams in the subset): each spans several tiles and ends in a ragged tail.
SUBSETS = [("c1", 1), ("c2", 3), ("c3", 4), ("c4", 2), ("c5", 3)]


@pytest.mark.parametrize("kernel", ["auto", "valu"])
@pytest.mark.parametrize("name,n", SUBSETS)
def test_subset_parity(name, n, kernel):
    cfg, w = _subset(name, n)
    if name == "c5":                      # keep the oracle to seconds: cap the ragged lengths
        w = wl.generate(cfg.replace(t_min=512, t_max=4096), streams=w.streams)
    weights = wl.make_weights(cfg, bias_scale=0.05)
    log(f"[parity] {name} streams={w.streams.tolist()} kernel={kernel}")
    det = detector(cfg, weights, kernel)
    if kernel == "auto" and name != "c1":
        assert det.kernel_kind == "mfma"
    sc, md, _, woff = gpu_score(det, w, pad=64)
    o_sc, o_md, info = oracle_score(cfg, w, weights)
    assert np.array_equal(woff, info["window_offsets"])
    r = check_scores(sc, o_sc, cfg.dtype, f"{name}/{kernel}")
    check_md(md, o_md, info["md_scale"], cfg.dtype, f"{name}/{kernel}")
    log(f"[parity] {name} {kernel}: {len(sc)} windows, max err/tol {r:.3f}")
    det.close()


# Every config, each subset scored as its own batch so the calibration sets match: c4 with four
# full streams (900 calibration windows, an MLE fit), c5 with three streams at their real ragged
# lengths (45554, 9528 and 29047 steps: 84 K windows, many 256-window tiles per stream).
@pytest.mark.parametrize("name,n", [("c1", 1), ("c2", 3), ("c3", 4), ("c4", 4), ("c5", 3)])
def test_threshold_and_flags(name, n):
    cfg, w = _subset(name, n)
    weights = wl.make_weights(cfg)
    log(f"[threshold] {name} streams={w.streams.tolist()} lengths={np.diff(w.stream_offsets).tolist()}")
    det = detector(cfg, weights)
    sc, md, _, woff = gpu_score(det, w)
    o_sc, _, _ = oracle_score(cfg, w, weights)
    check_scores(sc, o_sc, cfg.dtype, f"{name} threshold subset")
    import torch
    scores_t = torch.from_numpy(sc).cuda()
    so_t = torch.from_numpy(w.stream_offsets).cuda()
    wo_t = torch.from_numpy(woff).cuda()
    thr_g, info_g, fl = det.threshold(scores_t, so_t, wo_t, flags=True)
    fl = fl.cpu().numpy()
    # the oracle's threshold on the oracle's scores: within the score tolerance
    cal_o = oracle.calibration_scores(o_sc, w.stream_offsets, window=cfg.window, stride=cfg.stride)
    thr_o, info_o = oracle.pot_threshold(cal_o)
    rel = TOL[cfg.dtype][0]
    assert abs(thr_g - thr_o) <= rel * abs(thr_o) + 1e-6, (thr_g, thr_o, info_g, info_o)
    # the oracle's threshold on the GPU's own scores: same order statistic and fit
    cal_g = oracle.calibration_scores(sc.astype(np.float64), w.stream_offsets, window=cfg.window,
                                      stride=cfg.stride)
    thr_og, info_og = oracle.pot_threshold(cal_g)
    assert info_g["n"] == info_og["n"] and info_g["n_peaks"] == info_og["n_peaks"]
    assert info_g["t"] == info_og["t"]
    assert info_g["method"] == info_og["method"]
    assert abs(thr_g - np.float32(thr_og)) <= 1e-6 * abs(thr_og), (thr_g, thr_og)
    # flags from the threshold call, and from the score call given the threshold
    check_flags(fl, o_sc, thr_o, thr_g, cfg.dtype, name)
    assert np.array_equal(fl, (sc > np.float32(thr_g)).astype(np.uint8))
    sc2, _, fl2, _ = gpu_score(det, w, threshold=thr_g, flags=True)
    assert np.array_equal(fl2, fl) and np.array_equal(sc2, sc)
    log(f"[threshold] {name}: gpu {thr_g:.6g} oracle {thr_o:.6g} ({info_g['method']}, "
        f"N_t={info_g['n_peaks']}), flagged {int(fl.sum())}")
    det.close()


# Scores that no detector produces but the threshold call accepts: negative values (whose float
# keys order in reverse), heavy ties at the level quantile, all-negative sets and calibration
# sets small enough for the method of moments or the bare quantile. The radix select's digits and
# counts must give the oracle's order statistic and peak count exactly.
@pytest.mark.parametrize("case", ["normal", "ties", "negative", "small_moments", "single_peak"])
def test_threshold_on_arbitrary_scores(case):
    import torch
    cfg = wl.CONFIGS["c2"].replace(window=16, stride=2)
    det = detector(cfg, wl.make_weights(cfg))
    lengths = {"small_moments": [500, 300], "single_peak": [260]}.get(case, [3000, 1234, 4100])
    so = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    woff = det.window_offsets(so)
    nw = int(woff[-1])
    rng = np.random.default_rng(20240712)
    if case == "ties":
        sc = np.round(rng.normal(0.0, 1.0, nw), 1)
    elif case == "negative":
        sc = -rng.exponential(2.0, nw)
    else:
        sc = rng.normal(0.0, 1.0, nw)
    sc = sc.astype(np.float32)
    thr_g, info_g, fl = det.threshold(torch.from_numpy(sc).cuda(), torch.from_numpy(so).cuda(),
                                      torch.from_numpy(woff).cuda(), flags=True)
    cal = oracle.calibration_scores(sc.astype(np.float64), so, window=cfg.window, stride=cfg.stride)
    thr_o, info_o = oracle.pot_threshold(cal)
    assert info_g["n"] == info_o["n"] and info_g["n_peaks"] == info_o["n_peaks"], (info_g, info_o)
    assert info_g["t"] == info_o["t"] and info_g["method"] == info_o["method"], (info_g, info_o)
    assert abs(thr_g - np.float32(thr_o)) <= 1e-6 * abs(thr_o) + 1e-30, (thr_g, thr_o)
    assert np.array_equal(fl.cpu().numpy(), (sc > np.float32(thr_g)).astype(np.uint8))
    log(f"[threshold] {case}: n={info_g['n']} N_t={info_g['n_peaks']} method={info_g['method']} "
        f"t={info_g['t']:.6g} z={thr_g:.6g}")
    det.close()


def test_valu_and_mfma_agree_and_are_deterministic():
    cfg, w = _subset("c3", 2)
    weights = wl.make_weights(cfg, bias_scale=0.05)
    dm = detector(cfg, weights, "mfma")
    dv = detector(cfg, weights, "valu")
    a = gpu_score(dm, w)
    b = gpu_score(dm, w)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), "matrix-core run not deterministic"
    v1 = gpu_score(dv, w)
    v2 = gpu_score(dv, w)
    assert np.array_equal(v1[0], v2[0]) and np.array_equal(v1[1], v2[1]), "vector run not deterministic"
    np.testing.assert_allclose(a[0], v1[0], rtol=2e-4, atol=2e-6)


@pytest.mark.parametrize("name", ["c2", "c5"])
def test_batch_composition_is_bitwise(name):
    """A stream's scores are bitwise identical whether scored alone or inside a batch."""
    cfg = wl.CONFIGS[name]
    if name == "c5":
        cfg = cfg.replace(t_min=512, t_max=3000)
    ids = np.array([5, 1, 9, 3, 7])
    wb = wl.generate(cfg, streams=ids)
    weights = wl.make_weights(cfg)
    det = detector(cfg, weights)
    sc, md, _, woff = gpu_score(det, wb)
    for i, s in enumerate(ids):
        wa = wl.generate(cfg, streams=[s])
        sa, ma, _, _ = gpu_score(det, wa)
        assert np.array_equal(sa, sc[woff[i]:woff[i + 1]]), f"stream {s}"
        assert np.array_equal(ma, md[woff[i]:woff[i + 1]]), f"stream {s}"
    det.close()


# ------------------------------------------------------------------ edge shapes and cases
EDGE = [
    # metrics, window, stride, hidden, latent, dtype, act, lengths
    (5, 7, 3, 40, 9, "f32", "relu", [0, 6, 7, 8, 50, 1, 333]),      # odd M, W % S != 0, H not 32k
    (3, 16, 1, 20, 16, "f32", "tanh", [16, 17, 600, 2]),           # M padded to 4, tanh
    (8, 24, 5, 64, 4, "bf16", "relu", [100, 24, 0, 257]),          # bf16, W % S != 0, small L
    (16, 8, 8, 96, 16, "f32", "relu", [1000, 9, 64]),              # S == W
    (4, 4, 9, 33, 16, "f32", "relu", [40, 4, 13]),                 # S > W
    (12, 10, 2, 256, 16, "bf16", "tanh", [300, 55]),               # H at the matrix-core limit
    (2, 3, 1, 300, 20, "f32", "relu", [200, 3]),                   # H and L beyond it: vector kernel
]


@pytest.mark.parametrize("case", range(len(EDGE)))
@pytest.mark.parametrize("kernel", ["auto", "valu"])
def test_edge_shapes(case, kernel):
    M, W, S, H, L, dt, act, lengths = EDGE[case]
    cfg = wl.CONFIGS["c5"].replace(metrics=M, window=W, stride=S, hidden=H, latent=L, dtype=dt,
                                   act=act, n_streams=len(lengths), kind="ragged_mix")
    w = wl.generate(cfg, lengths=lengths)
    weights = wl.make_weights(cfg, bias_scale=0.1)
    log(f"[edge] case {case} {EDGE[case]} kernel={kernel}")
    det = detector(cfg, weights, kernel)
    sc, md, _, woff = gpu_score(det, w, pad=32)
    o_sc, o_md, info = oracle_score(cfg, w, weights)
    assert np.array_equal(woff, info["window_offsets"])
    check_scores(sc, o_sc, dt, f"edge{case}")
    check_md(md, o_md, info["md_scale"], dt, f"edge{case}")
    det.close()


@pytest.mark.parametrize("hidden", [32, 64, 128, 256])
@pytest.mark.parametrize("act", ["relu", "tanh"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_every_matrix_core_layout(dtype, act, hidden):
    """Each wave layout / activation / storage type instantiation of the matrix-core kernel,
    on ragged streams with several tiles, a partial tile and a stream shorter than a window."""
    cfg = wl.CONFIGS["c5"].replace(metrics=8, window=32, stride=2, hidden=hidden, latent=16,
                                   dtype=dtype, act=act, n_streams=4, kind="ragged_mix")
    lengths = [1200, 45, 31, 700]
    w = wl.generate(cfg, lengths=lengths)
    weights = wl.make_weights(cfg, bias_scale=0.1)
    log(f"[layout] {dtype} {act} H={hidden}")
    det = detector(cfg, weights, "mfma")
    sc, md, _, woff = gpu_score(det, w, pad=32)
    o_sc, o_md, info = oracle_score(cfg, w, weights)
    assert np.array_equal(woff, info["window_offsets"])
    check_scores(sc, o_sc, dtype, f"layout-{dtype}-{act}-{hidden}")
    check_md(md, o_md, info["md_scale"], dtype, f"layout-{dtype}-{act}-{hidden}")
    det.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kernel", ["auto", "valu"])
def test_constant_streams_score_exactly_zero(dtype, kernel):
    cfg = wl.CONFIGS["c2"].replace(dtype=dtype, window=16, hidden=64)
    w = wl.constant_streams(cfg, [40, 300, 16], [3.0, -0.5, 1024.0])
    weights = wl.make_weights(cfg)          # zero biases
    det = detector(cfg, weights, kernel)
    sc, md, _, _ = gpu_score(det, w)
    assert len(sc) == 25 + 285 + 1
    assert np.all(sc == 0.0) and np.all(md == 0.0)
    det.close()


def test_external_reference_statistics():
    cfg, w = _subset("c2", 2)
    weights = wl.make_weights(cfg)
    # caller-supplied statistics near the stream's own (far-off ones overflow fp32 scores)
    rng = np.random.default_rng(3)
    o_mean, o_std = oracle.ref_stats(w.values_f64(), w.stream_offsets, cfg.ref_frac)
    mean = (o_mean + 0.3 * o_std * rng.normal(size=o_mean.shape)).astype(np.float32)
    std = (o_std * rng.uniform(0.7, 1.4, size=o_std.shape)).astype(np.float32)
    det = detector(cfg, weights)
    sc, md, _, _ = gpu_score(det, w, ref=(mean, std))
    o_sc, o_md, info = oracle_score(cfg, w, weights, ref=(mean.astype(np.float64), std.astype(np.float64)))
    check_scores(sc, o_sc, "f32", "external stats")
    check_md(md, o_md, info["md_scale"], "f32", "external stats")


def test_reference_statistics_entry_point():
    import torch
    from paper_2407_09486_amd import binding
    for name in ("c2", "c4"):
        cfg, w = _subset(name, 3)
        det = detector(cfg, wl.make_weights(cfg))
        x, so = __import__("harness").upload(w)
        mean = torch.empty((3, cfg.metrics), device="cuda")
        std = torch.empty((3, cfg.metrics), device="cuda")
        binding.enova_detect_ref_stats(det.handle, x, so, 3, mean, std)
        o_mean, o_std = oracle.ref_stats(w.values_f64(), w.stream_offsets, cfg.ref_frac)
        np.testing.assert_allclose(mean.cpu().numpy(), o_mean, rtol=1e-6, atol=1e-6)
        np.testing.assert_allclose(std.cpu().numpy(), o_std, rtol=1e-6)


def test_nan_input_propagates_and_is_not_flagged():
    cfg = wl.CONFIGS["c1"].replace(t_len=400)
    w = wl.generate(cfg)
    w.x[300, 2] = np.nan
    weights = wl.make_weights(cfg)
    for kernel in ("auto", "valu"):
        det = detector(cfg, weights, kernel)
        sc, md, fl, woff = gpu_score(det, w, threshold=1.0, flags=True)
        k = np.arange(len(sc))
        hit = (k <= 300) & (k + cfg.window > 300)
        assert np.all(np.isnan(sc[hit])) and np.all(np.isnan(md[hit]))
        assert np.all(np.isfinite(sc[~hit]))
        assert np.all(fl[hit] == 0)


def test_empty_inputs():
    import torch
    from paper_2407_09486_amd import binding
    cfg = wl.CONFIGS["c2"]
    det = detector(cfg, wl.make_weights(cfg))
    w = wl.generate(cfg.replace(n_streams=3), lengths=[0, 10, 63])     # no window anywhere
    sc, md, _, woff = gpu_score(det, w)
    assert len(sc) == 0 and woff[-1] == 0
    x = torch.zeros((1, cfg.metrics), device="cuda")
    so = torch.zeros(1, dtype=torch.int64, device="cuda")
    binding.enova_detect_score(det.handle, x, so, so, 0, 0, None, None, math.nan, None, None, None)
    with pytest.raises(binding.EnovaError) as e:
        det.threshold(torch.zeros(0, device="cuda"), so, so)
    assert e.value.status == binding.ENOVA_ESHAPE
