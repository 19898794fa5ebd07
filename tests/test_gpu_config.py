"""GPU parity of the configuration scans (Section IV-A, Eqs. (4)-(6)) through the C ABI: every
window's OLS fits and t-test, and each stream's KDE limits and configuration, against the fp64
oracle ``oracle/config_scan.py`` on the same seeded series.

Tolerances. Both sides compute in fp64; the per-window outputs are stored as fp32, so they are
compared at 2e-7 relative to the magnitude of the reference (plus the same fraction of the
series' scale for values that cross zero). The t-test decision is exact except where |t| lies
within 1e-7 of the critical value (the two sides' critical values differ by ~1e-10). The
per-stream outputs (fp64 on both sides, different summation orders inside a bisection) agree to
1e-9 relative.
"""
import math

import numpy as np
import pytest

from harness import log
from oracle import config_scan as cs
from paper_2407_09486_amd import binding
from paper_2407_09486_amd import workloads as wl

pytestmark = pytest.mark.gpu

COLS = dict(col_f=0, col_r=1, col_t=4, col_m=5)


def _scanner(W, S, dtype="f32", alpha=0.05, q_extreme=0.99):
    return binding.ConfigScanner(len(wl.CONFIG_METRICS), W, S, col_finished=0, col_running=1, col_exec_time=4,
                                 col_mem_util=5, dtype=dtype, alpha=alpha, q_extreme=q_extreme)


def _upload(x, dtype):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(wl.to_bf16_bits(x).view(np.int16)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()


def _series(lengths, seed):
    # stream i takes the saturating (odd) or the unsaturated (even) kind of service by its parity
    parts = [wl.config_series(2, T, seed=seed + i).x[(i % 2) * T:(i % 2 + 1) * T] for i, T in enumerate(lengths)]
    x = np.concatenate(parts) if parts else np.zeros((0, 7), np.float32)
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    return x, offs


def _check_scan(gpu, ref, tc, what):
    a, b, t, sig, g0, g1 = (v.cpu().numpy() for v in gpu)
    for name, got, exp in (("a", a, ref["a"]), ("b", b, ref["b"]), ("g0", g0, ref["g0"]), ("g1", g1, ref["g1"])):
        scale = float(np.abs(exp).mean()) if exp.size else 0.0
        err = np.abs(got.astype(np.float64) - exp)
        assert np.all(err <= 2e-7 * (np.abs(exp) + scale) + 1e-30), (what, name, float(err.max()))
    fin = np.isfinite(ref["t"])
    assert np.array_equal(np.isinf(t), ~fin), what
    assert np.array_equal(np.sign(t[~fin]), np.sign(ref["t"][~fin])), what
    err = np.abs(t[fin].astype(np.float64) - ref["t"][fin])
    assert np.all(err <= 2e-7 * (np.abs(ref["t"][fin]) + 1.0)), (what, "t", float(err.max()) if err.size else 0)
    near = np.abs(np.abs(ref["t"]) - tc) <= 1e-7 * tc
    assert np.array_equal(sig[~near], ref["sig"][~near]), what


def _run_scan(x, offs, W, S, dtype="f32", alpha=0.05):
    import torch
    sc = _scanner(W, S, dtype, alpha)
    woff = sc.window_offsets(offs)
    n = int(woff[-1])
    xd = _upload(x, dtype)
    out = sc.scan(xd, torch.from_numpy(offs).cuda(), torch.from_numpy(woff).cuda(), n)
    torch.cuda.synchronize()
    sc.close()
    return out, woff


@pytest.mark.parametrize("W,S,lengths", [(64, 1, [700, 63, 64, 300, 0, 1000]),
                                         (17, 3, [400, 16, 17, 21, 950]),
                                         (3, 1, [50, 3, 2]),
                                         (600, 7, [2000, 1300])])
def test_window_scan_matches_oracle(W, S, lengths):
    log(f"config scan W={W} S={S} lengths={lengths}")
    x, offs = _series(lengths, seed=W + S)
    out, woff = _run_scan(x, offs, W, S)
    xr = x.astype(np.float64)
    ref = cs.window_scan(xr, offs, window=W, stride=S, col_f=0, col_r=1, col_m=5)
    assert len(ref["b"]) == woff[-1]
    _check_scan(out, ref, cs.t_critical(0.05, W - 2), f"W={W} S={S}")


def test_window_scan_degenerate_windows():
    """A stretch of constant n^r (no relation: b = 0, t = 0) and a stretch where n^f and m^u are
    exact lines in n^r (|t| = inf, significant)."""
    x, offs = _series([400], seed=3)
    x[100:200, 1] = 42.0
    x[250:350, 0] = 2.0 + 0.25 * x[250:350, 1]
    x[250:350, 5] = 0.125 + 0.0078125 * x[250:350, 1]
    W = 32
    out, woff = _run_scan(x, offs, W, 1)
    ref = cs.window_scan(x.astype(np.float64), offs, window=W, stride=1, col_f=0, col_r=1, col_m=5)
    _check_scan(out, ref, cs.t_critical(0.05, W - 2), "degenerate")
    b, t, sig = out[1].cpu().numpy(), out[2].cpu().numpy(), out[3].cpu().numpy()
    assert np.all(b[100:169] == 0.0) and np.all(t[100:169] == 0.0) and np.all(sig[100:169] == 0)
    assert np.all(np.isinf(t[250:319])) and np.all(sig[250:319] == 1)


def test_window_scan_bf16_input():
    x, offs = _series([500, 300], seed=11)
    xb = wl.bf16_bits_to_f32(wl.to_bf16_bits(x)).reshape(x.shape)
    out, woff = _run_scan(x, offs, 48, 2, dtype="bf16")
    ref = cs.window_scan(xb.astype(np.float64), offs, window=48, stride=2, col_f=0, col_r=1, col_m=5)
    _check_scan(out, ref, cs.t_critical(0.05, 46), "bf16")


@pytest.mark.parametrize("W,S,alpha,q", [(64, 1, 0.05, 0.99), (600, 7, 0.01, 0.95), (5, 2, 0.2, 0.9)])
def test_recommend_matches_oracle(W, S, alpha, q):
    import torch
    lengths = [1500, 900, W - 1, 4000, 2000, 1200]
    x, offs = _series(lengths, seed=100 + W)
    log(f"config recommend W={W} S={S} alpha={alpha} q={q}")
    sc = _scanner(W, S, alpha=alpha, q_extreme=q)
    sig, nl, tl, mns, gm = (v.cpu().numpy() for v in sc.recommend(_upload(x, "f32"), torch.from_numpy(offs).cuda()))
    sc.close()
    ref = cs.stream_config(x.astype(np.float64), offs, window=W, stride=S, alpha=alpha, q_extreme=q, **COLS)
    assert np.array_equal(sig, ref["sig"])
    for got, exp in ((nl, ref["n_limit"]), (tl, ref["t_limit"]), (mns, ref["max_num_seqs"]), (gm, ref["gpu_memory"])):
        assert np.array_equal(np.isnan(got), np.isnan(exp))
        ok = ~np.isnan(exp)
        np.testing.assert_allclose(got[ok], exp[ok], rtol=1e-9, atol=0)
    # both regimes occur among these streams' last windows
    valid = ~np.isnan(ref["n_limit"])
    assert 0 < int(sig[valid].sum()) < int(valid.sum())


def test_recommend_constant_window_is_a_point_mass():
    import torch
    x, offs = _series([300], seed=7)
    x[-64:, 0] = 17.0
    x[-64:, 4] = 2.5
    sc = _scanner(64, 1)
    sig, nl, tl, mns, gm = (v.cpu().numpy() for v in sc.recommend(_upload(x, "f32"), torch.from_numpy(offs).cuda()))
    sc.close()
    assert nl[0] == 17.0 and tl[0] == 2.5 and mns[0] == 42.5


def test_full_size_sampled():
    """The benchmark workload (1024 services x 16384 one-minute steps x 7 metrics, W = 64, S = 1):
    sampled windows and streams against the oracle's functions."""
    import torch
    w = wl.config_series(1024, 16384, seed=20240712)
    x = w.x
    offs = w.stream_offsets
    W = 64
    out, woff = _run_scan(x, offs, W, 1)
    a, b, t, sig, g0, g1 = (v.cpu().numpy() for v in out)
    tc = cs.t_critical(0.05, W - 2)
    rng = np.random.default_rng(0)
    for _ in range(400):
        s = int(rng.integers(0, 1024))
        k = int(rng.integers(0, woff[s + 1] - woff[s]))
        win = x[offs[s] + k:offs[s] + k + W].astype(np.float64)
        f = cs.ols(win[:, 1], win[:, 0])
        g = cs.ols(win[:, 1], win[:, 5])
        i = woff[s] + k
        for got, exp in ((a[i], f["a"]), (b[i], f["b"]), (t[i], f["t"]), (g0[i], g["a"]), (g1[i], g["b"])):
            assert abs(got - exp) <= 2e-7 * (abs(exp) + 1.0), (s, k)
        if abs(abs(f["t"]) - tc) > 1e-7 * tc:
            assert sig[i] == (abs(f["t"]) > tc), (s, k)
    sc = _scanner(W, 1)
    rs = [v.cpu().numpy() for v in sc.recommend(_upload(x, "f32"), torch.from_numpy(offs).cuda())]
    sc.close()
    pick = rng.choice(1024, 24, replace=False)
    sub = np.concatenate([x[offs[s]:offs[s + 1]] for s in pick]).astype(np.float64)
    ref = cs.stream_config(sub, np.arange(25) * 16384, window=W, stride=1, **COLS)
    assert np.array_equal(rs[0][pick], ref["sig"])
    for got, key in zip(rs[1:], ("n_limit", "t_limit", "max_num_seqs", "gpu_memory")):
        np.testing.assert_allclose(got[pick], ref[key], rtol=1e-9, atol=0)


def test_recommend_longest_window():
    """W = 4096 (the largest window the per-service kernel holds): more than the default dynamic
    LDS, a non-trivial sort and KDE over 4096 values."""
    import torch
    W = 4096
    x, offs = _series([5000, 4500, 4096, 4095], seed=77)
    log(f"config recommend W={W}")
    sc = _scanner(W, 3)
    sig, nl, tl, mns, gm = (v.cpu().numpy() for v in sc.recommend(_upload(x, "f32"), torch.from_numpy(offs).cuda()))
    sc.close()
    ref = cs.stream_config(x.astype(np.float64), offs, window=W, stride=3, **COLS)
    assert np.array_equal(sig, ref["sig"])
    for got, exp in ((nl, ref["n_limit"]), (tl, ref["t_limit"]), (mns, ref["max_num_seqs"]), (gm, ref["gpu_memory"])):
        assert np.array_equal(np.isnan(got), np.isnan(exp))
        ok = ~np.isnan(exp)
        np.testing.assert_allclose(got[ok], exp[ok], rtol=1e-9, atol=0)
