"""Pins of the oracle's encoder, KL score and MD against library routines (CPU only)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from torch.distributions import Normal, kl_divergence

import oracle
from paper_2407_09486_amd import workloads as wl


def _lib_window(x_stream, k, cfg, Wt, mean, std, act):
    """The same window computed with torch library layers (float64)."""
    W, S, M = cfg.window, cfg.stride, cfg.metrics
    seg = torch.tensor(x_stream[k * S:k * S + W])                    # [W, M]
    v = ((seg - torch.tensor(mean)) / torch.tensor(std)).reshape(-1)   # row-major: j = t*M + m
    w = {k2: torch.tensor(v2) for k2, v2 in Wt.as_f64().items()}
    actf = torch.relu if act == "relu" else torch.tanh
    h = actf(F.linear(v, w["w1"], w["b1"]))
    mu = F.linear(h, w["wmu"], w["bmu"])
    lv = F.linear(h, w["wlv"], w["blv"])
    kl = kl_divergence(Normal(mu, torch.exp(0.5 * lv)), Normal(torch.zeros_like(mu), torch.ones_like(mu))).sum()
    hd = actf(F.linear(mu, w["wd1"], w["bd1"]))
    mrec = F.linear(hd, w["wd2"], w["bd2"])
    md = (v - mrec).mean()
    return dict(v=v.numpy(), h=h.numpy(), mu=mu.numpy(), lv=lv.numpy(), hd=hd.numpy(),
                mrec=mrec.numpy(), score=float(kl), md=float(md))


@pytest.mark.parametrize("act", ["relu", "tanh"])
def test_window_matches_torch_layers(act):
    cfg = wl.CONFIGS["c1"].replace(n_streams=1, t_len=200, window=12, stride=3, hidden=20, latent=7,
                                   metrics=5, act=act)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg, bias_scale=0.3)
    x = w.values_f64()
    mean, std = oracle.ref_stats(x, w.stream_offsets, cfg.ref_frac)
    for k in (0, 5, 30, 62):
        got = oracle.window_debug(x, k, window=cfg.window, stride=cfg.stride, weights=Wt.as_f64(),
                                  mean=mean[0], std=std[0], act=act)
        exp = _lib_window(x, k, cfg, Wt, mean[0], std[0], act)
        for key in ("v", "h", "mu", "lv", "hd", "mrec"):
            np.testing.assert_allclose(got[key], exp[key], rtol=1e-11, atol=1e-12, err_msg=key)
        assert got["score"] == pytest.approx(exp["score"], rel=1e-11, abs=1e-13)
        assert got["md"] == pytest.approx(exp["md"], rel=1e-10, abs=1e-13)


def test_batch_driver_matches_single_windows_ragged():
    cfg = wl.CONFIGS["c5"].replace(n_streams=5, window=8, hidden=16, metrics=3, t_min=5, t_max=40)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg, bias_scale=0.2)
    x = w.values_f64()
    sc, md, info = oracle.score(x, w.stream_offsets, window=8, stride=1, weights=Wt.as_f64(),
                                return_stats=True)
    woff = info["window_offsets"]
    for s in range(w.n_streams):
        xs = x[w.stream_offsets[s]:w.stream_offsets[s + 1]]
        for k in range(int(woff[s + 1] - woff[s])):
            d = oracle.window_debug(xs, k, window=8, stride=1, weights=Wt.as_f64(),
                                    mean=info["mean"][s], std=info["std"][s])
            assert sc[woff[s] + k] == d["score"] and md[woff[s] + k] == d["md"]


def test_kl_zero_posterior_is_exactly_zero():
    """mu = 0 and log-variance 0 make the posterior the prior: KL = 0 exactly."""
    cfg = wl.CONFIGS["c1"].replace(window=4, hidden=6, latent=3, metrics=2)
    Wt = wl.make_weights(cfg)
    for k in ("wmu", "wlv"):
        getattr(Wt, k)[:] = 0.0
    x = np.random.default_rng(0).normal(size=(10, 2))
    d = oracle.window_debug(x, 0, window=4, stride=1, weights=Wt.as_f64(), mean=np.zeros(2), std=np.ones(2))
    assert d["score"] == 0.0


def test_kl_monte_carlo():
    """E_q[log q(z) - log p(z)] estimated from 10^6 samples agrees within 4 standard errors."""
    cfg = wl.CONFIGS["c1"].replace(window=6, hidden=10, latent=4, metrics=3)
    Wt = wl.make_weights(cfg, bias_scale=0.5)
    x = np.random.default_rng(1).normal(size=(20, 3)) * 2
    d = oracle.window_debug(x, 2, window=6, stride=1, weights=Wt.as_f64(), mean=np.zeros(3), std=np.ones(3))
    mu, lv = d["mu"], d["lv"]
    sd = np.exp(0.5 * lv)
    rng = np.random.default_rng(2)
    z = mu + sd * rng.standard_normal((1_000_000, len(mu)))
    logq = -0.5 * (((z - mu) / sd) ** 2).sum(1) - np.log(sd).sum() - 0.5 * len(mu) * math.log(2 * math.pi)
    logp = -0.5 * (z ** 2).sum(1) - 0.5 * len(mu) * math.log(2 * math.pi)
    r = logq - logp
    se = r.std() / math.sqrt(len(r))
    assert abs(r.mean() - d["score"]) < 4 * se


def test_kl_lower_bound_and_nonnegative():
    """KL = 1/2 sum(mu^2 + e^lv - 1 - lv) >= 1/2 |mu|^2 >= 0 since e^u - 1 - u >= 0."""
    cfg = wl.CONFIGS["c3"].replace(n_streams=4, t_len=300, window=16, hidden=32, metrics=4)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg, bias_scale=0.5)
    x = w.values_f64()
    mean, std = oracle.ref_stats(x, w.stream_offsets, 0.5)
    for s in range(4):
        xs = x[w.stream_offsets[s]:w.stream_offsets[s + 1]]
        for k in (0, 17, 60):
            d = oracle.window_debug(xs, k, window=16, stride=4, weights=Wt.as_f64(), mean=mean[s], std=std[s])
            assert d["score"] >= 0.5 * float(d["mu"] @ d["mu"]) - 1e-12 >= -1e-12


def test_md_column_sum_identity():
    """mean(m') = (1^T Wd2 hd + sum(bd2)) / D: the decoder's mean needs only column sums of Wd2."""
    cfg = wl.CONFIGS["c2"].replace(window=10, hidden=12, metrics=4, latent=5)
    Wt = wl.make_weights(cfg, bias_scale=0.4)
    x = np.random.default_rng(5).normal(size=(40, 4))
    d = oracle.window_debug(x, 3, window=10, stride=1, weights=Wt.as_f64(), mean=np.zeros(4), std=np.ones(4))
    w = Wt.as_f64()
    u = w["wd2"].sum(axis=0)
    mean_rec = (u @ d["hd"] + w["bd2"].sum()) / w["wd2"].shape[0]
    assert d["md"] == pytest.approx(d["v"].mean() - mean_rec, rel=1e-12, abs=1e-14)


def _bf16_table():
    """Every non-negative bfloat16 value in bit-pattern order (patterns 0 .. 0x7f80). The last
    entry, pattern 0x7f80 (+inf), stands at 2^128: IEEE rounding overflows to infinity exactly
    where the nearest value of an unbounded exponent range would be 2^128."""
    bits = np.arange(0, 0x7f81, dtype=np.uint32) << 16
    tab = bits.view(np.float32).astype(np.float64)
    tab[-1] = 2.0 ** 128
    return tab


def _nearest_bf16(d):
    """Brute force: the nearest entry of the full bfloat16 table, ties to the even bit pattern."""
    tab = _bf16_table()
    d = np.asarray(d, np.float64)
    a = np.abs(d)
    hi = np.searchsorted(tab, a, side="left")           # tab[hi-1] < a <= tab[hi]
    hi = np.clip(hi, 1, len(tab) - 1)
    lo = hi - 1
    dlo, dhi = a - tab[lo], tab[hi] - a
    pick = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo % 2 == 0, lo, hi)))
    r = np.where(a == 0, 0.0, tab[pick])
    r = np.where((r == 2.0 ** 128) | (a >= 2.0 ** 128), np.inf, r)
    return np.copysign(r, d)


def _bf16_probe_values():
    rng = np.random.default_rng(11)
    tab = _bf16_table()[:-1]                            # finite values only
    mag = np.exp2(rng.uniform(-140, 129, 20000))
    i = rng.integers(0, len(tab) - 1, 4000)
    mids = 0.5 * (tab[i] + tab[i + 1])                   # exact ties
    near = np.concatenate([mids * (1 + 2.0 ** -40), mids * (1 - 2.0 ** -40)])  # off-tie by less than fp32 resolves
    special = np.array([0.0, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135, 2.0 ** -126, tab[-1],
                        0.5 * (tab[-1] + 2.0 ** 128), 0.5 * (tab[-1] + 2.0 ** 128) * (1 - 2.0 ** -30)])
    v = np.concatenate([mag, mids, near, special])
    sign = np.where(rng.random(len(v)) < 0.5, -1.0, 1.0)
    return v * sign


def test_bf16_round_is_the_nearest_bf16_value():
    """The oracle's fp64 -> bfloat16 rounding is the nearest representable value, ties to even,
    including values that a detour through fp32 would round to a tie (1 +- 2^-40 off a midpoint)."""
    v = _bf16_probe_values()
    got = oracle.bf16_round(v)
    exp = _nearest_bf16(v)
    bad = ~((got == exp) | (np.isinf(got) & np.isinf(exp) & (np.sign(got) == np.sign(exp))))
    assert not bad.any(), (v[bad][:5], got[bad][:5], exp[bad][:5])


def test_bf16_round_matches_torch_on_fp32_values():
    """On fp32-representable inputs one rounding from fp64 equals torch's float32 -> bfloat16
    conversion (round to nearest even)."""
    rng = np.random.default_rng(12)
    v = (rng.standard_normal(50000) * np.exp2(rng.integers(-30, 30, 50000))).astype(np.float32)
    exp = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(oracle.bf16_round(v.astype(np.float64)), exp)


def test_bf16_mode_rounds_normalised_values():
    """bf16 workload: the staged v is (x - mean) / std evaluated in fp64, then rounded once to
    the nearest bfloat16; the rest of the window stays fp64."""
    cfg = wl.CONFIGS["c4"].replace(n_streams=1, t_len=64, window=8, stride=2, metrics=4, hidden=8)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg)
    x = w.values_f64()
    mean = np.array([0.1, -0.3, 2.0, 0.0])
    std = np.array([1.3, 0.7, 3.1, 1.0])
    d = oracle.window_debug(x, 2, window=8, stride=2, weights=Wt.as_f64(), mean=mean, std=std, bf16=True)
    v = ((x[4:12] - mean) / std).reshape(-1)
    assert np.array_equal(d["v"], _nearest_bf16(v))
    d32 = oracle.window_debug(x, 2, window=8, stride=2, weights=Wt.as_f64(), mean=mean, std=std)
    assert np.array_equal(d32["v"], v)
    # the encoder runs on the rounded values in fp64
    w1 = Wt.as_f64()
    a = w1["w1"] @ d["v"] + w1["b1"]
    np.testing.assert_allclose(d["h"], np.maximum(a, 0.0), rtol=1e-12, atol=1e-14)
