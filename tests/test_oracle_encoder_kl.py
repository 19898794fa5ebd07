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


def test_bf16_mode_rounds_normalised_values():
    """bf16 workload: staged v is bf16(fp32(x - mean) * fp32(1/std)); the rest is fp64."""
    cfg = wl.CONFIGS["c4"].replace(n_streams=1, t_len=64, window=8, stride=2, metrics=4, hidden=8)
    w = wl.generate(cfg)
    Wt = wl.make_weights(cfg)
    x = w.values_f64()
    mean = np.array([0.1, -0.3, 2.0, 0.0])
    std = np.array([1.3, 0.7, 3.1, 1.0])
    d = oracle.window_debug(x, 2, window=8, stride=2, weights=Wt.as_f64(), mean=mean, std=std, bf16=True)
    seg = x[4:12].astype(np.float32)
    v32 = (seg - mean.astype(np.float32)) * (np.float32(1.0) / std.astype(np.float32))
    vb = wl.bf16_bits_to_f32(wl.to_bf16_bits(v32.astype(np.float32))).reshape(-1)
    assert np.array_equal(d["v"], vb.astype(np.float64))
