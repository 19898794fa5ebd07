"""Oracle of one semi-supervised ELBO training step (Section IV-B, Eq. (9)) -- TEST
INFRASTRUCTURE ONLY, plain fp64 numpy.

The VAE of Section IV-B (one hidden layer of width H, a diagonal-Gaussian posterior with mean
and log-variance heads of width L, prior N(0, I), a decoder with one hidden layer) is trained on
labelled windows by maximising

    L = 1/B sum_i [ l_i * E_q log p(m_i | z)  -  (1 + l_i)/2 * beta(k) * KL(q(z | m_i) || p(z)) ]

with l_i = +1 for a normal window and -1 for an anomalous one, so the KL term acts on normal
windows only and the reconstruction term pushes anomalies away. Readings taken here (the
paper fixes none of them): one reparameterised sample z = mu + exp(lv/2) * eps with eps given;
a unit-variance Gaussian decoder, log p(m|z) = -1/2 |v - m'|^2 - D/2 log(2 pi); beta(k) from a
PI controller on the batch KL of the normal windows (ControlVAE form: e = KL_set - KL,
P = Kp / (1 + exp(e)), I <- I - Ki e, beta = clamp(P + I + beta_min, beta_min, beta_max));
Adam on the loss J = -L. Gradients are derived by hand below and pinned in
``tests/test_oracle_elbo.py`` against finite differences and torch autograd.

Read literally, L is unbounded above in the anomalous windows' term: -log p grows without
limit as the decoder drifts away from them (the posterior variance of those windows inflates and
the loss diverges within tens of Adam steps, even with a few anomalies per thousand windows).
An optional ``margin`` m bounds that term: an anomalous window contributes
min(e_i, m) + D/2 log(2 pi) with e_i = 1/2 |v_i - m'_i|^2, so it is pushed away only until its
reconstruction error reaches m; m = inf is the equation as printed.
"""
from __future__ import annotations

import math

import numpy as np

PARAMS = ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")


def _act(a, act):
    return np.maximum(a, 0.0) if act == "relu" else np.tanh(a)


def _dact(a, act):
    """Derivative of the activation at the pre-activation a (ReLU: 0 at a <= 0)."""
    if act == "relu":
        return (a > 0.0).astype(np.float64)
    t = np.tanh(a)
    return 1.0 - t * t


def forward(p, V, eps, act="relu"):
    """Every intermediate of the forward pass of a batch V [B, D] (fp64)."""
    f = {}
    f["a1"] = V @ p["w1"].T + p["b1"]
    f["h"] = _act(f["a1"], act)
    f["mu"] = f["h"] @ p["wmu"].T + p["bmu"]
    f["lv"] = f["h"] @ p["wlv"].T + p["blv"]
    f["sd"] = np.exp(0.5 * f["lv"])
    f["z"] = f["mu"] + f["sd"] * eps
    f["a2"] = f["z"] @ p["wd1"].T + p["bd1"]
    f["hd"] = _act(f["a2"], act)
    f["mr"] = f["hd"] @ p["wd2"].T + p["bd2"]
    D = V.shape[1]
    f["err"] = 0.5 * np.sum((V - f["mr"]) ** 2, axis=1)
    f["logp"] = -f["err"] - 0.5 * D * math.log(2.0 * math.pi)
    f["kl"] = 0.5 * np.sum(f["mu"] ** 2 + np.exp(f["lv"]) - 1.0 - f["lv"], axis=1)
    return f


def _logp_eff(f, l, margin):
    """log p of every window, with an anomalous window's -log p capped at margin + D/2 log 2 pi."""
    const = f["logp"] + f["err"]                       # -D/2 log(2 pi)
    return np.where(l < 0, -np.minimum(f["err"], margin) + const, f["logp"])


def objective(p, V, labels, eps, beta, act="relu", margin=math.inf):
    """L of Eq. (9) for a given beta (the quantity the training maximises)."""
    f = forward(p, V, eps, act)
    l = np.asarray(labels, np.float64)
    return float(np.mean(l * _logp_eff(f, l, margin) - 0.5 * (1.0 + l) * beta * f["kl"]))


def gradients(p, V, labels, eps, beta, act="relu", f=None, margin=math.inf):
    """Gradients of J = -L with respect to every parameter (hand-derived backward pass)."""
    if f is None:
        f = forward(p, V, eps, act)
    B = V.shape[0]
    l = np.asarray(labels, np.float64)[:, None]
    g = {}
    # reconstruction: dJ/dm' = l/B (m' - v), for an anomalous window only below the margin
    active = ((l[:, 0] > 0) | (f["err"] < margin))[:, None]
    g_mr = np.where(active, l / B * (f["mr"] - V), 0.0)
    g["wd2"] = g_mr.T @ f["hd"]
    g["bd2"] = g_mr.sum(axis=0)
    g_a2 = (g_mr @ p["wd2"]) * _dact(f["a2"], act)
    g["wd1"] = g_a2.T @ f["z"]
    g["bd1"] = g_a2.sum(axis=0)
    g_z = g_a2 @ p["wd1"]
    # KL acts on normal windows: dJ/dmu += c mu, dJ/dlv += c (e^lv - 1)/2, c = (1+l)/2 beta/B
    c = 0.5 * (1.0 + l) * beta / B
    g_mu = g_z + c * f["mu"]
    g_lv = g_z * eps * 0.5 * f["sd"] + c * 0.5 * (np.exp(f["lv"]) - 1.0)
    g["wmu"] = g_mu.T @ f["h"]
    g["bmu"] = g_mu.sum(axis=0)
    g["wlv"] = g_lv.T @ f["h"]
    g["blv"] = g_lv.sum(axis=0)
    g_a1 = (g_mu @ p["wmu"] + g_lv @ p["wlv"]) * _dact(f["a1"], act)
    g["w1"] = g_a1.T @ V
    g["b1"] = g_a1.sum(axis=0)
    return g


def pi_beta(kl, state, kl_set, kp, ki, beta_min, beta_max):
    """PI controller of the KL weight: returns (beta, new integral state)."""
    e = kl_set - kl
    integ = state - ki * e
    p_term = kp / (1.0 + math.exp(e)) if e < 700 else 0.0
    beta = min(max(p_term + integ + beta_min, beta_min), beta_max)
    return beta, integ


def adam(p, g, m, v, k, lr, b1=0.9, b2=0.999, eps=1e-8):
    """One Adam step (k >= 1 is the step number) on every parameter; returns new (p, m, v)."""
    np_, nm, nv = {}, {}, {}
    for name in PARAMS:
        nm[name] = b1 * m[name] + (1.0 - b1) * g[name]
        nv[name] = b2 * v[name] + (1.0 - b2) * g[name] ** 2
        mh = nm[name] / (1.0 - b1 ** k)
        vh = nv[name] / (1.0 - b2 ** k)
        np_[name] = p[name] - lr * mh / (np.sqrt(vh) + eps)
    return np_, nm, nv


def train_step(p, m, v, k, integ, V, labels, eps, *, act="relu", lr=1e-3, kl_set=3.0, kp=0.01,
               ki=1e-4, beta_min=0.0, beta_max=1.0, margin=math.inf):
    """Step k (>= 1): forward, beta(k) from the batch KL of the normal windows, backward, Adam.
    Returns (p, m, v, integ, info) with info = loss J, mean log p, mean KL, beta."""
    f = forward(p, V, eps, act)
    l = np.asarray(labels, np.float64)
    normal = l > 0
    kl_batch = float(f["kl"][normal].mean()) if normal.any() else 0.0
    beta, integ = pi_beta(kl_batch, integ, kl_set, kp, ki, beta_min, beta_max)
    g = gradients(p, V, labels, eps, beta, act, f, margin)
    J = -float(np.mean(l * _logp_eff(f, l, margin) - 0.5 * (1.0 + l) * beta * f["kl"]))
    p, m, v = adam(p, g, m, v, k, lr)
    return p, m, v, integ, {"loss": J, "logp": float(f["logp"].mean()), "kl": kl_batch, "beta": beta}
