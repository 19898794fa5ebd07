"""Pins of the oracle's ELBO training step (Eq. (9)): hand-derived gradients against central
finite differences and against torch autograd (fp64), Adam against torch.optim.Adam, the PI
controller's closed-form cases, and the label semantics of the objective."""
import math

import numpy as np
import pytest

from oracle import elbo


def _problem(seed=0, B=12, D=10, H=7, L=3):
    rng = np.random.default_rng(seed)
    p = {"w1": rng.normal(0, 0.4, (H, D)), "b1": rng.normal(0, 0.1, H),
         "wmu": rng.normal(0, 0.4, (L, H)), "bmu": rng.normal(0, 0.1, L),
         "wlv": rng.normal(0, 0.3, (L, H)), "blv": rng.normal(0, 0.1, L),
         "wd1": rng.normal(0, 0.4, (H, L)), "bd1": rng.normal(0, 0.1, H),
         "wd2": rng.normal(0, 0.4, (D, H)), "bd2": rng.normal(0, 0.1, D)}
    V = rng.normal(0, 1, (B, D))
    labels = np.where(rng.random(B) < 0.75, 1.0, -1.0)
    eps = rng.normal(0, 1, (B, L))
    return p, V, labels, eps


def test_gradients_match_finite_differences():
    p, V, labels, eps = _problem(1)
    beta = 0.7
    g = elbo.gradients(p, V, labels, eps, beta, "tanh")
    rng = np.random.default_rng(5)
    h = 1e-6
    for name in elbo.PARAMS:
        for _ in range(4):
            idx = tuple(rng.integers(0, s) for s in p[name].shape)
            q1 = {k: v.copy() for k, v in p.items()}
            q2 = {k: v.copy() for k, v in p.items()}
            q1[name][idx] += h
            q2[name][idx] -= h
            fd = -(elbo.objective(q1, V, labels, eps, beta, "tanh") -
                   elbo.objective(q2, V, labels, eps, beta, "tanh")) / (2 * h)
            assert g[name][idx] == pytest.approx(fd, rel=1e-5, abs=1e-8), (name, idx)


@pytest.mark.parametrize("act", ["relu", "tanh"])
def test_gradients_match_torch_autograd(act):
    torch = pytest.importorskip("torch")
    p, V, labels, eps = _problem(2)
    beta = 0.4
    g = elbo.gradients(p, V, labels, eps, beta, act)
    tp = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
    Vt, lt, et = (torch.tensor(a, dtype=torch.float64) for a in (V, labels, eps))
    A = torch.relu if act == "relu" else torch.tanh
    h = A(Vt @ tp["w1"].T + tp["b1"])
    mu = h @ tp["wmu"].T + tp["bmu"]
    lv = h @ tp["wlv"].T + tp["blv"]
    z = mu + torch.exp(0.5 * lv) * et
    mr = A(z @ tp["wd1"].T + tp["bd1"]) @ tp["wd2"].T + tp["bd2"]
    logp = -0.5 * ((Vt - mr) ** 2).sum(1) - 0.5 * V.shape[1] * math.log(2 * math.pi)
    kl = 0.5 * (mu ** 2 + torch.exp(lv) - 1 - lv).sum(1)
    J = -(lt * logp - 0.5 * (1 + lt) * beta * kl).mean()
    J.backward()
    for name in elbo.PARAMS:
        np.testing.assert_allclose(g[name], tp[name].grad.numpy(), rtol=1e-10, atol=1e-12)


def test_adam_matches_torch():
    torch = pytest.importorskip("torch")
    p, V, labels, eps = _problem(3)
    m = {k: np.zeros_like(v) for k, v in p.items()}
    v = {k: np.zeros_like(x) for k, x in p.items()}
    tp = [torch.tensor(p[k], dtype=torch.float64, requires_grad=True) for k in elbo.PARAMS]
    opt = torch.optim.Adam(tp, lr=1e-2, betas=(0.9, 0.999), eps=1e-8)
    for k in (1, 2, 3):
        g = elbo.gradients(p, V, labels, eps, 0.5, "relu")
        p, m, v = elbo.adam(p, g, m, v, k, 1e-2)
        for t, name in zip(tp, elbo.PARAMS):
            t.grad = torch.tensor(g[name])
        opt.step()
        for t, name in zip(tp, elbo.PARAMS):
            np.testing.assert_allclose(p[name], t.detach().numpy(), rtol=1e-12, atol=1e-14)
        # torch stepped on the oracle's gradients at the oracle's parameters: keep them equal
        for t, name in zip(tp, elbo.PARAMS):
            t.data = torch.tensor(p[name])


def test_pi_controller_cases():
    # at the set point the error is 0: P = Kp/2 and the integral does not move
    b, i = elbo.pi_beta(3.0, 0.2, 3.0, kp=0.01, ki=1e-3, beta_min=0.0, beta_max=1.0)
    assert i == 0.2 and b == pytest.approx(0.005 + 0.2)
    # KL above the set point raises the weight, below lowers it; both clamped
    b_hi, i_hi = elbo.pi_beta(5.0, 0.2, 3.0, 0.01, 1e-3, 0.0, 1.0)
    b_lo, i_lo = elbo.pi_beta(1.0, 0.2, 3.0, 0.01, 1e-3, 0.0, 1.0)
    assert i_hi > 0.2 > i_lo and b_hi > b > b_lo
    assert elbo.pi_beta(1e9, 10.0, 3.0, 0.01, 1e-3, 0.0, 1.0)[0] == 1.0
    assert elbo.pi_beta(-1e3, -10.0, 3.0, 0.01, 1e-3, 0.0, 1.0)[0] == 0.0


def test_labels_gate_the_kl_term_and_flip_the_reconstruction():
    p, V, _, eps = _problem(4)
    B = V.shape[0]
    anomal = -np.ones(B)
    f = elbo.forward(p, V, eps, "relu")
    # all anomalous: L = -mean log p, whatever beta is
    for beta in (0.0, 0.5, 3.0):
        assert elbo.objective(p, V, anomal, eps, beta, "relu") == pytest.approx(-f["logp"].mean())
    # all normal, eps = 0: z = mu and L = mean(log p) - beta mean(KL) with the closed-form KL
    z0 = np.zeros_like(eps)
    f0 = elbo.forward(p, V, z0, "relu")
    kl = 0.5 * np.sum(f0["mu"] ** 2 + np.exp(f0["lv"]) - 1 - f0["lv"], axis=1)
    assert elbo.objective(p, V, np.ones(B), z0, 0.8, "relu") == pytest.approx(f0["logp"].mean() - 0.8 * kl.mean())


def test_training_lowers_the_loss_on_normal_windows():
    rng = np.random.default_rng(9)
    p, _, _, _ = _problem(6, B=64, D=8, H=16, L=2)
    base = rng.normal(0, 1, (8, 2))
    V = rng.normal(0, 1, (64, 2)) @ base.T + 0.05 * rng.normal(0, 1, (64, 8))   # rank-2 data
    labels = np.ones(64)
    m = {k: np.zeros_like(v) for k, v in p.items()}
    v = {k: np.zeros_like(x) for k, x in p.items()}
    integ = 0.0
    recon = []                      # 1/2 |v - m'|^2: -log p without its constant
    for k in range(1, 301):
        eps = rng.normal(0, 1, (64, 2))
        p, m, v, integ, info = elbo.train_step(p, m, v, k, integ, V, labels, eps, act="tanh", lr=1e-2)
        recon.append(-info["logp"] - 4.0 * math.log(2 * math.pi))
    assert np.mean(recon[-20:]) < 0.5 * np.mean(recon[:20])


def _margin_between(err, labels):
    """A margin half-way between two neighbouring anomalous reconstruction errors."""
    e = np.sort(err[labels < 0])
    i = len(e) // 2
    return 0.5 * (e[i - 1] + e[i])


def test_margin_gradients_match_finite_differences():
    p, V, labels, eps = _problem(7, B=16)
    labels[:6] = -1.0
    f = elbo.forward(p, V, eps, "tanh")
    margin = _margin_between(f["err"], labels)
    beta = 0.3
    g = elbo.gradients(p, V, labels, eps, beta, "tanh", margin=margin)
    rng = np.random.default_rng(8)
    h = 1e-6
    for name in elbo.PARAMS:
        for _ in range(4):
            idx = tuple(rng.integers(0, s) for s in p[name].shape)
            q1 = {k: v.copy() for k, v in p.items()}
            q2 = {k: v.copy() for k, v in p.items()}
            q1[name][idx] += h
            q2[name][idx] -= h
            fd = -(elbo.objective(q1, V, labels, eps, beta, "tanh", margin) -
                   elbo.objective(q2, V, labels, eps, beta, "tanh", margin)) / (2 * h)
            assert g[name][idx] == pytest.approx(fd, rel=1e-5, abs=1e-8), (name, idx)


def test_margin_matches_torch_clamp_and_infinite_margin_is_the_literal_objective():
    torch = pytest.importorskip("torch")
    p, V, labels, eps = _problem(10, B=20)
    labels[::3] = -1.0
    f = elbo.forward(p, V, eps, "relu")
    margin = _margin_between(f["err"], labels)
    g = elbo.gradients(p, V, labels, eps, 0.6, "relu", margin=margin)
    tp = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
    Vt, lt, et = (torch.tensor(a, dtype=torch.float64) for a in (V, labels, eps))
    h = torch.relu(Vt @ tp["w1"].T + tp["b1"])
    mu = h @ tp["wmu"].T + tp["bmu"]
    lv = h @ tp["wlv"].T + tp["blv"]
    z = mu + torch.exp(0.5 * lv) * et
    mr = torch.relu(z @ tp["wd1"].T + tp["bd1"]) @ tp["wd2"].T + tp["bd2"]
    err = 0.5 * ((Vt - mr) ** 2).sum(1)
    c = 0.5 * V.shape[1] * math.log(2 * math.pi)
    kl = 0.5 * (mu ** 2 + torch.exp(lv) - 1 - lv).sum(1)
    term = torch.where(lt > 0, -err - c, torch.clamp(err, max=margin) + c)
    J = -(term - 0.5 * (1 + lt) * 0.6 * kl).mean()
    J.backward()
    for name in elbo.PARAMS:
        np.testing.assert_allclose(g[name], tp[name].grad.numpy(), rtol=1e-10, atol=1e-12)
    # margin = inf is Eq. (9) as printed
    g_inf = elbo.gradients(p, V, labels, eps, 0.6, "relu", margin=math.inf)
    g_lit = elbo.gradients(p, V, labels, eps, 0.6, "relu")
    for name in elbo.PARAMS:
        assert np.array_equal(g_inf[name], g_lit[name])
    assert elbo.objective(p, V, labels, eps, 0.6, "relu", math.inf) == elbo.objective(p, V, labels, eps, 0.6, "relu")


def test_margin_keeps_training_bounded_where_the_literal_objective_diverges():
    """With anomalies in the batch the printed objective has no lower bound on J: Adam inflates
    the anomalies' posterior variance and J runs away; a margin stops the push at e_i = margin."""
    p0, V, labels, _ = _problem(11, B=64, D=12, H=16, L=3)
    labels[:] = 1.0
    labels[:6] = -1.0
    rng = np.random.default_rng(12)
    eps = rng.normal(0, 1, (64, 3))
    D = V.shape[1]
    out = {}
    for margin in (math.inf, 2.0 * D):
        p = {k: v.copy() for k, v in p0.items()}
        m = {k: np.zeros_like(v) for k, v in p.items()}
        v = {k: np.zeros_like(x) for k, x in p.items()}
        integ = 0.0
        losses = []
        with np.errstate(over="ignore", invalid="ignore"):
            for k in range(1, 101):
                p, m, v, integ, info = elbo.train_step(p, m, v, k, integ, V, labels, eps, act="relu",
                                                       lr=1e-2, margin=margin)
                losses.append(info["loss"])
        out[margin] = losses
    c = 0.5 * D * math.log(2 * math.pi)
    assert out[math.inf][-1] < -1e6
    # every anomalous term is at most margin + c, and the normal terms are >= 0 in J
    bounded = out[2.0 * D]
    assert min(bounded) >= -(6 / 64) * (2.0 * D + c) - 1e-9
    assert bounded[-1] < 0.5 * bounded[0]
