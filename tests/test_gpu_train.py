"""GPU parity of the training step (Eq. (9)) through the C ABI: the step's summary (J, mean log p,
mean KL of the normal windows, beta), the gradients of J and the Adam update against the fp64
oracle of ``oracle/elbo.py`` on the same seeded batch.

Tolerances. The device computes in fp32 with sums of at most a few thousand terms per GEMM
element, so every gradient array is compared in the max norm with a relative bound of 1e-4 of
its largest entry (fp32 unit round-off 6e-8 times the reduction length, with margin).
ReLU's derivative is a decision taken on a pre-activation: where the fp64 pre-activation lies
within the fp32 rounding of zero the two sides may decide differently, so the ReLU cases check
that the seeded batch keeps every pre-activation away from zero (margin 1e-5) before comparing;
at the full training size a batch drawn at random cannot keep all 2 M pre-activations clear, so
the random batch's ReLU case compares the gradients at 2e-2 and a second full-size ReLU batch,
filtered by the oracle's forward pass to windows whose pre-activations are all clear of zero,
is compared at the tight tolerances.
The first Adam step moves each parameter by lr * g / (|g| + eps), i.e. by about lr times the sign
of its gradient: where |g| is far above the gradient tolerance the sign is fixed and the updated
parameters must match to fp32 rounding; elsewhere the move must stay within lr.
"""
import math

import numpy as np
import pytest

from harness import log
from oracle import elbo
from paper_2407_09486_amd import binding
from paper_2407_09486_amd import workloads as wl

pytestmark = pytest.mark.gpu

HYPER = dict(lr=1e-3, kl_set=3.0, kp=0.01, ki=1e-4, beta_min=0.0, beta_max=1.0)
GRAD_RTOL = 1e-4


def _cfg(metrics, window, hidden, latent, act):
    return wl.CONFIGS["c1"].replace(metrics=metrics, window=window, hidden=hidden, latent=latent, act=act)


def _init(cfg, seed=11):
    w = wl.make_weights(cfg, seed=seed, bias_scale=0.1)
    return {k: np.asarray(getattr(w, k), np.float32) for k in elbo.PARAMS}


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def _trainer(cfg, p0, margin=math.inf):
    return binding.Trainer(cfg.d, cfg.hidden, cfg.latent, p0, act=cfg.act, margin=margin, **HYPER)


def _oracle_state(p0):
    p = {k: v.astype(np.float64) for k, v in p0.items()}
    m = {k: np.zeros_like(v) for k, v in p.items()}
    v = {k: np.zeros_like(x) for k, x in p.items()}
    return p, m, v


def _relu_margin(p, batch, act):
    """Smallest |pre-activation| of the oracle's forward pass (inf for tanh)."""
    if act != "relu":
        return np.inf
    f = elbo.forward(p, batch.V.astype(np.float64), batch.eps.astype(np.float64), act)
    return float(min(np.abs(f["a1"]).min(), np.abs(f["a2"]).min()))


def _check_grads(g_gpu, g_ref, rtol, what):
    for k in elbo.PARAMS:
        ref = g_ref[k]
        scale = float(np.abs(ref).max())
        err = float(np.abs(g_gpu[k].astype(np.float64) - ref).max())
        assert err <= rtol * scale + 1e-12, f"{what}: gradient {k}: max err {err:.3e} vs scale {scale:.3e}"


def _check_info(info, ref, rtol, what):
    for i, key in enumerate(("loss", "logp", "kl", "beta")):
        assert abs(info[i] - ref[key]) <= rtol * max(1.0, abs(ref[key])), (what, key, info[i], ref[key])


def _clear_batch(cfg, B, seed, delta):
    """B seeded windows whose oracle pre-activations (encoder and decoder hidden layers) all lie
    more than delta from ReLU's kink: candidates are drawn batch by batch from consecutive seeds
    and filtered by the oracle's own fp64 forward pass at the initial parameters."""
    p = {k: v.astype(np.float64) for k, v in _init(cfg).items()}
    parts, s, n = [], seed, 0
    while n < B:
        b = wl.training_batch(cfg, B, seed=s)
        f = elbo.forward(p, b.V.astype(np.float64), b.eps.astype(np.float64), "relu")
        ok = (np.abs(f["a1"]).min(axis=1) > delta) & (np.abs(f["a2"]).min(axis=1) > delta)
        parts.append((b.V[ok], b.labels[ok], b.eps[ok]))
        n += int(ok.sum())
        s += 1
    V, lab, eps = (np.concatenate([q[i] for q in parts])[:B] for i in range(3))
    return wl.TrainBatch(V=np.ascontiguousarray(V), labels=np.ascontiguousarray(lab), eps=np.ascontiguousarray(eps))


def _one_step(cfg, B, seed, anomaly_frac=0.1, labels=None, margin=math.inf, batch=None):
    import torch
    p0 = _init(cfg)
    if batch is None:
        batch = wl.training_batch(cfg, B, seed=seed, anomaly_frac=anomaly_frac)
    if labels is not None:
        batch.labels[:] = labels
    log(f"train step D={cfg.d} H={cfg.hidden} L={cfg.latent} B={B} act={cfg.act} seed={seed} margin={margin}")
    tr = _trainer(cfg, p0, margin)
    info = torch.zeros(4, dtype=torch.float32, device="cuda")
    tr.step(_dev(batch.V), _dev(batch.labels), _dev(batch.eps), info)
    g_gpu, p_gpu = tr.grads(), tr.params()
    info_h = info.cpu().numpy().astype(np.float64)
    tr.close()
    p, m, v = _oracle_state(p0)
    V, lab, eps = (batch.V.astype(np.float64), batch.labels.astype(np.float64), batch.eps.astype(np.float64))
    f = elbo.forward(p, V, eps, cfg.act)
    normal = lab > 0
    kl_b = float(f["kl"][normal].mean()) if normal.any() else 0.0
    beta, _ = elbo.pi_beta(kl_b, 0.0, HYPER["kl_set"], HYPER["kp"], HYPER["ki"], HYPER["beta_min"],
                           HYPER["beta_max"])
    g_ref = elbo.gradients(p, V, lab, eps, beta, cfg.act, f, margin)
    p1, _, _, _, ref_info = elbo.train_step(p, m, v, 1, 0.0, V, lab, eps, act=cfg.act, margin=margin, **HYPER)
    return dict(p0=p0, batch=batch, info=info_h, g_gpu=g_gpu, p_gpu=p_gpu, g_ref=g_ref, p1=p1,
                ref_info=ref_info, margin=_relu_margin(p, batch, cfg.act), err=f["err"], labels=lab)


def _check_adam_first_step(r, lr, what):
    for k in elbo.PARAMS:
        g = r["g_ref"][k]
        fixed = np.abs(g) > 20 * GRAD_RTOL * np.abs(g).max()
        d = np.abs(r["p_gpu"][k].astype(np.float64) - r["p1"][k])
        assert float(d[fixed].max(initial=0.0)) <= 2e-7 * (1 + np.abs(r["p1"][k][fixed]).max(initial=0.0)), (what, k)
        move = np.abs(r["p_gpu"][k].astype(np.float64) - r["p0"][k].astype(np.float64))
        assert float(move.max()) <= lr * 1.001 + 1e-7, (what, k)


@pytest.mark.parametrize("act,seed", [("relu", 2), ("tanh", 4)])
def test_step_matches_oracle_ragged_tiles(act, seed):
    """D = 102, H = 70, L = 16, B = 133: every product has a ragged tile in each dimension."""
    cfg = _cfg(6, 17, 70, 16, act)
    r = _one_step(cfg, 133, seed)
    assert r["margin"] > 1e-5, "seeded batch too close to a ReLU kink for a tight comparison"
    _check_info(r["info"], r["ref_info"], 1e-5, act)
    _check_grads(r["g_gpu"], r["g_ref"], GRAD_RTOL, act)
    _check_adam_first_step(r, HYPER["lr"], act)


def test_step_matches_oracle_whole_tiles():
    """D = 32 x 16 = 512, H = 128, L = 16, B = 512: every large product is a whole number of the
    register-streamed kernel's tiles (the encoder and dJ/da1-type products with the reduction
    split over the waves, the decoder output with the columns split, the weight gradients with
    both operands row-contiguous and the reduction split over blocks as well)."""
    cfg = _cfg(16, 32, 128, 16, "tanh")
    r = _one_step(cfg, 512, 6)
    _check_info(r["info"], r["ref_info"], 1e-5, "whole tiles")
    _check_grads(r["g_gpu"], r["g_ref"], GRAD_RTOL, "whole tiles")
    _check_adam_first_step(r, HYPER["lr"], "whole tiles")


@pytest.mark.parametrize("what,B,frac,labels", [("one window", 1, 0.0, None),
                                                ("all anomalous", 40, 0.0, -1.0),
                                                ("all normal", 40, 0.0, 1.0)])
def test_step_degenerate_batches(what, B, frac, labels):
    cfg = _cfg(4, 8, 33, 3, "tanh")
    r = _one_step(cfg, B, 9, anomaly_frac=frac, labels=labels)
    _check_info(r["info"], r["ref_info"], 1e-5, what)
    _check_grads(r["g_gpu"], r["g_ref"], GRAD_RTOL, what)
    if labels == -1.0:
        # no normal window: the KL term and its controller input vanish
        assert r["info"][2] == 0.0
    _check_adam_first_step(r, HYPER["lr"], what)


def test_anomaly_margin_step():
    """A finite margin between the anomalous windows' reconstruction errors: those above it get
    no gradient. The margin sits half-way between two neighbouring errors, far from both."""
    cfg = _cfg(6, 17, 70, 16, "tanh")
    probe = _one_step(cfg, 133, 4)
    e = np.sort(probe["err"][probe["labels"] < 0])
    i = int(np.argmax(np.diff(e)[: len(e) - 1]))
    margin = float(0.5 * (e[i] + e[i + 1]))
    assert e[i + 1] - e[i] > 1e-3 * margin
    r = _one_step(cfg, 133, 4, margin=margin)
    assert 0 < np.sum(r["err"][r["labels"] < 0] >= margin) < np.sum(r["labels"] < 0)
    _check_info(r["info"], r["ref_info"], 1e-5, "margin")
    _check_grads(r["g_gpu"], r["g_ref"], GRAD_RTOL, "margin")
    _check_adam_first_step(r, HYPER["lr"], "margin")


def test_long_reduction_is_split_and_exact():
    """B = 3000 windows: the weight gradients reduce over the batch in several slices."""
    cfg = _cfg(8, 32, 64, 16, "tanh")
    r = _one_step(cfg, 3000, 21)
    _check_info(r["info"], r["ref_info"], 1e-5, "split")
    _check_grads(r["g_gpu"], r["g_ref"], GRAD_RTOL, "split")


@pytest.mark.parametrize("act", ["tanh", "relu"])
def test_full_training_size(act):
    """The training workload: D = 64 x 16 = 1024, H = 128, L = 16, B = 8192 windows."""
    cfg = _cfg(16, 64, 128, 16, act)
    r = _one_step(cfg, 8192, 5)
    _check_info(r["info"], r["ref_info"], 1e-5 if act == "tanh" else 1e-4, act)
    _check_grads(r["g_gpu"], r["g_ref"], GRAD_RTOL if act == "tanh" else 2e-2, act)


def test_full_training_size_relu_clear_of_the_kink():
    """ReLU at the full training size with the tight tolerances: 8192 windows whose every
    pre-activation is more than 1e-3 from zero (well above the fp32 rounding of a 1024-term
    pre-activation, ~1e-4), so both sides take every derivative decision alike; the summary,
    every gradient array and the first Adam step then match as closely as with tanh."""
    cfg = _cfg(16, 64, 128, 16, "relu")
    batch = _clear_batch(cfg, 8192, 500, 1e-3)
    r = _one_step(cfg, 8192, 0, batch=batch)
    assert r["margin"] > 1e-3
    _check_info(r["info"], r["ref_info"], 1e-5, "relu clear")
    _check_grads(r["g_gpu"], r["g_ref"], GRAD_RTOL, "relu clear")
    _check_adam_first_step(r, HYPER["lr"], "relu clear")


@pytest.mark.parametrize("margin", [math.inf, 102.0])
def test_several_steps_follow_the_oracle(margin):
    """Five steps on fresh batches: the summary of every step (including the controller's beta)
    tracks the oracle, and the parameters stay close to the oracle's trajectory."""
    import torch
    cfg = _cfg(6, 17, 70, 16, "tanh")
    p0 = _init(cfg)
    tr = _trainer(cfg, p0, margin)
    p, m, v = _oracle_state(p0)
    integ = 0.0
    info = torch.zeros(4, dtype=torch.float32, device="cuda")
    lr = HYPER["lr"]
    for k in range(1, 6):
        b = wl.training_batch(cfg, 96, seed=100 + k)
        log(f"train step {k} margin {margin}")
        tr.step(_dev(b.V), _dev(b.labels), _dev(b.eps), info)
        p, m, v, integ, ref = elbo.train_step(p, m, v, k, integ, b.V.astype(np.float64),
                                              b.labels.astype(np.float64), b.eps.astype(np.float64),
                                              act=cfg.act, margin=margin, **HYPER)
        _check_info(info.cpu().numpy().astype(np.float64), ref, 1e-4, f"step {k}")
    pg = tr.params()
    tr.close()
    for name in elbo.PARAMS:
        d = np.abs(pg[name].astype(np.float64) - p[name])
        assert float(d.max()) <= 2 * 5 * lr, name
        assert float(np.mean(d > 1e-2 * lr)) <= 0.02, (name, float(np.mean(d > 1e-2 * lr)))


def test_steps_are_deterministic():
    import torch
    cfg = _cfg(8, 32, 64, 16, "relu")
    p0 = _init(cfg)
    out = []
    for _ in range(2):
        tr = _trainer(cfg, p0)
        for k in range(3):
            b = wl.training_batch(cfg, 2000, seed=200 + k)
            tr.step(_dev(b.V), _dev(b.labels), _dev(b.eps))
        torch.cuda.synchronize()
        out.append(tr.params())
        tr.close()
    for name in elbo.PARAMS:
        assert np.array_equal(out[0][name], out[1][name]), name


def test_batch_size_may_change_between_steps():
    """A trainer keeps working when the batch grows (buffers regrow) and shrinks again."""
    import torch
    cfg = _cfg(4, 8, 33, 3, "tanh")
    p0 = _init(cfg)
    tr = _trainer(cfg, p0)
    p, m, v = _oracle_state(p0)
    integ = 0.0
    info = torch.zeros(4, dtype=torch.float32, device="cuda")
    for k, B in enumerate((5, 700, 17), start=1):
        b = wl.training_batch(cfg, B, seed=300 + k)
        tr.step(_dev(b.V), _dev(b.labels), _dev(b.eps), info)
        p, m, v, integ, ref = elbo.train_step(p, m, v, k, integ, b.V.astype(np.float64),
                                              b.labels.astype(np.float64), b.eps.astype(np.float64),
                                              act=cfg.act, **HYPER)
        _check_info(info.cpu().numpy().astype(np.float64), ref, 1e-4, f"B={B}")
    tr.close()


def test_graph_replay_matches_eager_steps():
    """The default step replays a captured HIP graph; a second trainer launches every kernel
    eagerly. Same seeded batches, same order: after every step the summary, and at the end the
    parameters and gradients, are bit-identical. Between replays the stream also runs unrelated
    eager work and the host synchronises; new batch pointers and a new batch size re-capture."""
    import torch
    cfg = _cfg(8, 32, 64, 16, "relu")
    p0 = _init(cfg)
    ga, eb = _trainer(cfg, p0), _trainer(cfg, p0)
    eb.set_graph(False)
    b1 = wl.training_batch(cfg, 2000, seed=401)
    b2 = wl.training_batch(cfg, 700, seed=402)
    d1 = [_dev(a) for a in (b1.V, b1.labels, b1.eps)]
    d2 = [_dev(a) for a in (b2.V, b2.labels, b2.eps)]
    ia = torch.zeros(4, dtype=torch.float32, device="cuda")
    ib = torch.zeros(4, dtype=torch.float32, device="cuda")
    junk = torch.randn(1 << 20, device="cuda")
    plan = [d1, d1, d1, d2, d2, d1, d1]
    for k, d in enumerate(plan):
        log(f"graph replay step {k} batch {d[0].shape[0]}")
        ga.step(*d, ia)
        junk.mul_(0.5).add_(1.0)                      # eager work between replays
        eb.step(*d, ib)
        torch.cuda.synchronize()
        if k == 2:                                    # same pointers, contents rewritten in place
            d1[0].copy_(_dev(wl.training_batch(cfg, 2000, seed=403).V))
        assert np.array_equal(ia.cpu().numpy(), ib.cpu().numpy()), k
    pa, pb = ga.params(), eb.params()
    qa, qb = ga.grads(), eb.grads()
    for name in elbo.PARAMS:
        assert np.array_equal(pa[name], pb[name]), name
        assert np.array_equal(qa[name], qb[name]), name
    ga.set_graph(False)                               # frees the graph; eager steps continue from the same state
    ga.step(*d2, ia)
    eb.step(*d2, ib)
    torch.cuda.synchronize()
    assert np.array_equal(ia.cpu().numpy(), ib.cpu().numpy())
    ga.close()
    eb.close()
