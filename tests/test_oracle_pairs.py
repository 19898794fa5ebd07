"""Pin of the oracle's sampled-window driver (``oracle.score_pairs``), CPU only.

The full-size parity tests check the library on sampled (stream, window) pairs that the oracle
scores one by one. That driver must give, for every pair, exactly what the whole-batch driver
gives at the same position: the same window of the same stream, normalised with that stream's
statistics. Bit-for-bit equality is asserted (both drivers run the same fp64 window evaluation,
so any difference is a pairing or statistics mistake, not rounding).
"""
import numpy as np
import pytest

import oracle
from paper_2407_09486_amd import workloads as wl


def _ragged(seed, M, lengths):
    rng = np.random.default_rng(seed)
    offs = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(lengths, out=offs[1:])
    x = rng.standard_normal((int(offs[-1]), M)) * rng.uniform(0.5, 3.0, M) + rng.uniform(-2, 2, M)
    return x, offs


@pytest.mark.parametrize("bf16,act,ext,stride", [(False, "relu", False, 1), (False, "tanh", True, 3),
                                                 (True, "relu", False, 2), (True, "tanh", True, 1)])
def test_pairs_equal_batch_bit_for_bit(bf16, act, ext, stride):
    W, M = 7, 3
    # ragged: empty, shorter than a window, exactly one window, a stride past the end, longer streams
    lengths = [0, 5, 7, 9, 40, 0, 61, 6, 33]
    x, offs = _ragged(100 + stride, M, lengths)
    cfg = wl.CONFIGS["c5"].replace(window=W, stride=stride, metrics=M, hidden=11, latent=4, act=act)
    Wt = wl.make_weights(cfg, bias_scale=0.3).as_f64()
    n = len(lengths)
    ref = None
    if ext:
        rng = np.random.default_rng(7)
        ref = (rng.uniform(-1, 1, (n, M)), rng.uniform(0.5, 2.0, (n, M)))
    kw = dict(window=W, stride=stride, weights=Wt, act=act, bf16=bf16,
              ref_mean=None if ref is None else ref[0], ref_std=None if ref is None else ref[1])
    sc, md, info = oracle.score(x, offs, return_stats=True, **kw)
    woff = info["window_offsets"]
    nwin = np.diff(woff)
    assert nwin[0] == 0 and nwin[1] == 0 and nwin[2] == 1 and nwin[7] == 0
    pairs = [(s, k) for s in range(n) for k in range(int(nwin[s]))]
    rng = np.random.default_rng(3)
    order = rng.permutation(len(pairs))                  # pairs in any order, streams interleaved
    ps = np.array([pairs[i][0] for i in order], np.int32)
    pk = np.array([pairs[i][1] for i in order], np.int64)
    psc, pmd, pscale = oracle.score_pairs(x, offs, ps, pk, **kw)
    pos = woff[ps] + pk
    assert np.array_equal(psc, sc[pos])
    assert np.array_equal(pmd, md[pos])
    assert np.array_equal(pscale, info["md_scale"][pos])
    # repeated pairs and a single pair give the same values
    psc2, _, _ = oracle.score_pairs(x, offs, np.r_[ps[:3], ps[:3]], np.r_[pk[:3], pk[:3]], **kw)
    assert np.array_equal(psc2, np.r_[sc[pos[:3]], sc[pos[:3]]])
    one, _, _ = oracle.score_pairs(x, offs, ps[-1:], pk[-1:], **kw)
    assert one[0] == sc[pos[-1]]


def test_pairs_use_each_streams_own_statistics():
    """Two streams with identical rows but different scales give identical scores only when each
    pair is normalised with its own stream's reference statistics."""
    W, M = 5, 2
    rng = np.random.default_rng(9)
    a = rng.standard_normal((30, M))
    x = np.concatenate([a, 4.0 * a + 3.0])
    offs = np.array([0, 30, 60], np.int64)
    cfg = wl.CONFIGS["c5"].replace(window=W, stride=1, metrics=M, hidden=6, latent=3)
    Wt = wl.make_weights(cfg, bias_scale=0.2).as_f64()
    ks = np.arange(26, dtype=np.int64)
    s0, m0, _ = oracle.score_pairs(x, offs, np.zeros(26, np.int32), ks, window=W, stride=1, weights=Wt)
    s1, m1, _ = oracle.score_pairs(x, offs, np.ones(26, np.int32), ks, window=W, stride=1, weights=Wt)
    np.testing.assert_allclose(s1, s0, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(m1, m0, rtol=1e-10, atol=1e-13)
    assert not np.allclose(s0, s0[::-1])                 # the windows themselves differ


def test_pairs_reject_out_of_range_windows():
    x, offs = _ragged(1, 2, [10, 4])
    cfg = wl.CONFIGS["c5"].replace(window=5, stride=1, metrics=2, hidden=4, latent=2)
    Wt = wl.make_weights(cfg).as_f64()
    with pytest.raises(AssertionError):
        oracle.score_pairs(x, offs, np.array([0], np.int32), np.array([6], np.int64), window=5, stride=1, weights=Wt)
    with pytest.raises(AssertionError):
        oracle.score_pairs(x, offs, np.array([1], np.int32), np.array([0], np.int64), window=5, stride=1, weights=Wt)
