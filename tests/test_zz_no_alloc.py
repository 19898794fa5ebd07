"""The allocation-free scoring entry point (enova_detect_score_noalloc) against enova_detect_score.

Both run the same kernels; the allocation-free one takes its workspace from the library's fixed
per-device scratch array instead of the detector's own workspace. Outputs must be bit-identical,
on consecutive calls whose second input is smaller (the array keeps the previous call's contents),
across detectors of different shapes sharing the array, with and without caller-given statistics
and flags, on both scoring kernels; a call needing more scratch than the array holds is refused
before any launch.
"""
import math

import numpy as np
import pytest

from harness import detector, log, upload
from paper_2407_09486_amd import binding
from paper_2407_09486_amd import workloads as wl

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 16 << 20


def _run(det, w, noalloc, ref=None, threshold=math.nan):
    import torch
    x, so = upload(w)
    woff = det.window_offsets(w.stream_offsets)
    N = int(woff[-1])
    wo = torch.from_numpy(woff).cuda()
    sc = torch.full((N,), -7.0, dtype=torch.float32, device="cuda")
    md = torch.full((N,), -7.0, dtype=torch.float32, device="cuda")
    fl = torch.full((N,), 9, dtype=torch.uint8, device="cuda")
    rm = rs = None
    if ref is not None:
        rm = torch.from_numpy(np.ascontiguousarray(ref[0], np.float32)).cuda()
        rs = torch.from_numpy(np.ascontiguousarray(ref[1], np.float32)).cuda()
    fn = binding.enova_detect_score_noalloc if noalloc else binding.enova_detect_score
    fn(det.handle, x, so, wo, w.n_streams, N, rm, rs, threshold, sc, md, fl)
    torch.cuda.synchronize()
    return sc.cpu().numpy(), md.cpu().numpy(), fl.cpu().numpy()


def _same(a, b, what):
    for name, u, v in zip(("scores", "md", "flags"), a, b):
        assert np.array_equal(u, v, equal_nan=True), f"{what}: {name} differ"


def _workload(name, streams, **over):
    cfg = wl.CONFIGS[name].replace(**over) if over else wl.CONFIGS[name]
    return cfg, wl.generate(cfg, streams=np.asarray(streams))


@pytest.mark.parametrize("kernel", ["auto", "valu"])
def test_noalloc_matches_score_on_consecutive_calls(kernel):
    cfg, big = _workload("c5", [0, 3, 7, 11, 12], t_min=512, t_max=20000)
    _, small = _workload("c5", [5, 2], t_min=300, t_max=900)
    weights = wl.make_weights(cfg, bias_scale=0.05)
    det = detector(cfg, weights, kernel)
    log(f"[noalloc] c5 shape kernel={det.kernel_kind} big={np.diff(big.stream_offsets).tolist()} "
        f"small={np.diff(small.stream_offsets).tolist()}")
    ref_big = _run(det, big, False)
    ref_small = _run(det, small, False)
    # first call: the larger input; second call: a smaller one over what the first left behind
    _same(_run(det, big, True), ref_big, "first call")
    _same(_run(det, small, True), ref_small, "second, smaller call")
    # with flags, and with caller-given statistics (no statistics in the scratch)
    thr = float(np.quantile(ref_big[0], 0.97))
    _same(_run(det, big, True, threshold=thr), _run(det, big, False, threshold=thr), "flags")
    rng = np.random.default_rng(4)
    ref = (rng.uniform(-1, 1, (small.n_streams, cfg.metrics)), rng.uniform(0.5, 2, (small.n_streams, cfg.metrics)))
    _same(_run(det, small, True, ref=ref), _run(det, small, False, ref=ref), "given statistics")
    det.close()


def test_noalloc_shared_by_detectors_of_different_shapes():
    cfg4, w4 = _workload("c4", [1, 9, 4])
    cfg3, w3 = _workload("c3", [2, 8, 5, 1])
    d4 = detector(cfg4, wl.make_weights(cfg4, bias_scale=0.05))
    d3 = detector(cfg3, wl.make_weights(cfg3, bias_scale=0.05))
    log(f"[noalloc] c4 x {w4.n_streams} streams and c3 x {w3.n_streams} streams interleaved")
    r4 = _run(d4, w4, False)
    r3 = _run(d3, w3, False)
    for _ in range(2):
        _same(_run(d4, w4, True), r4, "c4 shape")
        _same(_run(d3, w3, True), r3, "c3 shape")
    d4.close()
    d3.close()


def test_noalloc_refuses_more_than_its_scratch():
    """2^20 mostly empty streams need 2 * 2^20 * 16 * 4 bytes of statistics alone (> 16 MiB):
    refused on the host before any launch. With caller-given statistics the same call needs only
    the tile offsets and block map (about 12.6 MB), fits, and matches the other entry point."""
    import torch
    cfg = wl.CONFIGS["c5"]
    det = detector(cfg, wl.make_weights(cfg))
    n = 1 << 20
    lengths = np.zeros(n, np.int64)
    lengths[-1] = 200
    offs = np.zeros(n + 1, np.int64)
    np.cumsum(lengths, out=offs[1:])
    log(f"[noalloc] refusal with {n} streams")
    assert 2 * n * cfg.metrics * 4 > SCRATCH_BYTES
    up = lambda v: (v + 255) // 256 * 256
    assert up((n + 1) * 8) + up(((137 + 255) // 256 + n) * 4) <= SCRATCH_BYTES
    x = torch.zeros((200, cfg.metrics), dtype=torch.float32, device="cuda")
    so = torch.from_numpy(offs).cuda()
    woff = det.window_offsets(offs)
    N = int(woff[-1])
    wo = torch.from_numpy(woff).cuda()
    sc = torch.zeros(N, dtype=torch.float32, device="cuda")
    with pytest.raises(binding.EnovaError) as ei:
        binding.enova_detect_score_noalloc(det.handle, x, so, wo, n, N, None, None, math.nan, sc, None, None)
    assert ei.value.status == 2 and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert float(sc.abs().sum()) == 0.0                  # nothing was launched
    # the same call with caller-given statistics fits (tiles and map only) and matches the other entry
    rm = torch.zeros((n, cfg.metrics), dtype=torch.float32, device="cuda")
    rs = torch.ones((n, cfg.metrics), dtype=torch.float32, device="cuda")
    sc2 = torch.zeros(N, dtype=torch.float32, device="cuda")
    binding.enova_detect_score_noalloc(det.handle, x, so, wo, n, N, rm, rs, math.nan, sc, None, None)
    binding.enova_detect_score(det.handle, x, so, wo, n, N, rm, rs, math.nan, sc2, None, None)
    torch.cuda.synchronize()
    assert torch.equal(sc, sc2)
    det.close()
