"""C-ABI contract checks that need no GPU: the library loads, exports every declared entry
point, and rejects invalid arguments on the host before touching a device."""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

from paper_2407_09486_amd import binding
from paper_2407_09486_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _ensure_built():
    if not os.path.exists(binding.LIB_PATH):
        from paper_2407_09486_amd import build
        build.build_library()


def declared_functions():
    names = []
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b(enova_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    _ensure_built()
    L = ctypes.CDLL(binding.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 12, names
    for n in names:
        assert hasattr(L, n), f"{n} declared in include/ but not exported"
    assert set(names) == set(binding.EXPORTS)


def test_status_strings():
    _ensure_built()
    L = binding.lib()
    for s in range(7):
        assert L.enova_status_str(s)
    assert L.enova_status_str(99) == b"unknown status"


def _init_status(**over):
    cfg = dict(metrics=8, window=32, stride=1, hidden=32, latent=16)
    cfg.update(over)
    c = binding.make_config(**{k: v for k, v in cfg.items() if k in ("metrics", "window", "stride", "hidden", "latent")})
    for k in ("dtype", "act", "kernel", "ref_frac"):
        if k in over:
            setattr(c, k, over[k])
    W = wl.make_weights(wl.CONFIGS["c1"])
    w = binding.weights_for_library(W)
    keep = [np.ascontiguousarray(v) for v in w.values()]
    ws = binding.enova_detect_weights(**{k: ctypes.c_void_p(v.ctypes.data) for k, v in zip(w.keys(), keep)})
    h = ctypes.c_void_p()
    st = binding.lib().enova_detect_init(ctypes.byref(c), ctypes.byref(ws), ctypes.byref(h))
    return st, h.value


@pytest.mark.parametrize("over", [dict(metrics=0), dict(window=0), dict(stride=-1), dict(hidden=0),
                                  dict(latent=0), dict(latent=65), dict(dtype=7), dict(act=3),
                                  dict(kernel=9), dict(ref_frac=0.0), dict(ref_frac=1.5),
                                  dict(window=4096, metrics=32)])
def test_init_rejects_bad_config(over):
    _ensure_built()
    st, h = _init_status(**over)
    assert st == binding.ENOVA_EINVAL and not h
    assert binding.lib().enova_last_error()


@pytest.mark.parametrize("over,text", [(dict(hidden=300, kernel=binding.ENOVA_KERNEL_MFMA), "H=300 L=16"),
                                       (dict(hidden=1100, kernel=binding.ENOVA_KERNEL_VALU), "hidden width 1100")])
def test_unsupported_shapes_are_named_in_the_error(over, text):
    """Shapes no kernel takes are refused on the host before any device call, and the message
    names the shape (it is formatted before the half-built detector is released)."""
    _ensure_built()
    st, h = _init_status(**over)
    assert st == binding.ENOVA_EUNSUPPORTED and not h
    assert text in binding.lib().enova_last_error().decode()


def test_null_arguments_are_rejected():
    _ensure_built()
    L = binding.lib()
    assert L.enova_detect_init(None, None, None) == binding.ENOVA_EINVAL
    h = ctypes.c_void_p()
    c = binding.make_config(8, 32, 1, 32)
    assert L.enova_detect_init(ctypes.byref(c), None, ctypes.byref(h)) == binding.ENOVA_EINVAL
    so = np.array([0, 10], np.int64)
    out = np.zeros(2, np.int64)
    assert L.enova_detect_window_offsets(None, so.ctypes.data, 1, out.ctypes.data) == binding.ENOVA_EINVAL
    assert L.enova_detect_score(None, None, None, None, 0, 0, None, None, 0.0, None, None, None,
                                None) == binding.ENOVA_EINVAL
    assert L.enova_detect_destroy(None) == binding.ENOVA_OK
    mode = ctypes.c_int32()
    assert L.enova_detect_ext_mode(None, ctypes.byref(mode)) == binding.ENOVA_EINVAL
    thr = ctypes.c_float()
    assert L.enova_detect_threshold(None, None, None, None, 1, 1, 0.98, 1e-3, ctypes.byref(thr), None,
                                    None, None) == binding.ENOVA_EINVAL


def test_streaming_entry_points_reject_null_handles():
    _ensure_built()
    L = binding.lib()
    h = ctypes.c_void_p()
    off = np.array([0, 0], np.int64)
    assert L.enova_stream_create(None, 1, None, None, None, off.ctypes.data, 0.98, 1e-3, 16,
                                 ctypes.byref(h), None) == binding.ENOVA_EINVAL
    assert L.enova_stream_push(None, None, None, None, None, None, None) == binding.ENOVA_EINVAL
    assert L.enova_stream_state(None, None, None, None, None, None) == binding.ENOVA_EINVAL
    assert L.enova_stream_destroy(None) == binding.ENOVA_OK


@pytest.mark.parametrize("over", [dict(inputs=0), dict(hidden=0), dict(latent=0), dict(act=5), dict(lr=0.0),
                                  dict(adam_b1=1.0), dict(adam_b2=-0.1), dict(adam_eps=0.0),
                                  dict(beta_min=1.0, beta_max=0.5), dict(anomaly_margin=0.0),
                                  dict(anomaly_margin=float("nan"))])
def test_training_entry_points_reject_bad_arguments(over):
    _ensure_built()
    L = binding.lib()
    base = dict(inputs=8, hidden=4, latent=2, act=binding.ENOVA_RELU, lr=1e-3, adam_b1=0.9, adam_b2=0.999,
                adam_eps=1e-8, kl_set=3.0, kp=0.01, ki=1e-4, beta_min=0.0, beta_max=1.0,
                anomaly_margin=float("inf"))
    base.update(over)
    c = binding.enova_train_config(**base)
    keep = [np.zeros(64, np.float32) for _ in range(10)]
    ws = binding.enova_detect_weights(*[ctypes.c_void_p(a.ctypes.data) for a in keep])
    h = ctypes.c_void_p()
    assert L.enova_train_init(ctypes.byref(c), ctypes.byref(ws), ctypes.byref(h)) == binding.ENOVA_EINVAL
    assert not h.value and L.enova_last_error()
    assert L.enova_train_init(None, None, None) == binding.ENOVA_EINVAL
    assert L.enova_train_step(None, None, None, None, 4, None, None) == binding.ENOVA_EINVAL
    assert L.enova_train_params_get(None, None, None) == binding.ENOVA_EINVAL
    assert L.enova_train_grads_get(None, None, None) == binding.ENOVA_EINVAL
    assert L.enova_train_set_timing(None, 1) == binding.ENOVA_EINVAL
    assert L.enova_train_set_graph(None, 1) == binding.ENOVA_EINVAL
    a, b = ctypes.c_double(), ctypes.c_double()
    assert L.enova_train_kernel_times(None, ctypes.byref(a), ctypes.byref(b)) == binding.ENOVA_EINVAL
    assert L.enova_train_destroy(None) == binding.ENOVA_OK


def test_binding_refuses_host_tensors():
    import torch
    with pytest.raises(ValueError):
        binding._dptr(torch.zeros(3))


def test_config_t_critical_matches_scipy():
    _ensure_built()
    from scipy import stats
    for alpha in (0.05, 0.01, 0.2):
        for dof in (1, 2, 3, 10, 62, 1000, 100000):
            v = binding.enova_config_t_critical(alpha, dof)
            # lgamma of large arguments limits the library to ~1e-10 relative at dof ~ 1e5
            assert v == pytest.approx(stats.t.ppf(1 - alpha / 2, dof), rel=1e-9)


@pytest.mark.parametrize("over", [dict(window=2), dict(window=4097), dict(stride=0), dict(metrics=0),
                                  dict(col_running=7), dict(col_mem_util=-1), dict(alpha=0.0), dict(alpha=1.0),
                                  dict(q_extreme=1.0), dict(dtype=5)])
def test_config_init_rejects_bad_params(over):
    _ensure_built()
    L = binding.lib()
    base = dict(metrics=7, window=64, stride=1, dtype=binding.ENOVA_F32, col_finished=0, col_running=1,
                col_exec_time=4, col_mem_util=5, alpha=0.05, q_extreme=0.99)
    base.update(over)
    p = binding.enova_config_params(**base)
    h = ctypes.c_void_p()
    assert L.enova_config_init(ctypes.byref(p), ctypes.byref(h)) == binding.ENOVA_EINVAL and not h.value
    assert L.enova_config_init(None, None) == binding.ENOVA_EINVAL
    assert L.enova_config_scan(None, None, None, None, 1, 1, None, None, None, None, None, None,
                               None) == binding.ENOVA_EINVAL
    assert L.enova_config_recommend(None, None, None, 1, None, None, None, None, None, None) == binding.ENOVA_EINVAL
    v = ctypes.c_double()
    assert L.enova_config_t_critical(0.05, 0, ctypes.byref(v)) == binding.ENOVA_EINVAL
    assert L.enova_config_destroy(None) == binding.ENOVA_OK


def test_output_variants_reject_bad_arguments():
    _ensure_built()
    L = binding.lib()
    assert L.enova_detect_score_ext(None, None, None, None, 1, 1, None, None, 0, None, None, None, None,
                                    None) == binding.ENOVA_EINVAL
    v = ctypes.c_double()
    assert L.enova_detect_ext_time(None, ctypes.byref(v)) == binding.ENOVA_EINVAL


@pytest.mark.parametrize("argv", [["--gpus", "2"], ["--gpus", "8", "--steps", "1"]])
def test_bench_refuses_more_than_one_gpu(argv):
    """The bench measures one GPU's share; asked for several it exits with status 2 and says so
    before touching a device."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""
