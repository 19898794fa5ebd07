"""Thin ctypes binding of libenova_detect (include/enova_detect.h).

Every function keeps the C name and only marshals arguments: torch tensors become device
pointers, numpy arrays become host pointers, ``torch.cuda.current_stream()`` becomes the
``hipStream_t``. All computation happens in the library's HIP kernels; if the library is
missing this module raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libenova_detect.so")

ENOVA_OK, ENOVA_EINVAL, ENOVA_ESHAPE, ENOVA_ENOMEM, ENOVA_EHIP, ENOVA_EUNSUPPORTED, ENOVA_ENUMERIC = range(7)
ENOVA_F32, ENOVA_BF16 = 0, 1
ENOVA_RELU, ENOVA_TANH = 0, 1
ENOVA_KERNEL_AUTO, ENOVA_KERNEL_VALU, ENOVA_KERNEL_MFMA = 0, 1, 2

EXPORTS = ["enova_detect_init", "enova_detect_destroy", "enova_detect_window_offsets",
           "enova_detect_ref_stats", "enova_detect_score", "enova_detect_threshold",
           "enova_detect_flag", "enova_detect_set_timing", "enova_detect_kernel_times",
           "enova_detect_kernel_kind", "enova_stream_create", "enova_stream_push",
           "enova_stream_state", "enova_stream_kernel_times", "enova_stream_destroy",
           "enova_train_init", "enova_train_step", "enova_train_params_get", "enova_train_grads_get",
           "enova_train_set_timing", "enova_train_set_graph", "enova_train_kernel_times", "enova_train_destroy",
           "enova_detect_score_ext", "enova_detect_ext_time", "enova_detect_ext_mode", "enova_config_t_critical", "enova_config_init", "enova_config_destroy", "enova_config_window_offsets",
           "enova_config_scan", "enova_config_recommend", "enova_config_set_timing", "enova_config_kernel_time",
           "enova_detect_score_noalloc", "enova_status_str", "enova_last_error"]


class EnovaError(RuntimeError):
    def __init__(self, status, func, msg):
        super().__init__(f"{func} -> status {status}: {msg}")
        self.status = status


class enova_detect_config(ctypes.Structure):
    _fields_ = [("metrics", ctypes.c_int32), ("window", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("latent", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("act", ctypes.c_int32), ("kernel", ctypes.c_int32), ("ref_frac", ctypes.c_float)]


class enova_detect_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")]


class enova_train_config(ctypes.Structure):
    _fields_ = [("inputs", ctypes.c_int32), ("hidden", ctypes.c_int32), ("latent", ctypes.c_int32),
                ("act", ctypes.c_int32), ("lr", ctypes.c_float), ("adam_b1", ctypes.c_float),
                ("adam_b2", ctypes.c_float), ("adam_eps", ctypes.c_float), ("kl_set", ctypes.c_float),
                ("kp", ctypes.c_float), ("ki", ctypes.c_float), ("beta_min", ctypes.c_float),
                ("beta_max", ctypes.c_float), ("anomaly_margin", ctypes.c_float)]


class enova_config_params(ctypes.Structure):
    _fields_ = [("metrics", ctypes.c_int32), ("window", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("col_finished", ctypes.c_int32), ("col_running", ctypes.c_int32),
                ("col_exec_time", ctypes.c_int32), ("col_mem_util", ctypes.c_int32), ("alpha", ctypes.c_double),
                ("q_extreme", ctypes.c_double)]


class enova_train_params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")]


_lib = None


def lib():
    """Load the library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2407_09486_amd.build` "
                           "(or __graft_entry__.build())")
    # torch's GPU runtime first: the library then binds to the HIP runtime already in the process
    # (the one that owns the tensors and streams it is given). Loaded and initialised the other
    # way round, torch can fail to find the device.
    import torch
    torch.cuda.is_available()
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, F, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double
    st = ctypes.c_int
    L.enova_detect_init.argtypes = [ctypes.POINTER(enova_detect_config),
                                    ctypes.POINTER(enova_detect_weights), ctypes.POINTER(P)]
    L.enova_detect_destroy.argtypes = [P]
    L.enova_detect_window_offsets.argtypes = [P, P, I32, P]
    L.enova_detect_ref_stats.argtypes = [P, P, P, I32, P, P, P]
    L.enova_detect_score.argtypes = [P, P, P, P, I32, I64, P, P, F, P, P, P, P]
    L.enova_detect_score_noalloc.argtypes = [P, P, P, P, I32, I64, P, P, F, P, P, P, P]
    L.enova_detect_threshold.argtypes = [P, P, P, P, I32, I64, D, D, P, P, P, P]
    L.enova_detect_flag.argtypes = [P, P, I64, F, P, P]
    L.enova_detect_set_timing.argtypes = [P, I32]
    L.enova_detect_kernel_times.argtypes = [P, P, P]
    L.enova_detect_kernel_kind.argtypes = [P, P]
    L.enova_stream_create.argtypes = [P, I32, P, P, P, P, D, D, I32, ctypes.POINTER(P), P]
    L.enova_stream_push.argtypes = [P, P, P, P, P, P, P]
    L.enova_stream_state.argtypes = [P, P, P, P, P, P]
    L.enova_stream_kernel_times.argtypes = [P, P, P]
    L.enova_stream_destroy.argtypes = [P]
    L.enova_train_init.argtypes = [ctypes.POINTER(enova_train_config), ctypes.POINTER(enova_detect_weights),
                                   ctypes.POINTER(P)]
    L.enova_train_step.argtypes = [P, P, P, P, I32, P, P]
    L.enova_train_params_get.argtypes = [P, ctypes.POINTER(enova_train_params), P]
    L.enova_train_grads_get.argtypes = [P, ctypes.POINTER(enova_train_params), P]
    L.enova_train_set_timing.argtypes = [P, I32]
    L.enova_train_set_graph.argtypes = [P, I32]
    L.enova_train_kernel_times.argtypes = [P, P, P]
    L.enova_train_destroy.argtypes = [P]
    L.enova_detect_score_ext.argtypes = [P, P, P, P, I32, I64, P, P, I32, P, P, P, P, P]
    L.enova_detect_ext_time.argtypes = [P, P]
    L.enova_detect_ext_mode.argtypes = [P, P]
    L.enova_config_t_critical.argtypes = [D, I32, P]
    L.enova_config_init.argtypes = [ctypes.POINTER(enova_config_params), ctypes.POINTER(P)]
    L.enova_config_destroy.argtypes = [P]
    L.enova_config_window_offsets.argtypes = [P, P, I32, P]
    L.enova_config_scan.argtypes = [P, P, P, P, I32, I64, P, P, P, P, P, P, P]
    L.enova_config_recommend.argtypes = [P, P, P, I32, P, P, P, P, P, P]
    L.enova_config_set_timing.argtypes = [P, I32]
    L.enova_config_kernel_time.argtypes = [P, P]
    for name in EXPORTS[:-2]:
        getattr(L, name).restype = st
    L.enova_status_str.argtypes = [st]
    L.enova_status_str.restype = ctypes.c_char_p
    L.enova_last_error.argtypes = []
    L.enova_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status, func):
    if status != ENOVA_OK:
        raise EnovaError(status, func, lib().enova_last_error().decode())


def _dptr(t):
    """Device pointer of a torch tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _hptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


# ----------------------------------------------------------------------------- C entry points
def enova_detect_init(config: enova_detect_config, weights: dict):
    """weights: host numpy arrays w1 (float32, or uint16 bf16 bits), b1, wmu, bmu, wlv, blv,
    wd1, bd1, wd2, bd2 (float32), row-major as in the header. Returns the handle (int)."""
    keep = {}
    for k, v in weights.items():
        keep[k] = np.ascontiguousarray(v)
    names = [f[0] for f in enova_detect_weights._fields_]
    w = enova_detect_weights(**{k: _hptr(keep[k]) for k in names})
    h = ctypes.c_void_p()
    _check(lib().enova_detect_init(ctypes.byref(config), ctypes.byref(w), ctypes.byref(h)),
           "enova_detect_init")
    return h.value


def enova_detect_destroy(handle):
    _check(lib().enova_detect_destroy(ctypes.c_void_p(handle)), "enova_detect_destroy")


def enova_detect_window_offsets(handle, stream_offsets_host):
    so = np.ascontiguousarray(stream_offsets_host, dtype=np.int64)
    out = np.zeros(len(so), np.int64)
    _check(lib().enova_detect_window_offsets(ctypes.c_void_p(handle), _hptr(so), len(so) - 1, _hptr(out)),
           "enova_detect_window_offsets")
    return out


def enova_detect_ref_stats(handle, x, stream_offsets, n_streams, out_mean, out_std, stream=None):
    _check(lib().enova_detect_ref_stats(ctypes.c_void_p(handle), _dptr(x), _dptr(stream_offsets),
                                        int(n_streams), _dptr(out_mean), _dptr(out_std), _stream(stream)),
           "enova_detect_ref_stats")


def enova_detect_score(handle, x, stream_offsets, window_offsets, n_streams, n_windows,
                       ref_mean, ref_std, threshold, out_scores, out_md, out_flags, stream=None):
    _check(lib().enova_detect_score(ctypes.c_void_p(handle), _dptr(x), _dptr(stream_offsets),
                                    _dptr(window_offsets), int(n_streams), int(n_windows),
                                    _dptr(ref_mean), _dptr(ref_std), float(threshold),
                                    _dptr(out_scores), _dptr(out_md), _dptr(out_flags), _stream(stream)),
           "enova_detect_score")


def enova_detect_score_noalloc(handle, x, stream_offsets, window_offsets, n_streams, n_windows,
                               ref_mean, ref_std, threshold, out_scores, out_md, out_flags, stream=None):
    _check(lib().enova_detect_score_noalloc(ctypes.c_void_p(handle), _dptr(x), _dptr(stream_offsets),
                                            _dptr(window_offsets), int(n_streams), int(n_windows),
                                            _dptr(ref_mean), _dptr(ref_std), float(threshold),
                                            _dptr(out_scores), _dptr(out_md), _dptr(out_flags), _stream(stream)),
           "enova_detect_score_noalloc")


def enova_detect_threshold(handle, scores, stream_offsets, window_offsets, n_streams, n_windows,
                           level=0.98, q=1e-3, out_flags=None, stream=None):
    """Returns (threshold, info dict)."""
    thr = ctypes.c_float()
    info = (ctypes.c_double * 6)()
    _check(lib().enova_detect_threshold(ctypes.c_void_p(handle), _dptr(scores), _dptr(stream_offsets),
                                        _dptr(window_offsets), int(n_streams), int(n_windows),
                                        float(level), float(q), ctypes.byref(thr), info,
                                        _dptr(out_flags), _stream(stream)),
           "enova_detect_threshold")
    return thr.value, {"t": info[0], "n": int(info[1]), "n_peaks": int(info[2]), "gamma": info[3],
                       "sigma": info[4], "method": ("t", "moments", "mle")[int(info[5])]}


def enova_detect_flag(handle, scores, n_windows, threshold, out_flags, stream=None):
    _check(lib().enova_detect_flag(ctypes.c_void_p(handle), _dptr(scores), int(n_windows),
                                   float(threshold), _dptr(out_flags), _stream(stream)),
           "enova_detect_flag")


def enova_detect_set_timing(handle, enable):
    _check(lib().enova_detect_set_timing(ctypes.c_void_p(handle), 1 if enable else 0),
           "enova_detect_set_timing")


def enova_detect_kernel_times(handle):
    a, b = ctypes.c_double(), ctypes.c_double()
    _check(lib().enova_detect_kernel_times(ctypes.c_void_p(handle), ctypes.byref(a), ctypes.byref(b)),
           "enova_detect_kernel_times")
    return a.value, b.value


def enova_detect_kernel_kind(handle):
    k = ctypes.c_int32()
    _check(lib().enova_detect_kernel_kind(ctypes.c_void_p(handle), ctypes.byref(k)),
           "enova_detect_kernel_kind")
    return k.value


def enova_stream_create(handle, n_streams, ref_mean, ref_std, calib_scores, calib_offsets_host,
                        level=0.98, q=1e-3, peak_cap=4096, stream=None):
    """Returns the streaming-set handle (int). calib_offsets_host: numpy int64 [n+1]."""
    off = np.ascontiguousarray(calib_offsets_host, dtype=np.int64)
    h = ctypes.c_void_p()
    _check(lib().enova_stream_create(ctypes.c_void_p(handle), int(n_streams), _dptr(ref_mean), _dptr(ref_std),
                                     _dptr(calib_scores), _hptr(off), float(level), float(q), int(peak_cap),
                                     ctypes.byref(h), _stream(stream)),
           "enova_stream_create")
    return h.value


def enova_stream_push(shandle, x_step, out_scores=None, out_md=None, out_flags=None, stream=None):
    """Returns 1 if the push scored windows, else 0."""
    due = ctypes.c_int32()
    _check(lib().enova_stream_push(ctypes.c_void_p(shandle), _dptr(x_step), _dptr(out_scores), _dptr(out_md),
                                   _dptr(out_flags), ctypes.byref(due), _stream(stream)),
           "enova_stream_push")
    return due.value


def enova_stream_state(shandle, n_streams, stream=None):
    """Returns (t, z, n, n_peaks) as numpy arrays."""
    t = np.zeros(n_streams, np.float64)
    z = np.zeros(n_streams, np.float64)
    n = np.zeros(n_streams, np.int64)
    k = np.zeros(n_streams, np.int32)
    _check(lib().enova_stream_state(ctypes.c_void_p(shandle), _hptr(t), _hptr(z), _hptr(n), _hptr(k),
                                    _stream(stream)),
           "enova_stream_state")
    return t, z, n, k


def enova_stream_kernel_times(shandle):
    a, b = ctypes.c_double(), ctypes.c_double()
    _check(lib().enova_stream_kernel_times(ctypes.c_void_p(shandle), ctypes.byref(a), ctypes.byref(b)),
           "enova_stream_kernel_times")
    return a.value, b.value


def enova_stream_destroy(shandle):
    _check(lib().enova_stream_destroy(ctypes.c_void_p(shandle)), "enova_stream_destroy")


TRAIN_PARAMS = ("w1", "b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")


def enova_train_init(config: enova_train_config, weights: dict):
    """weights: host float32 arrays in the layout of enova_detect_weights. Returns the handle."""
    keep = {k: np.ascontiguousarray(weights[k], dtype=np.float32) for k in TRAIN_PARAMS}
    w = enova_detect_weights(**{k: _hptr(keep[k]) for k in TRAIN_PARAMS})
    h = ctypes.c_void_p()
    _check(lib().enova_train_init(ctypes.byref(config), ctypes.byref(w), ctypes.byref(h)), "enova_train_init")
    return h.value


def enova_train_step(thandle, V, labels, eps, batch, out_info=None, stream=None):
    _check(lib().enova_train_step(ctypes.c_void_p(thandle), _dptr(V), _dptr(labels), _dptr(eps), int(batch),
                                  _dptr(out_info), _stream(stream)),
           "enova_train_step")


def _train_get(fn, name, thandle, shapes, stream):
    out = {k: np.zeros(shapes[k], np.float32) for k in TRAIN_PARAMS}
    p = enova_train_params(**{k: _hptr(out[k]) for k in TRAIN_PARAMS})
    _check(fn(ctypes.c_void_p(thandle), ctypes.byref(p), _stream(stream)), name)
    return out


def enova_train_params_get(thandle, shapes, stream=None):
    """Returns the current parameters as host float32 arrays of the given shapes."""
    return _train_get(lib().enova_train_params_get, "enova_train_params_get", thandle, shapes, stream)


def enova_train_grads_get(thandle, shapes, stream=None):
    """Returns the last step's gradients of J as host float32 arrays of the given shapes."""
    return _train_get(lib().enova_train_grads_get, "enova_train_grads_get", thandle, shapes, stream)


def enova_train_set_timing(thandle, enable):
    _check(lib().enova_train_set_timing(ctypes.c_void_p(thandle), int(bool(enable))), "enova_train_set_timing")


def enova_train_set_graph(thandle, enable):
    _check(lib().enova_train_set_graph(ctypes.c_void_p(thandle), int(bool(enable))), "enova_train_set_graph")


def enova_train_kernel_times(thandle):
    """Returns (milliseconds in the last step's matrix products, milliseconds of the whole step)."""
    a, b = ctypes.c_double(), ctypes.c_double()
    _check(lib().enova_train_kernel_times(ctypes.c_void_p(thandle), ctypes.byref(a), ctypes.byref(b)),
           "enova_train_kernel_times")
    return a.value, b.value


def enova_train_destroy(thandle):
    _check(lib().enova_train_destroy(ctypes.c_void_p(thandle)), "enova_train_destroy")


ENOVA_NORM_REFERENCE, ENOVA_NORM_WINDOW = 0, 1


def enova_detect_score_ext(handle, x, stream_offsets, window_offsets, n_streams, n_windows, ref_mean, ref_std, norm,
                           out_scores=None, out_md=None, out_md_metric=None, out_recon=None, stream=None):
    _check(lib().enova_detect_score_ext(ctypes.c_void_p(handle), _dptr(x), _dptr(stream_offsets),
                                        _dptr(window_offsets), int(n_streams), int(n_windows), _dptr(ref_mean),
                                        _dptr(ref_std), int(norm), _dptr(out_scores), _dptr(out_md),
                                        _dptr(out_md_metric), _dptr(out_recon), _stream(stream)),
           "enova_detect_score_ext")


def enova_detect_ext_time(handle):
    v = ctypes.c_double()
    _check(lib().enova_detect_ext_time(ctypes.c_void_p(handle), ctypes.byref(v)), "enova_detect_ext_time")
    return v.value


def enova_detect_ext_mode(handle):
    v = ctypes.c_int32()
    _check(lib().enova_detect_ext_mode(ctypes.c_void_p(handle), ctypes.byref(v)), "enova_detect_ext_mode")
    return v.value


def enova_config_t_critical(alpha, dof):
    v = ctypes.c_double()
    _check(lib().enova_config_t_critical(float(alpha), int(dof), ctypes.byref(v)), "enova_config_t_critical")
    return v.value


class ConfigScanner:
    """Owns one configuration-scan handle (Section IV-A scans); methods call the C entry points."""

    def __init__(self, metrics, window, stride, col_finished, col_running, col_exec_time, col_mem_util,
                 dtype="f32", alpha=0.05, q_extreme=0.99):
        self.params = enova_config_params(metrics=metrics, window=window, stride=stride,
                                          dtype={"f32": ENOVA_F32, "bf16": ENOVA_BF16}[dtype],
                                          col_finished=col_finished, col_running=col_running,
                                          col_exec_time=col_exec_time, col_mem_util=col_mem_util,
                                          alpha=alpha, q_extreme=q_extreme)
        h = ctypes.c_void_p()
        _check(lib().enova_config_init(ctypes.byref(self.params), ctypes.byref(h)), "enova_config_init")
        self.handle = h.value

    def window_offsets(self, stream_offsets_host):
        so = np.ascontiguousarray(stream_offsets_host, dtype=np.int64)
        out = np.zeros(len(so), np.int64)
        _check(lib().enova_config_window_offsets(ctypes.c_void_p(self.handle), _hptr(so), len(so) - 1, _hptr(out)),
               "enova_config_window_offsets")
        return out

    def scan(self, x, stream_offsets, window_offsets, n_windows, stream=None):
        """Returns device tensors (intercept, slope, t, significant, mem_intercept, mem_slope)."""
        import torch
        dev = x.device
        n = stream_offsets.numel() - 1
        f = [torch.empty(max(n_windows, 1), dtype=torch.float32, device=dev)[:n_windows] for _ in range(5)]
        sig = torch.empty(max(n_windows, 1), dtype=torch.uint8, device=dev)[:n_windows]
        _check(lib().enova_config_scan(ctypes.c_void_p(self.handle), _dptr(x), _dptr(stream_offsets),
                                       _dptr(window_offsets), n, int(n_windows), _dptr(f[0]), _dptr(f[1]),
                                       _dptr(f[2]), _dptr(sig), _dptr(f[3]), _dptr(f[4]), _stream(stream)),
               "enova_config_scan")
        return f[0], f[1], f[2], sig, f[3], f[4]

    def recommend(self, x, stream_offsets, stream=None):
        """Returns device tensors (significant, n_limit, t_limit, max_num_seqs, gpu_memory)."""
        import torch
        dev = x.device
        n = stream_offsets.numel() - 1
        sig = torch.empty(max(n, 1), dtype=torch.uint8, device=dev)[:n]
        d = [torch.empty(max(n, 1), dtype=torch.float64, device=dev)[:n] for _ in range(4)]
        _check(lib().enova_config_recommend(ctypes.c_void_p(self.handle), _dptr(x), _dptr(stream_offsets), n,
                                            _dptr(sig), _dptr(d[0]), _dptr(d[1]), _dptr(d[2]), _dptr(d[3]),
                                            _stream(stream)),
               "enova_config_recommend")
        return sig, d[0], d[1], d[2], d[3]

    def set_timing(self, enable=True):
        _check(lib().enova_config_set_timing(ctypes.c_void_p(self.handle), int(bool(enable))),
               "enova_config_set_timing")

    def kernel_time(self):
        v = ctypes.c_double()
        _check(lib().enova_config_kernel_time(ctypes.c_void_p(self.handle), ctypes.byref(v)), "enova_config_kernel_time")
        return v.value

    def close(self):
        if self.handle:
            _check(lib().enova_config_destroy(ctypes.c_void_p(self.handle)), "enova_config_destroy")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ----------------------------------------------------------------------------- convenience
def make_config(metrics, window, stride, hidden, latent=16, dtype="f32", act="relu",
                kernel="auto", ref_frac=0.5) -> enova_detect_config:
    return enova_detect_config(
        metrics=metrics, window=window, stride=stride, hidden=hidden, latent=latent,
        dtype={"f32": ENOVA_F32, "bf16": ENOVA_BF16}[dtype],
        act={"relu": ENOVA_RELU, "tanh": ENOVA_TANH}[act],
        kernel={"auto": ENOVA_KERNEL_AUTO, "valu": ENOVA_KERNEL_VALU, "mfma": ENOVA_KERNEL_MFMA}[kernel],
        ref_frac=ref_frac)


class Detector:
    """Owns one library handle; methods call the C entry points on torch's current stream."""

    def __init__(self, metrics, window, stride, hidden, weights: dict, latent=16, dtype="f32",
                 act="relu", kernel="auto", ref_frac=0.5):
        self.cfg = make_config(metrics, window, stride, hidden, latent, dtype, act, kernel, ref_frac)
        self.dtype = dtype
        self.handle = enova_detect_init(self.cfg, weights)

    def close(self):
        if self.handle:
            enova_detect_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def kernel_kind(self):
        return {1: "valu", 2: "mfma"}[enova_detect_kernel_kind(self.handle)]

    def ext_fused(self):
        return enova_detect_ext_mode(self.handle) == 1

    def window_offsets(self, stream_offsets_host):
        return enova_detect_window_offsets(self.handle, stream_offsets_host)

    def score(self, x, stream_offsets, window_offsets, n_windows, ref_mean=None, ref_std=None,
              threshold=math.nan, md=True, flags=False, stream=None):
        import torch
        dev = x.device
        n = stream_offsets.numel() - 1
        scores = torch.empty(max(n_windows, 1), dtype=torch.float32, device=dev)[:n_windows]
        mdv = torch.empty(max(n_windows, 1), dtype=torch.float32, device=dev)[:n_windows] if md else None
        fl = torch.empty(max(n_windows, 1), dtype=torch.uint8, device=dev)[:n_windows] if flags else None
        enova_detect_score(self.handle, x, stream_offsets, window_offsets, n, n_windows, ref_mean, ref_std,
                           threshold, scores, mdv, fl, stream)
        return scores, mdv, fl

    def score_ext(self, x, stream_offsets, window_offsets, n_windows, norm="reference", ref_mean=None,
                  ref_std=None, stream=None, scores_only=False):
        """Output variants: returns device tensors (scores, md, md_metric [N, M], recon_err); with
        scores_only the last three are None (the decoder is then not evaluated)."""
        import torch
        dev = x.device
        n = stream_offsets.numel() - 1
        M = self.cfg.metrics
        k = 1 if scores_only else 3
        f = [torch.empty(max(n_windows, 1), dtype=torch.float32, device=dev)[:n_windows] for _ in range(k)]
        f += [None] * (3 - k)
        mdm = None if scores_only else torch.empty((max(n_windows, 1), M), dtype=torch.float32, device=dev)[:n_windows]
        enova_detect_score_ext(self.handle, x, stream_offsets, window_offsets, n, n_windows, ref_mean, ref_std,
                               {"reference": ENOVA_NORM_REFERENCE, "window": ENOVA_NORM_WINDOW}[norm], f[0], f[1],
                               mdm, f[2], stream)
        return f[0], f[1], mdm, f[2]

    def threshold(self, scores, stream_offsets, window_offsets, level=0.98, q=1e-3, flags=False,
                  stream=None):
        import torch
        n = stream_offsets.numel() - 1
        nw = scores.numel()
        fl = torch.empty(max(nw, 1), dtype=torch.uint8, device=scores.device)[:nw] if flags else None
        thr, info = enova_detect_threshold(self.handle, scores, stream_offsets, window_offsets, n, nw,
                                           level, q, fl, stream)
        return thr, info, fl


class StreamSet:
    """Owns one streaming-set handle of a Detector (which must stay open)."""

    def __init__(self, det: Detector, ref_mean, ref_std, calib_scores, calib_offsets_host, level=0.98,
                 q=1e-3, peak_cap=4096, stream=None):
        self.det = det
        self.n = len(calib_offsets_host) - 1
        self.handle = enova_stream_create(det.handle, self.n, ref_mean, ref_std, calib_scores,
                                          calib_offsets_host, level, q, peak_cap, stream)

    def push(self, x_step, scores=None, md=None, flags=None, stream=None):
        return enova_stream_push(self.handle, x_step, scores, md, flags, stream)

    def state(self, stream=None):
        return enova_stream_state(self.handle, self.n, stream)

    def kernel_times(self):
        return enova_stream_kernel_times(self.handle)

    def close(self):
        if self.handle:
            enova_stream_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Trainer:
    """Owns one trainer handle: semi-supervised ELBO steps of a D -> H -> L VAE on the device."""

    def __init__(self, inputs, hidden, latent, weights: dict, act="relu", lr=1e-3, adam_b1=0.9,
                 adam_b2=0.999, adam_eps=1e-8, kl_set=3.0, kp=0.01, ki=1e-4, beta_min=0.0, beta_max=1.0,
                 margin=math.inf):
        self.cfg = enova_train_config(inputs=inputs, hidden=hidden, latent=latent,
                                      act={"relu": ENOVA_RELU, "tanh": ENOVA_TANH}[act], lr=lr,
                                      adam_b1=adam_b1, adam_b2=adam_b2, adam_eps=adam_eps, kl_set=kl_set,
                                      kp=kp, ki=ki, beta_min=beta_min, beta_max=beta_max,
                                      anomaly_margin=margin)
        D, H, L = inputs, hidden, latent
        self.shapes = {"w1": (H, D), "b1": (H,), "wmu": (L, H), "bmu": (L,), "wlv": (L, H), "blv": (L,),
                       "wd1": (H, L), "bd1": (H,), "wd2": (D, H), "bd2": (D,)}
        self.handle = enova_train_init(self.cfg, weights)

    def step(self, V, labels, eps, info=None, stream=None):
        enova_train_step(self.handle, V, labels, eps, V.shape[0], info, stream)

    def params(self, stream=None):
        return enova_train_params_get(self.handle, self.shapes, stream)

    def set_timing(self, enable=True):
        enova_train_set_timing(self.handle, enable)

    def set_graph(self, enable=True):
        enova_train_set_graph(self.handle, enable)

    def kernel_times(self):
        return enova_train_kernel_times(self.handle)

    def grads(self, stream=None):
        return enova_train_grads_get(self.handle, self.shapes, stream)

    def close(self):
        if self.handle:
            enova_train_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def weights_for_library(wt, dtype="f32") -> dict:
    """Host arrays in the library's layout from a ``workloads.Weights``."""
    d = {k: np.ascontiguousarray(getattr(wt, k), dtype=np.float32)
         for k in ("b1", "wmu", "bmu", "wlv", "blv", "wd1", "bd1", "wd2", "bd2")}
    d["w1"] = (np.ascontiguousarray(wt.w1_bits) if dtype == "bf16"
               else np.ascontiguousarray(wt.w1, dtype=np.float32))
    return d
