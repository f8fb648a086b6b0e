"""Thin ctypes binding of libfedoptima.so.

Functions carry the C names and only marshal arguments: torch tensors become
device pointers (``data_ptr()``), numpy arrays host pointers, streams the raw
``hipStream_t`` of a ``torch.cuda.Stream``.  Every step of the hot path runs in
the library's HIP kernels; there is no Python or CPU fallback, and loading
fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfedoptima.so")

FO_OK, FO_SKIPPED, FO_EMPTY, FO_FULL = 0, 1, 2, 3
FO_EINVAL, FO_ENOMEM, FO_EHIP, FO_ESTATE = -1, -2, -3, -4
FO_BUF_PARAMS, FO_BUF_GRADS, FO_BUF_LOGITS, FO_BUF_LOSS, FO_BUF_MOMENTUM = range(5)

EXPORTS = [
    "fo_config_param_count", "fo_config_num_classes", "fo_model_create", "fo_model_destroy",
    "fo_server_step", "fo_model_steps", "fo_model_buffer_size", "fo_model_read", "fo_model_write",
    "fo_async_aggregate", "fo_set_stream", "fo_set_max_delay", "fo_queues_create", "fo_queues_destroy",
    "fo_queues_push", "fo_queues_push_model", "fo_pick_device", "fo_queues_in_service",
    "fo_queues_release", "fo_aggregate_pending", "fo_aggregate_pending_all", "fo_queues_stats",
    "fo_queues_counters", "fo_queues_add_device", "fo_last_error", "fo_profile_enable", "fo_profile_read",
    "fo_set_graph_mode", "fo_gemm_bf16", "fo_conv2d_bf16", "fo_gemm_bf16_noalloc", "fo_queues_push_batch",
    "fo_queues_push_model_batch", "fo_device_step", "fo_queues_set_policy", "fo_queues_set_device_active",
    "fo_queues_sender_status", "fo_queues_log_enable", "fo_queues_log_read", "fo_pipeline_run",
    "fo_net_units", "fo_select_split", "fo_aux_network",
]
FO_NET_VGG5, FO_NET_MOBILENETV3_LARGE, FO_NET_TRANSFORMER6, FO_NET_TRANSFORMER12, FO_NET_VGG16 = range(1, 6)
FO_SCHED_COUNTER, FO_SCHED_FIFO = 0, 1
FO_EV_PUSH, FO_EV_MODEL, FO_EV_PICK, FO_EV_RELEASE, FO_EV_AGG, FO_EV_LEAVE, FO_EV_JOIN = range(1, 8)
FO_LAYOUT_ROW_K, FO_LAYOUT_K_ROW = 0, 1


class FoError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"fedoptima status {status}: {msg}")
        self.status = status


class fo_vec(C.Structure):
    _fields_ = [("ptr", C.c_void_p), ("n", C.c_int64)]


class fo_acts(C.Structure):
    _fields_ = [("x", C.c_void_p), ("lengths", C.c_void_p), ("batch", C.c_int32)]


class fo_kernel_stat(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("launches", C.c_int64), ("ms", C.c_double), ("flops", C.c_double),
                ("mfma_flops", C.c_double)]


class fo_queue_stats(C.Structure):
    _fields_ = [("K", C.c_int32), ("n_slots", C.c_int64), ("omega", C.c_int64), ("queued", C.c_int64),
                ("in_service", C.c_int64), ("models_pending", C.c_int64), ("admitted", C.c_int64),
                ("refused", C.c_int64), ("picks", C.c_int64), ("peak_queued", C.c_int64),
                ("version", C.c_int64), ("turn_on_signals", C.c_int64), ("active_devices", C.c_int32),
                ("policy", C.c_int32)]


class fo_unit(C.Structure):
    _fields_ = [("kind", C.c_int32), ("k", C.c_int32), ("stride", C.c_int32), ("c_in", C.c_int32),
                ("c_out", C.c_int32), ("h_out", C.c_int32), ("w_out", C.c_int32), ("expand", C.c_int32),
                ("heads", C.c_int32), ("hidden", C.c_int32), ("norm", C.c_int32), ("se", C.c_int32),
                ("params", C.c_int64), ("fwd_flops", C.c_double), ("out_elems", C.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class fo_pipeline_config(C.Structure):
    _fields_ = [("seconds", C.c_double), ("iter_seconds", C.c_void_p), ("H", C.c_int32), ("p_drop", C.c_double),
                ("interval_seconds", C.c_double), ("slow_max", C.c_double), ("seed", C.c_uint64),
                ("bank_x", C.c_void_p), ("bank_labels", C.c_void_p), ("bank_lengths", C.c_void_p),
                ("bank_n", C.c_int32), ("local_bank", C.c_void_p), ("n_local", C.c_int32), ("alpha", C.c_float),
                ("max_inflight", C.c_int32)]


class fo_pipeline_stats(C.Structure):
    _fields_ = [("wall_seconds", C.c_double), ("idle_seconds", C.c_double), ("steps", C.c_int64),
                ("samples", C.c_int64), ("aggregations", C.c_int64), ("skipped", C.c_int64), ("sent", C.c_int64),
                ("not_sent", C.c_int64), ("models_sent", C.c_int64), ("leaves", C.c_int64), ("rejoins", C.c_int64),
                ("device_iterations", C.c_int64)]


_lib = None


def lib():
    """Loads the library (raises if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2504_13850_amd.build.build()")
        # One HIP runtime per process: torch ships its own copy of the runtime
        # under the same soname, so loading torch first binds the library to it
        # and torch's streams and device pointers are valid in the library.
        import torch  # noqa: F401
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_float
        sig = {
            "fo_config_param_count": (i64, [i32]),
            "fo_config_num_classes": (i32, [i32]),
            "fo_model_create": (C.c_int, [i32, i32, vp, i64, vp, C.POINTER(vp)]),
            "fo_model_destroy": (None, [vp]),
            "fo_server_step": (C.c_int, [vp, C.POINTER(fo_acts), vp, i32]),
            "fo_device_step": (C.c_int, [vp, vp, vp, i32, vp]),
            "fo_model_steps": (i64, [vp, i32]),
            "fo_model_buffer_size": (i64, [vp, i32]),
            "fo_model_read": (C.c_int, [vp, i32, vp, i64]),
            "fo_model_write": (C.c_int, [vp, i32, vp, i64]),
            "fo_async_aggregate": (C.c_int, [C.POINTER(fo_vec), C.POINTER(fo_vec), f32, i32]),
            "fo_set_stream": (C.c_int, [vp]),
            "fo_set_max_delay": (C.c_int, [i64]),
            "fo_queues_create": (C.c_int, [i32, i64, i32, i32, i64, vp, C.POINTER(vp)]),
            "fo_queues_destroy": (None, [vp]),
            "fo_queues_push": (C.c_int, [vp, i32, vp, vp, vp, i32]),
            "fo_queues_push_model": (C.c_int, [vp, i32, vp, i64, i64]),
            "fo_queues_push_batch": (C.c_int, [vp, i32, vp, vp, vp, vp, vp]),
            "fo_queues_push_model_batch": (C.c_int, [vp, i32, vp, vp, i64, vp]),
            "fo_pick_device": (i32, [vp]),
            "fo_queues_in_service": (C.c_int, [vp, C.POINTER(fo_acts), C.POINTER(vp), C.POINTER(i64),
                                               C.POINTER(i64)]),
            "fo_queues_release": (C.c_int, [vp]),
            "fo_aggregate_pending": (C.c_int, [vp, C.POINTER(fo_vec), f32, C.POINTER(i32), C.POINTER(i64)]),
            "fo_aggregate_pending_all": (C.c_int, [vp, C.POINTER(fo_vec), f32, C.POINTER(i32), C.POINTER(i32)]),
            "fo_queues_stats": (C.c_int, [vp, C.POINTER(fo_queue_stats)]),
            "fo_queues_counters": (C.c_int, [vp, vp, i32]),
            "fo_queues_add_device": (i32, [vp]),
            "fo_queues_set_policy": (C.c_int, [vp, i32]),
            "fo_queues_set_device_active": (C.c_int, [vp, i32, i32]),
            "fo_queues_sender_status": (i32, [vp, i32]),
            "fo_queues_log_enable": (C.c_int, [vp, i64]),
            "fo_queues_log_read": (C.c_int, [vp, vp, i64, C.POINTER(i64)]),
            "fo_net_units": (i32, [i32, i32, i32, C.POINTER(fo_unit), i32]),
            "fo_select_split": (C.c_int, [C.POINTER(fo_unit), i32, i32, i32, i32, vp, vp, vp, C.POINTER(i32)]),
            "fo_aux_network": (i32, [C.POINTER(fo_unit), i32, i32, i32, C.POINTER(fo_unit), i32]),
            "fo_pipeline_run": (C.c_int, [vp, vp, C.POINTER(fo_vec), C.POINTER(fo_pipeline_config),
                                          C.POINTER(fo_pipeline_stats)]),
            "fo_last_error": (C.c_char_p, []),
            "fo_profile_enable": (C.c_int, [i32]),
            "fo_set_graph_mode": (C.c_int, [i32]),
            "fo_profile_read": (i32, [C.POINTER(fo_kernel_stat), i32]),
            "fo_gemm_bf16": (C.c_int, [i32, i32, i32, i32, vp, vp, i64, i32, vp, vp, i64, vp, i64, i32, vp, vp]),
            "fo_conv2d_bf16": (C.c_int, [i32, i32, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, i32,
                                         vp, vp]),
            "fo_gemm_bf16_noalloc": (C.c_int, [i32, i32, i32, i32, vp, vp, i64, i32, vp, vp, i64, vp, i64, i32,
                                               vp]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def last_error() -> str:
    return lib().fo_last_error().decode()


def _check(st, allowed=(FO_OK,)):
    if st not in allowed:
        raise FoError(st, last_error())
    return st


def _dptr(t):
    """Device (or host) address of a torch tensor / numpy array / int / None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------------ configs
def fo_config_param_count(cid: int) -> int:
    return lib().fo_config_param_count(cid)


def fo_config_num_classes(cid: int) -> int:
    return lib().fo_config_num_classes(cid)


# ------------------------------------------------------------------ model
def fo_model_create(cid: int, max_batch: int, host_init: np.ndarray, stream=None):
    h = np.ascontiguousarray(host_init, dtype=np.float32)
    out = C.c_void_p()
    _check(lib().fo_model_create(cid, max_batch, h.ctypes.data, h.size, _stream(stream), C.byref(out)))
    return out


def fo_model_destroy(model):
    lib().fo_model_destroy(model)


def make_acts(x, lengths=None, batch=None) -> fo_acts:
    b = batch if batch is not None else int(x.shape[0])
    return fo_acts(_dptr(x), _dptr(lengths), b)


def fo_server_step(model, acts, labels, device_id: int):
    if not isinstance(acts, fo_acts):
        acts = make_acts(*acts) if isinstance(acts, tuple) else make_acts(acts)
    return _check(lib().fo_server_step(model, C.byref(acts), _dptr(labels), device_id))


def fo_device_step(model, x, labels, batch: int, acts_out):
    return _check(lib().fo_device_step(model, _dptr(x), _dptr(labels), int(batch), _dptr(acts_out)))


def fo_set_graph_mode(enable: bool):
    _check(lib().fo_set_graph_mode(1 if enable else 0))


def fo_model_steps(model, device_id: int = -1) -> int:
    return lib().fo_model_steps(model, device_id)


def fo_model_read(model, which: int) -> np.ndarray:
    n = lib().fo_model_buffer_size(model, which)
    if n < 0:
        raise FoError(FO_EINVAL, f"model has no buffer {which}")
    out = np.empty(n, np.float32)
    _check(lib().fo_model_read(model, which, out.ctypes.data, n))
    return out


def fo_model_write(model, which: int, host: np.ndarray):
    h = np.ascontiguousarray(host, dtype=np.float32)
    _check(lib().fo_model_write(model, which, h.ctypes.data, h.size))


# ------------------------------------------------------------------ aggregation
def fo_async_aggregate(global_, local, alpha: float, staleness: int) -> int:
    g = fo_vec(_dptr(global_), int(global_.numel()))
    l = fo_vec(_dptr(local), int(local.numel()))
    return _check(lib().fo_async_aggregate(C.byref(g), C.byref(l), float(alpha), int(staleness)),
                  (FO_OK, FO_SKIPPED))


def fo_set_stream(stream):
    _check(lib().fo_set_stream(_stream(stream)))


def fo_set_max_delay(D: int):
    _check(lib().fo_set_max_delay(int(D)))


# ------------------------------------------------------------------ scheduler + pool
def fo_queues_create(K: int, slot_bytes: int, batch: int, with_lengths: bool, n_slots: int, stream=None):
    out = C.c_void_p()
    _check(lib().fo_queues_create(K, slot_bytes, batch, int(bool(with_lengths)), n_slots, _stream(stream),
                                  C.byref(out)))
    return out


def fo_queues_destroy(q):
    lib().fo_queues_destroy(q)


def fo_queues_push(q, k: int, x=None, labels=None, lengths=None, on_host: bool = False) -> int:
    return _check(lib().fo_queues_push(q, k, _dptr(x), _dptr(labels), _dptr(lengths), int(on_host)),
                  (FO_OK, FO_FULL))


def fo_queues_push_batch(q, k, x_ptrs=None, label_ptrs=None, length_ptrs=None) -> np.ndarray:
    """n arrivals: k, x_ptrs, label_ptrs, length_ptrs are sequences of device ids and
    raw device addresses (ints).  Returns the per-entry status (FO_OK / FO_FULL)."""
    kk = np.ascontiguousarray(k, dtype=np.int32)
    n = int(kk.size)
    arr = lambda v: None if v is None else np.ascontiguousarray(v, dtype=np.uint64)
    xs, ls, ns = arr(x_ptrs), arr(label_ptrs), arr(length_ptrs)
    st = np.zeros(n, np.int32)
    _check(lib().fo_queues_push_batch(q, n, kk.ctypes.data, _dptr(xs), _dptr(ls), _dptr(ns), st.ctypes.data))
    return st


def fo_queues_push_model_batch(q, k, local_ptrs, length: int, t_k):
    kk = np.ascontiguousarray(k, dtype=np.int32)
    ps = np.ascontiguousarray(local_ptrs, dtype=np.uint64)
    tt = np.ascontiguousarray(t_k, dtype=np.int64)
    _check(lib().fo_queues_push_model_batch(q, int(kk.size), kk.ctypes.data, ps.ctypes.data, int(length),
                                            tt.ctypes.data))


def fo_queues_push_model(q, k: int, local, t_k: int):
    n = 0 if local is None else int(local.numel())
    _check(lib().fo_queues_push_model(q, k, _dptr(local), n, int(t_k)))


def fo_pick_device(q) -> int:
    r = lib().fo_pick_device(q)
    if r == -3:
        raise FoError(FO_ESTATE, last_error())
    return r


def fo_queues_in_service(q):
    acts = fo_acts()
    lab = C.c_void_p()
    seq = C.c_int64()
    slot = C.c_int64()
    _check(lib().fo_queues_in_service(q, C.byref(acts), C.byref(lab), C.byref(seq), C.byref(slot)))
    return acts, lab.value, seq.value, slot.value


def fo_queues_release(q):
    _check(lib().fo_queues_release(q))


def fo_aggregate_pending(q, global_, alpha: float):
    g = fo_vec(_dptr(global_), int(global_.numel()))
    k = C.c_int32()
    s = C.c_int64()
    st = _check(lib().fo_aggregate_pending(q, C.byref(g), float(alpha), C.byref(k), C.byref(s)),
                (FO_OK, FO_SKIPPED, FO_EMPTY))
    return st, k.value, s.value


def fo_aggregate_pending_all(q, global_, alpha: float):
    g = fo_vec(_dptr(global_), int(global_.numel()))
    a = C.c_int32()
    s = C.c_int32()
    _check(lib().fo_aggregate_pending_all(q, C.byref(g), float(alpha), C.byref(a), C.byref(s)))
    return a.value, s.value


def fo_queues_stats(q) -> fo_queue_stats:
    st = fo_queue_stats()
    _check(lib().fo_queues_stats(q, C.byref(st)))
    return st


def fo_queues_counters(q, K: int) -> list:
    out = np.zeros(K, np.int64)
    _check(lib().fo_queues_counters(q, out.ctypes.data, K))
    return out.tolist()


def fo_queues_add_device(q) -> int:
    r = lib().fo_queues_add_device(q)
    if r < 0:
        raise FoError(FO_EINVAL, last_error())
    return r


def fo_queues_set_policy(q, policy: int):
    _check(lib().fo_queues_set_policy(q, policy))


def fo_queues_set_device_active(q, k: int, active: bool):
    _check(lib().fo_queues_set_device_active(q, k, 1 if active else 0))


def fo_queues_sender_status(q, k: int) -> int:
    r = lib().fo_queues_sender_status(q, k)
    if r < 0:
        raise FoError(FO_EINVAL, last_error())
    return r


def fo_queues_log_enable(q, max_events: int):
    _check(lib().fo_queues_log_enable(q, max_events))


def fo_queues_log_read(q, max_events: int) -> np.ndarray:
    """The pool's event record as an int64 array [n][4] (type, device, a, b)."""
    out = np.zeros((max(max_events, 0), 4), np.int64)
    n = C.c_int64(0)
    _check(lib().fo_queues_log_read(q, out.ctypes.data, max_events, C.byref(n)))
    return out[:min(n.value, max_events)]


def fo_pipeline_run(q, model, global_vec, cfg: dict) -> fo_pipeline_stats:
    """Runs the concurrent pipeline; cfg holds the fo_pipeline_config fields
    (iter_seconds as a sequence of floats, device buffers as tensors)."""
    iters = np.ascontiguousarray(cfg["iter_seconds"], np.float64)
    c = fo_pipeline_config()
    c.seconds = cfg["seconds"]
    c.iter_seconds = iters.ctypes.data
    c.H = cfg["H"]
    c.p_drop = cfg.get("p_drop", 0.0)
    c.interval_seconds = cfg.get("interval_seconds", 1.0)
    c.slow_max = cfg.get("slow_max", 1.0)
    c.seed = cfg.get("seed", 0)
    c.bank_x = _dptr(cfg["bank_x"])
    c.bank_labels = _dptr(cfg["bank_labels"])
    c.bank_lengths = _dptr(cfg.get("bank_lengths"))
    c.bank_n = cfg["bank_n"]
    c.local_bank = _dptr(cfg["local_bank"])
    c.n_local = cfg["n_local"]
    c.alpha = cfg.get("alpha", 0.5)
    c.max_inflight = cfg.get("max_inflight", 2)
    g = fo_vec(_dptr(global_vec), int(global_vec.numel()))
    st = fo_pipeline_stats()
    _check(lib().fo_pipeline_run(q, model, C.byref(g), C.byref(c), C.byref(st)))
    return st


# ------------------------------------------------------------------ pre-processor
def fo_net_units(net: int, classes: int, in_hw: int):
    """The unit table of a network, as a ctypes array of fo_unit."""
    n = lib().fo_net_units(net, classes, in_hw, None, 0)
    if n < 0:
        raise FoError(FO_EINVAL, last_error())
    arr = (fo_unit * n)()
    lib().fo_net_units(net, classes, in_hw, arr, n)
    return arr


def fo_select_split(units, batch: int, bytes_per_value: int, flops_per_s, bytes_per_s):
    """Returns (split l, per-split costs)."""
    o = np.ascontiguousarray(flops_per_s, np.float64)
    b = np.ascontiguousarray(bytes_per_s, np.float64)
    costs = np.zeros(len(units), np.float64)
    l = C.c_int32()
    _check(lib().fo_select_split(units, len(units), batch, bytes_per_value, len(o), o.ctypes.data, b.ctypes.data,
                                 costs.ctypes.data, C.byref(l)))
    return l.value, costs


def fo_aux_network(units, split: int, classes: int):
    n = lib().fo_aux_network(units, len(units), split, classes, None, 0)
    if n < 0:
        raise FoError(FO_EINVAL, last_error())
    arr = (fo_unit * n)()
    lib().fo_aux_network(units, len(units), split, classes, arr, n)
    return arr


# ------------------------------------------------------------------ instrumentation
def fo_profile_enable(max_launches: int):
    _check(lib().fo_profile_enable(int(max_launches)))


def fo_profile_read(max_kernels: int = 64) -> list:
    """[{name, launches, ms, flops, mfma_flops}] for the launches recorded since enabling."""
    buf = (fo_kernel_stat * max_kernels)()
    n = lib().fo_profile_read(buf, max_kernels)
    if n < 0:
        raise FoError(n, last_error())
    return [dict(name=buf[i].name.decode(), launches=buf[i].launches, ms=buf[i].ms, flops=buf[i].flops,
                 mfma_flops=buf[i].mfma_flops) for i in range(min(n, max_kernels))]


# ------------------------------------------------------------------ kernel-level entry points
def fo_gemm_bf16(M, N, K, a_layout, A, A_lo, lda, b_layout, B, B_lo, ldb, C, ldc, splits=1, workspace=None,
                 stream=None):
    _check(lib().fo_gemm_bf16(M, N, K, a_layout, _dptr(A), _dptr(A_lo), lda, b_layout, _dptr(B), _dptr(B_lo), ldb,
                              _dptr(C), ldc, splits, _dptr(workspace), _stream(stream)))


def fo_gemm_bf16_noalloc(M, N, K, a_layout, A, A_lo, lda, b_layout, B, B_lo, ldb, C, ldc, splits=1,
                         stream=None):
    _check(lib().fo_gemm_bf16_noalloc(M, N, K, a_layout, _dptr(A), _dptr(A_lo), lda, b_layout, _dptr(B),
                                      _dptr(B_lo), ldb, _dptr(C), ldc, splits, _stream(stream)))


def fo_conv2d_bf16(pass_, Bn, H, W, Ci, Co, k, stride, pad, inp, inp_lo, in2, w, w_lo, out, splits=1,
                   workspace=None, stream=None):
    _check(lib().fo_conv2d_bf16(pass_, Bn, H, W, Ci, Co, k, stride, pad, _dptr(inp), _dptr(inp_lo), _dptr(in2),
                                _dptr(w), _dptr(w_lo), _dptr(out), splits, _dptr(workspace), _stream(stream)))
