"""ctypes binding of libasgd.so (include/asgd.h): same names, argument
marshalling only.  Every computation runs in the HIP library; a missing or
unloadable library raises instead of falling back to anything else.

Device buffers are passed as raw pointers (``tensor.data_ptr()``) and HIP
streams as integers (``torch.cuda.current_stream().cuda_stream``) or None.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_double, c_float, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libasgd.so")

ASGD_OK, ASGD_EINVAL, ASGD_ERANGE, ASGD_ENOMEM, ASGD_EHIP, ASGD_ESTATE = 0, -1, -2, -3, -4, -5
ASGD_VALIDATE = 0x1
ASGD_UNFUSED_OUTPUT = 0x2
ASGD_PARAM_W1, ASGD_PARAM_B1, ASGD_PARAM_W2, ASGD_PARAM_B2, ASGD_PARAM_WH, ASGD_PARAM_BH = 0, 1, 2, 3, 4, 5
ASGD_WEIGHTS_ALG2, ASGD_WEIGHTS_SAMPLES, ASGD_WEIGHTS_UNIFORM = 0, 1, 2
ASGD_DISPATCH_DYNAMIC, ASGD_DISPATCH_STATIC = 0, 1
HIDDEN = 128

# Every symbol include/asgd.h declares (checked by the CPU tests).
EXPORTS = (
    "asgd_model_init", "asgd_model_free", "asgd_model_set_stream", "asgd_model_copy",
    "asgd_model_num_params", "asgd_model_get_params", "asgd_model_set_params",
    "asgd_train_step", "asgd_model_last_loss", "asgd_predict_topk", "asgd_merge",
    "asgd_model_l2_per_param", "asgd_models_l2_per_param", "asgd_models_l2_per_param_noalloc",
    "asgd_merge_weights", "asgd_scale_batches",
    "asgd_debug_forward", "asgd_debug_touched_rows", "asgd_libsvm_scan", "asgd_libsvm_read",
    "asgd_model_set_timing",
    "asgd_model_get_timing", "asgd_elastic_create", "asgd_elastic_free", "asgd_elastic_round",
    "asgd_elastic_model", "asgd_last_error",
)
ASGD_CLOCK_TIMED, ASGD_CLOCK_VIRTUAL = 0, 1

# Kernel groups of asgd_model_get_timing.
KERNELS = ("gather", "sort", "out_fwd", "out_combine", "hidden", "out_bwd", "w1_update", "merge", "labels",
           "dense_fwd", "dense_bwd", "logits", "softmax", "dh")


class AsgdError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where} failed with status {status}: {msg}")
        self.status = status


class asgd_config(ctypes.Structure):
    _fields_ = [("n_features", c_int32), ("n_labels", c_int32), ("hidden", c_int32),
                ("extra_hidden_layers", c_int32), ("max_batch", c_int32), ("max_nnz", c_int32), ("max_label_nnz", c_int32),
                ("gemm_bf16", c_int32), ("flags", c_uint32)]


class asgd_csr(ctypes.Structure):
    _fields_ = [("n_rows", c_int32), ("n_cols", c_int32), ("nnz", c_int32),
                ("indptr", c_void_p), ("indices", c_void_p), ("values", c_void_p)]


class asgd_elastic_config(ctypes.Structure):
    _fields_ = [("n_replicas", c_int32), ("b_min", c_int32), ("b_max", c_int32), ("beta", c_double),
                ("lr", c_float), ("gamma", c_float), ("weight_mode", c_int32), ("perturb", c_int32),
                ("pert_thr", c_double), ("delta", c_double), ("megabatch", c_int64), ("dispatch", c_int32),
                ("clock", c_int32),
                ("c0", c_double), ("c1", c_double), ("c2", c_double), ("slow", c_double * 16)]


class asgd_libsvm_info(ctypes.Structure):
    _fields_ = [("n_rows", c_int64), ("nnz", c_int64), ("label_nnz", c_int64), ("n_features", c_int64),
                ("n_labels", c_int64), ("header_rows", c_int64)]


class asgd_elastic_log(ctypes.Structure):
    _fields_ = [("n_dispatch", c_int32), ("max_dispatch", c_int32), ("replica", POINTER(c_int32)),
                ("row0", POINTER(c_int32)), ("row1", POINTER(c_int32)), ("u", c_int32 * 16),
                ("samples", c_int64 * 16), ("b_used", c_int32 * 16), ("lr_used", c_float * 16),
                ("alpha", c_float * 16), ("l2_per_param", c_double * 16), ("b_next", c_int32 * 16),
                ("lr_next", c_float * 16), ("cursor", c_int32)]


_lib = None


def _declare(lib):
    P = c_void_p
    sig = {
        "asgd_model_init": (c_int32, [POINTER(c_void_p), POINTER(asgd_config), c_uint64, P]),
        "asgd_model_free": (c_int32, [P]),
        "asgd_model_set_stream": (c_int32, [P, P]),
        "asgd_model_copy": (c_int32, [P, P]),
        "asgd_model_num_params": (c_int32, [P, POINTER(c_int64)]),
        "asgd_model_get_params": (c_int32, [P, c_int32, P, c_size_t]),
        "asgd_model_set_params": (c_int32, [P, c_int32, P, c_size_t]),
        "asgd_train_step": (c_int32, [P, POINTER(asgd_csr), POINTER(asgd_csr), c_float, POINTER(c_float)]),
        "asgd_model_last_loss": (c_int32, [P, POINTER(c_float)]),
        "asgd_predict_topk": (c_int32, [P, POINTER(asgd_csr), c_int32, P, P]),
        "asgd_merge": (c_int32, [P, P, POINTER(c_void_p), POINTER(c_float), c_int32, c_float, c_int32]),
        "asgd_model_l2_per_param": (c_int32, [P, POINTER(c_double)]),
        "asgd_models_l2_per_param": (c_int32, [POINTER(c_void_p), c_int32, POINTER(c_double)]),
        "asgd_models_l2_per_param_noalloc": (c_int32, [POINTER(c_void_p), c_int32, P]),
        "asgd_merge_weights": (c_int32, [c_int32, POINTER(c_int32), POINTER(c_int32), POINTER(c_int64),
                                         c_int32, POINTER(c_double), c_double, c_double, POINTER(c_float)]),
        "asgd_scale_batches": (c_int32, [c_int32, POINTER(c_int32), POINTER(c_int32), POINTER(c_float),
                                         c_int32, c_int32, c_double]),
        "asgd_debug_forward": (c_int32, [P, POINTER(asgd_csr), POINTER(asgd_csr), P, P, P, P]),
        "asgd_debug_touched_rows": (c_int32, [P, POINTER(asgd_csr), P, POINTER(c_int32)]),
        "asgd_libsvm_scan": (c_int32, [ctypes.c_char_p, c_int32, POINTER(asgd_libsvm_info)]),
        "asgd_libsvm_read": (c_int32, [ctypes.c_char_p, c_int32, POINTER(asgd_libsvm_info), P, P, P, P, P]),
        "asgd_model_set_timing": (c_int32, [P, c_int32]),
        "asgd_model_get_timing": (c_int32, [P, c_int32, POINTER(c_double), POINTER(c_int64)]),
        "asgd_elastic_create": (c_int32, [POINTER(c_void_p), POINTER(asgd_elastic_config),
                                          POINTER(asgd_config), c_uint64, POINTER(c_void_p), P]),
        "asgd_elastic_free": (c_int32, [P]),
        "asgd_elastic_round": (c_int32, [P, POINTER(asgd_csr), POINTER(asgd_csr), P, P,
                                         POINTER(asgd_elastic_log)]),
        "asgd_elastic_model": (c_int32, [P, c_int32, POINTER(c_void_p)]),
        "asgd_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args


def library_path() -> str:
    return LIB_PATH


def load(build_if_missing: bool = True):
    """Load the in-tree libasgd.so (building it first only if it does not exist)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        if not build_if_missing:
            raise RuntimeError(f"HIP library {LIB_PATH} is not built")
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(LIB_PATH)
    _declare(lib)
    _lib = lib
    return lib


def _check(status: int, where: str):
    if status != ASGD_OK:
        raise AsgdError(status, where, load().asgd_last_error().decode())


def _ptr(t) -> int:
    """Raw device/host address of a tensor, an int, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(s) -> int:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


# ------------------------------------------------------------------ entry points
def asgd_last_error() -> str:
    return load().asgd_last_error().decode()


def asgd_model_init(n_features: int, n_labels: int, max_batch: int, max_nnz: int, max_label_nnz: int,
                    gemm_bf16: bool = True, seed: int = 0, stream=None, flags: int = 0,
                    hidden: int = HIDDEN, extra_hidden_layers: int = 0) -> int:
    cfg = asgd_config(n_features=n_features, n_labels=n_labels, hidden=hidden,
                      extra_hidden_layers=extra_hidden_layers, max_batch=max_batch, max_nnz=max_nnz,
                      max_label_nnz=max_label_nnz, gemm_bf16=1 if gemm_bf16 else 0, flags=flags)
    h = c_void_p()
    _check(load().asgd_model_init(byref(h), byref(cfg), c_uint64(seed & (2 ** 64 - 1)), _stream(stream)),
           "asgd_model_init")
    return h.value


def asgd_model_free(m: int):
    _check(load().asgd_model_free(m), "asgd_model_free")


def asgd_model_set_stream(m: int, stream):
    _check(load().asgd_model_set_stream(m, _stream(stream)), "asgd_model_set_stream")


def asgd_model_copy(dst: int, src: int):
    _check(load().asgd_model_copy(dst, src), "asgd_model_copy")


def asgd_model_num_params(m: int) -> int:
    v = c_int64()
    _check(load().asgd_model_num_params(m, byref(v)), "asgd_model_num_params")
    return v.value


def _param_shape(which: int, F: int, L: int):
    return {ASGD_PARAM_W1: (F, HIDDEN), ASGD_PARAM_B1: (HIDDEN,), ASGD_PARAM_W2: (L, HIDDEN),
            ASGD_PARAM_B2: (L,), ASGD_PARAM_WH: (HIDDEN, HIDDEN), ASGD_PARAM_BH: (HIDDEN,)}[which]


def asgd_model_get_params(m: int, which: int, shape) -> np.ndarray:
    out = np.empty(shape, np.float32)
    _check(load().asgd_model_get_params(m, which, out.ctypes.data, out.nbytes), "asgd_model_get_params")
    return out


def asgd_model_set_params(m: int, which: int, host: np.ndarray):
    a = np.ascontiguousarray(host, np.float32)
    _check(load().asgd_model_set_params(m, which, a.ctypes.data, a.nbytes), "asgd_model_set_params")


def asgd_train_step(m: int, x: asgd_csr, y: asgd_csr, lr: float, want_loss: bool = False):
    if want_loss:
        v = c_float()
        _check(load().asgd_train_step(m, byref(x), byref(y), c_float(lr), byref(v)), "asgd_train_step")
        return v.value
    _check(load().asgd_train_step(m, byref(x), byref(y), c_float(lr), None), "asgd_train_step")
    return None


def asgd_model_last_loss(m: int) -> float:
    v = c_float()
    _check(load().asgd_model_last_loss(m, byref(v)), "asgd_model_last_loss")
    return v.value


def asgd_predict_topk(m: int, x: asgd_csr, k: int, ids_dev, scores_dev=None):
    _check(load().asgd_predict_topk(m, byref(x), k, _ptr(ids_dev), _ptr(scores_dev)), "asgd_predict_topk")


def asgd_merge(global_m: int, prev_m, replicas, weights, gamma: float, broadcast: bool):
    n = len(replicas)
    arr = (c_void_p * n)(*replicas)
    w = (c_float * n)(*[float(v) for v in weights])
    _check(load().asgd_merge(global_m, prev_m, arr, w, n, c_float(gamma), 1 if broadcast else 0),
           "asgd_merge")


def asgd_model_l2_per_param(m: int) -> float:
    v = c_double()
    _check(load().asgd_model_l2_per_param(m, byref(v)), "asgd_model_l2_per_param")
    return v.value


def asgd_models_l2_per_param(models) -> list:
    n = len(models)
    arr = (c_void_p * n)(*models)
    out = (c_double * n)()
    _check(load().asgd_models_l2_per_param(arr, n, out), "asgd_models_l2_per_param")
    return list(out)


def asgd_models_l2_per_param_noalloc(models, out_dev):
    """Asynchronous; out_dev: device float64 [len(models)] (e.g. a torch tensor)."""
    n = len(models)
    arr = (c_void_p * n)(*models)
    _check(load().asgd_models_l2_per_param_noalloc(arr, n, _ptr(out_dev)), "asgd_models_l2_per_param_noalloc")


def asgd_merge_weights(u, b, samples=None, mode: int = ASGD_WEIGHTS_ALG2, l2_per_param=None,
                       pert_thr: float = 0.1, delta: float = 0.1) -> np.ndarray:
    n = len(u)
    U = (c_int32 * n)(*[int(v) for v in u])
    Bv = (c_int32 * n)(*[int(v) for v in b])
    S = (c_int64 * n)(*[int(v) for v in samples]) if samples is not None else None
    G = (c_double * n)(*[float(v) for v in l2_per_param]) if l2_per_param is not None else None
    out = (c_float * n)()
    _check(load().asgd_merge_weights(n, U, Bv, S, mode, G, c_double(pert_thr), c_double(delta), out),
           "asgd_merge_weights")
    return np.array(out[:], np.float32)


def asgd_scale_batches(u, b, lr, b_min: int, b_max: int, beta: float):
    n = len(u)
    U = (c_int32 * n)(*[int(v) for v in u])
    Bv = (c_int32 * n)(*[int(v) for v in b])
    LR = (c_float * n)(*[float(v) for v in lr])
    _check(load().asgd_scale_batches(n, U, Bv, LR, b_min, b_max, c_double(beta)), "asgd_scale_batches")
    return list(Bv[:]), [float(v) for v in LR[:]]


def asgd_debug_forward(m: int, x: asgd_csr, y, a1_dev=None, z_dev=None, lse_dev=None, loss_rows_dev=None):
    _check(load().asgd_debug_forward(m, byref(x), byref(y) if y is not None else None,
                                     _ptr(a1_dev), _ptr(z_dev), _ptr(lse_dev), _ptr(loss_rows_dev)),
           "asgd_debug_forward")


def asgd_debug_touched_rows(m: int, x: asgd_csr, ids_dev) -> int:
    c = c_int32()
    _check(load().asgd_debug_touched_rows(m, byref(x), _ptr(ids_dev), byref(c)), "asgd_debug_touched_rows")
    return c.value


def asgd_libsvm_scan(path: str, one_based: bool = False) -> asgd_libsvm_info:
    info = asgd_libsvm_info()
    _check(load().asgd_libsvm_scan(os.fsencode(path), 1 if one_based else 0, byref(info)), "asgd_libsvm_scan")
    return info


def asgd_libsvm_read(path: str, info: asgd_libsvm_info, one_based: bool = False):
    """(indptr, indices, values, label_indptr, label_indices) as host numpy arrays."""
    ip = np.zeros(info.n_rows + 1, np.int64)
    ix = np.zeros(max(info.nnz, 1), np.int32)
    va = np.zeros(max(info.nnz, 1), np.float32)
    lp = np.zeros(info.n_rows + 1, np.int64)
    lx = np.zeros(max(info.label_nnz, 1), np.int32)
    _check(load().asgd_libsvm_read(os.fsencode(path), 1 if one_based else 0, byref(info), ip.ctypes.data,
                                   ix.ctypes.data, va.ctypes.data, lp.ctypes.data, lx.ctypes.data),
           "asgd_libsvm_read")
    return ip, ix[:info.nnz], va[:info.nnz], lp, lx[:info.label_nnz]


def asgd_model_set_timing(m: int, enable: bool):
    _check(load().asgd_model_set_timing(m, 1 if enable else 0), "asgd_model_set_timing")


def asgd_model_get_timing(m: int, kernel: int):
    """(total milliseconds, launches) of a kernel group since the last read."""
    t, n = c_double(), c_int64()
    _check(load().asgd_model_get_timing(m, kernel, byref(t), byref(n)), "asgd_model_get_timing")
    return t.value, n.value


def asgd_elastic_create(cfg: asgd_elastic_config, model_cfg: asgd_config, seed: int, replica_streams,
                        global_stream) -> int:
    n = len(replica_streams)
    arr = (c_void_p * n)(*[_stream(s) for s in replica_streams])
    h = c_void_p()
    _check(load().asgd_elastic_create(byref(h), byref(cfg), byref(model_cfg), c_uint64(seed), arr,
                                      _stream(global_stream)), "asgd_elastic_create")
    return h.value


def asgd_elastic_free(e: int):
    _check(load().asgd_elastic_free(e), "asgd_elastic_free")


def asgd_elastic_round(e: int, x_all: asgd_csr, y_all: asgd_csr, x_indptr_host: np.ndarray,
                       y_indptr_host: np.ndarray, max_dispatch: int = 4096) -> dict:
    """One round; returns the round record as a dict of numpy arrays / lists."""
    xi = np.ascontiguousarray(x_indptr_host, np.int32)
    yi = np.ascontiguousarray(y_indptr_host, np.int32)
    rep = np.zeros(max_dispatch, np.int32)
    r0 = np.zeros(max_dispatch, np.int32)
    r1 = np.zeros(max_dispatch, np.int32)
    log = asgd_elastic_log()
    log.max_dispatch = max_dispatch
    log.replica = rep.ctypes.data_as(POINTER(c_int32))
    log.row0 = r0.ctypes.data_as(POINTER(c_int32))
    log.row1 = r1.ctypes.data_as(POINTER(c_int32))
    _check(load().asgd_elastic_round(e, byref(x_all), byref(y_all), xi.ctypes.data, yi.ctypes.data,
                                     byref(log)), "asgd_elastic_round")
    nd = log.n_dispatch
    if nd > max_dispatch:
        raise AsgdError(ASGD_ERANGE, "asgd_elastic_round", "dispatch log capacity exceeded")
    return dict(schedule=[(int(rep[i]), int(r0[i]), int(r1[i])) for i in range(nd)],
                u=list(log.u), samples=list(log.samples), b_used=list(log.b_used),
                lr_used=list(log.lr_used), alpha=np.array(log.alpha[:], np.float32),
                l2_per_param=list(log.l2_per_param), b_next=list(log.b_next),
                lr_next=list(log.lr_next), cursor=log.cursor)


def asgd_elastic_model(e: int, which: int) -> int:
    h = c_void_p()
    _check(load().asgd_elastic_model(e, which, byref(h)), "asgd_elastic_model")
    return h.value
