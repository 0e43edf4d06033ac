"""ctypes binding of librnnbkt.so (declared in include/rnnbkt.h).

Argument marshalling only: every computation runs in the library (host C++
for the planner and schedule, HIP kernels for the model).  Device buffers
are passed as torch tensors on the GPU, or as raw integer addresses; torch
is used for nothing but device memory and the current stream.

Loading fails loudly (``LibraryMissing``) when the library has not been
built; there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "librnnbkt.so")

OK = 0
EINVAL = -1
EUNSUPPORTED = -2
EHIP = -3

CELL_LSTM = 0
CELL_GRU = 1
CELL_LSTM_PEEPHOLE = 2
GEMM_FP32 = 0
GEMM_BF16 = 1


class LibraryMissing(RuntimeError):
    pass


class RnnbktError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"rnnbkt error {code}: {msg}")
        self.code = code


class ModelDesc(ctypes.Structure):
    _fields_ = [("cell", ctypes.c_int32), ("num_layers", ctypes.c_int32),
                ("input_dim", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("num_classes", ctypes.c_int32), ("bidirectional", ctypes.c_int32),
                ("gemm_dtype", ctypes.c_int32)]

    @classmethod
    def of(cls, cell, num_layers, input_dim, hidden, num_classes, bidirectional, gemm_dtype):
        return cls(int(cell), int(num_layers), int(input_dim), int(hidden), int(num_classes),
                   int(bidirectional), int(gemm_dtype))


_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_szp = ctypes.POINTER(ctypes.c_size_t)
_vp = ctypes.c_void_p
_descp = ctypes.POINTER(ModelDesc)

_SIGNATURES = {
    "rnnbkt_version": (ctypes.c_char_p, []),
    "rnnbkt_last_error": (ctypes.c_char_p, []),
    "rnnbkt_sync_check": (ctypes.c_int32, [_vp]),
    "rnnbkt_bucket_plan": (ctypes.c_int32, [_i32p, ctypes.c_int64, ctypes.c_int32, _i32p, _i32p,
                                            _i32p, _i64p]),
    "rnnbkt_epoch_schedule_ordered": (ctypes.c_int32, [_i32p, _i32p, ctypes.c_int64,
                                                       ctypes.c_int32, _u64p, ctypes.c_int32,
                                                       ctypes.c_int32, _u64p, _i64p, _i64p,
                                                       _i64p]),
    "rnnbkt_epoch_schedule": (ctypes.c_int32, [_i32p, _i32p, ctypes.c_int64, ctypes.c_int32,
                                               _u64p, ctypes.c_int32, _i64p, _i64p, _i64p]),
    "rnnbkt_param_count": (ctypes.c_int64, [_descp]),
    "rnnbkt_buffer_sizes": (ctypes.c_int32, [_descp, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_int64, _szp, _szp]),
    "rnnbkt_lstm_fwd": (ctypes.c_int32, [_descp, _vp, _vp, _vp, _i32p, ctypes.c_int32,
                                         ctypes.c_int32, _vp, ctypes.c_size_t, _vp,
                                         ctypes.c_size_t, _vp, _vp]),
    "rnnbkt_ctc_workspace_bytes": (ctypes.c_int32, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                    _szp]),
    "rnnbkt_lstm_fwd_ctc": (ctypes.c_int32, [_descp, _vp, _vp, _vp, _i32p, ctypes.c_int32, _i32p,
                                             ctypes.c_int32, ctypes.c_int32, _vp, ctypes.c_size_t,
                                             _vp, ctypes.c_size_t, _vp, ctypes.c_size_t, _vp,
                                             _vp]),
    "rnnbkt_lstm_bwd": (ctypes.c_int32, [_descp, _vp, _i32p, ctypes.c_int32, ctypes.c_int32,
                                         _vp, ctypes.c_size_t, _vp, ctypes.c_size_t, _vp, _vp]),
    "rnnbkt_lstm_bwd_noalloc": (ctypes.c_int32, [_descp, _vp, _i32p, ctypes.c_int32,
                                                 ctypes.c_int32, _vp, ctypes.c_size_t, _vp, _vp]),
    "rnnbkt_sgd_apply": (ctypes.c_int32, [_vp, _vp, ctypes.c_int64, ctypes.c_float, _vp]),
    "rnnbkt_epoch_aggregate": (ctypes.c_int32, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                                ctypes.c_int64, ctypes.c_void_p, ctypes.c_float,
                                                ctypes.c_void_p]),
    "rnnbkt_set_concurrency": (ctypes.c_int32, [ctypes.c_int32]),
    "rnnbkt_adadelta_apply": (ctypes.c_int32, [_vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_float,
                                               ctypes.c_float, ctypes.c_float, _vp]),
    "rnnbkt_top_hidden": (ctypes.c_int32, [_descp, _i32p, ctypes.c_int32, ctypes.c_int32, _vp,
                                           ctypes.c_size_t, _vp, _vp]),
    "rnnbkt_kernel_timer": (ctypes.c_int32, [ctypes.c_int32]),
    "rnnbkt_kernel_timer_read": (ctypes.c_int32, [ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                                                  _i64p, ctypes.POINTER(ctypes.c_double),
                                                  ctypes.POINTER(ctypes.c_double)]),
}

KERNEL_KINDS = {"step_fwd": 0, "step_bwd": 1, "gemm": 2, "xent": 3, "sgd": 4, "other": 5,
                "side": 6, "prepare": 7}
# Kinds whose time runs beside the recurrence rather than on the critical path.
OVERLAPPED_KINDS = ("side",)

_lib = None


def load():
    """Loads the in-tree library once; raises LibraryMissing if absent."""
    global _lib
    if _lib is not None:
        return _lib
    try:
        import torch  # noqa: F401  (its HIP runtime must be the one the library binds to)
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise LibraryMissing(
            f"{LIB_PATH} not found: build it with `python -m paper_1708_05604_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def exported_symbols():
    return list(_SIGNATURES)


def _check(code: int):
    if code != OK:
        raise RnnbktError(code, load().rnnbkt_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a: np.ndarray, typ):
    return a.ctypes.data_as(typ)


def _dev(t, dtype: Optional[str] = None) -> int:
    """Device address of a tensor (or an int address).  A tensor must be a
    contiguous GPU tensor of the expected element type."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("expected a GPU tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    if dtype is not None and str(t.dtype) != "torch." + dtype:
        raise TypeError(f"expected torch.{dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def version() -> str:
    return load().rnnbkt_version().decode()


def last_error() -> str:
    return load().rnnbkt_last_error().decode()


def sync_check(stream=None):
    _check(load().rnnbkt_sync_check(_stream(stream)))


def bucket_plan(lengths, K: int):
    """-> (bucket_upper int32[K_eff], bucket_of int32[n], K_eff, padded_steps)."""
    lib = load()
    L = _i32(lengths)
    n = L.size
    upper = np.zeros(max(int(K), 1), np.int32)
    bof = np.zeros(n, np.int32)
    keff = ctypes.c_int32(0)
    padded = ctypes.c_int64(0)
    _check(lib.rnnbkt_bucket_plan(_ptr(L, _i32p), n, int(K), _ptr(upper, _i32p),
                                  _ptr(bof, _i32p), ctypes.byref(keff), ctypes.byref(padded)))
    return upper[:keff.value].copy(), bof, keff.value, padded.value


ORDERINGS = {"ascending": 0, "descending": 1, "random_buckets": 2, "shuffled_batches": 3}


def epoch_schedule(lengths, bucket_of, K_eff: int, keys, B: int, ordering: str = "ascending",
                   order_keys=None):
    """-> list of int64 arrays (sequence indices of each batch, in feeding order)."""
    lib = load()
    L = _i32(lengths)
    bo = _i32(bucket_of)
    k = np.ascontiguousarray(keys, dtype=np.uint64)
    n = L.size
    if ordering not in ORDERINGS:
        raise RnnbktError(-1, f"unknown ordering {ordering!r}")
    ok = None
    if order_keys is not None:
        ok = np.ascontiguousarray(order_keys, dtype=np.uint64)
        if ok.size != n:
            raise RnnbktError(-1, "order_keys must have one entry per sequence")
    order = np.zeros(n, np.int64)
    starts = np.zeros(n + 1, np.int64)
    nb = ctypes.c_int64(0)
    if ordering == "ascending" and ok is None:
        _check(lib.rnnbkt_epoch_schedule(_ptr(L, _i32p), _ptr(bo, _i32p), n, int(K_eff),
                                         _ptr(k, _u64p), int(B), _ptr(order, _i64p),
                                         _ptr(starts, _i64p), ctypes.byref(nb)))
    else:
        _check(lib.rnnbkt_epoch_schedule_ordered(
            _ptr(L, _i32p), _ptr(bo, _i32p), n, int(K_eff), _ptr(k, _u64p), int(B),
            ORDERINGS[ordering], None if ok is None else _ptr(ok, _u64p),
            _ptr(order, _i64p), _ptr(starts, _i64p), ctypes.byref(nb)))
    return [order[starts[i]:starts[i + 1]].copy() for i in range(nb.value)]


def param_count(desc: ModelDesc) -> int:
    r = load().rnnbkt_param_count(ctypes.byref(desc))
    if r < 0:
        _check(int(r))
    return int(r)


def buffer_sizes(desc: ModelDesc, T_max: int, B: int, n_valid: int):
    """-> (reserve_bytes, workspace_bytes)."""
    r = ctypes.c_size_t(0)
    w = ctypes.c_size_t(0)
    _check(load().rnnbkt_buffer_sizes(ctypes.byref(desc), int(T_max), int(B), int(n_valid),
                                      ctypes.byref(r), ctypes.byref(w)))
    return r.value, w.value


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _need(t, count: int, what: str):
    if not isinstance(t, int) and t.numel() < count:
        raise ValueError(f"{what} holds {t.numel()} elements, needs {count}")


def _htop(desc) -> int:
    return desc.hidden * (2 if desc.bidirectional else 1)


def lstm_fwd(desc, params, x, labels, lengths, reserve, workspace, loss, stream=None):
    L = _i32(lengths)
    T, B = int(L[0]), int(L.size)
    _need(params, param_count(desc), "params")
    _need(x, T * B * desc.input_dim, "x")
    _need(labels, T * B, "labels")
    _need(loss, 1, "loss")
    _check(load().rnnbkt_lstm_fwd(ctypes.byref(desc), _dev(params, "float32"),
                                  _dev(x, "float32"), _dev(labels, "int32"), _ptr(L, _i32p),
                                  int(L[0]), int(L.size), _dev(reserve), _nbytes(reserve),
                                  _dev(workspace), _nbytes(workspace), _dev(loss, "float32"),
                                  _stream(stream)))


def ctc_workspace_bytes(T_max: int, B: int, U_max: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().rnnbkt_ctc_workspace_bytes(int(T_max), int(B), int(U_max), ctypes.byref(n)))
    return n.value


def lstm_fwd_ctc(desc, params, x, targets, target_lengths, lengths, reserve, workspace, ctc_ws,
                 loss, stream=None):
    """Forward pass with the CTC loss.  targets: device int32 [B, U_max]
    (row b's first target_lengths[b] entries hold its labels)."""
    L = _i32(lengths)
    TL = _i32(target_lengths)
    T, B = int(L[0]), int(L.size)
    if TL.size != B:
        raise ValueError("target_lengths must have one entry per sequence")
    if targets.dim() != 2 or targets.shape[0] != B:
        raise ValueError("targets must be [B, U_max]")
    U_max = int(targets.shape[1])
    _need(params, param_count(desc), "params")
    _need(x, T * B * desc.input_dim, "x")
    _need(loss, 1, "loss")
    _check(load().rnnbkt_lstm_fwd_ctc(ctypes.byref(desc), _dev(params, "float32"),
                                      _dev(x, "float32"), _dev(targets, "int32"), _ptr(TL, _i32p),
                                      U_max, _ptr(L, _i32p), T, B, _dev(reserve), _nbytes(reserve),
                                      _dev(workspace), _nbytes(workspace), _dev(ctc_ws),
                                      _nbytes(ctc_ws), _dev(loss, "float32"), _stream(stream)))


def lstm_bwd(desc, params, lengths, reserve, workspace, grads, stream=None):
    L = _i32(lengths)
    _need(params, param_count(desc), "params")
    _need(grads, param_count(desc), "grads")
    _check(load().rnnbkt_lstm_bwd(ctypes.byref(desc), _dev(params, "float32"), _ptr(L, _i32p),
                                  int(L[0]), int(L.size), _dev(reserve), _nbytes(reserve),
                                  _dev(workspace), _nbytes(workspace), _dev(grads, "float32"),
                                  _stream(stream)))


def lstm_bwd_noalloc(desc, params, lengths, reserve, grads, stream=None):
    """rnnbkt_lstm_bwd on the library's own scratch (no workspace)."""
    L = _i32(lengths)
    _need(params, param_count(desc), "params")
    _need(grads, param_count(desc), "grads")
    _check(load().rnnbkt_lstm_bwd_noalloc(ctypes.byref(desc), _dev(params, "float32"),
                                          _ptr(L, _i32p), int(L[0]), int(L.size), _dev(reserve),
                                          _nbytes(reserve), _dev(grads, "float32"),
                                          _stream(stream)))


def sgd_apply(params, grads, lr: float, stream=None, n: Optional[int] = None):
    count = params.numel() if n is None else int(n)
    if not isinstance(params, int) and count > min(params.numel(), grads.numel()):
        raise ValueError("n exceeds the tensors' sizes")
    _check(load().rnnbkt_sgd_apply(_dev(params, "float32"), _dev(grads, "float32"), count,
                                   float(lr), _stream(stream)))


def adadelta_apply(params, grads, acc_g2, acc_dx2, rho: float = 0.95, eps: float = 1e-6,
                   lr: float = 1.0, stream=None, n: Optional[int] = None):
    """One ADADELTA step in place (params, acc_g2, acc_dx2); the state tensors
    start at zero and are kept between steps."""
    count = params.numel() if n is None else int(n)
    if not isinstance(params, int) and count > min(params.numel(), grads.numel(),
                                                   acc_g2.numel(), acc_dx2.numel()):
        raise ValueError("n exceeds the tensors' sizes")
    _check(load().rnnbkt_adadelta_apply(_dev(params, "float32"), _dev(grads, "float32"),
                                        _dev(acc_g2, "float32"), _dev(acc_dx2, "float32"), count,
                                        float(rho), float(eps), float(lr), _stream(stream)))


def epoch_aggregate(replicas, prev, beta: float = 1e-6, stream=None, R: Optional[int] = None,
                    stride: Optional[int] = None, n: Optional[int] = None):
    """Eq. 3 in place: `replicas` is a [R, stride] float32 tensor (replica r in
    row r; or an address with R, stride and n given), `prev` holds V(t-1);
    both receive V(t) = mean over replicas - beta * prev."""
    if isinstance(replicas, int):
        if R is None or stride is None or n is None:
            raise ValueError("an address needs R, stride and n")
    else:
        if replicas.dim() != 2:
            raise ValueError("replicas must be a [R, stride] tensor")
        R = replicas.shape[0] if R is None else R
        stride = replicas.shape[1] if stride is None else stride
        n = stride if n is None else n
        if R > replicas.shape[0] or stride != replicas.shape[1] or n > stride:
            raise ValueError("R, stride or n do not match the replicas tensor")
    if not isinstance(prev, int) and prev.numel() < n:
        raise ValueError("prev holds fewer than n values")
    _check(load().rnnbkt_epoch_aggregate(_dev(replicas, "float32"), int(R), int(stride), int(n),
                                         _dev(prev, "float32"), float(beta), _stream(stream)))


def set_concurrency(streams: int):
    """Declares how many streams may run training calls at once (default 1)."""
    _check(load().rnnbkt_set_concurrency(int(streams)))


def top_hidden(desc, lengths, reserve, out, stream=None):
    L = _i32(lengths)
    _need(out, int(L[0]) * int(L.size) * _htop(desc), "out")
    _check(load().rnnbkt_top_hidden(ctypes.byref(desc), _ptr(L, _i32p), int(L[0]), int(L.size),
                                    _dev(reserve), _nbytes(reserve), _dev(out, "float32"),
                                    _stream(stream)))


def kernel_timer(enable: bool):
    _check(load().rnnbkt_kernel_timer(1 if enable else 0))


def kernel_timer_read(kind: str):
    """-> dict(ms, launches, flops, bytes) summed over the recorded launches."""
    ms = ctypes.c_double(0)
    fl = ctypes.c_double(0)
    by = ctypes.c_double(0)
    n = ctypes.c_int64(0)
    _check(load().rnnbkt_kernel_timer_read(KERNEL_KINDS[kind], ctypes.byref(ms), ctypes.byref(n),
                                           ctypes.byref(fl), ctypes.byref(by)))
    return {"ms": ms.value, "launches": n.value, "flops": fl.value, "bytes": by.value}
