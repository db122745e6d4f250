"""Thin ctypes binding of the C ABI in ``include/mi355am.h``.

Argument marshalling only: every function takes torch tensors that already
live on the GPU, passes their device pointers and the current HIP stream to
the native library, and raises ``AmError`` on a non-OK status.  All compute
happens in the library's HIP kernels.  If the library has not been built the
first call raises; there is no fallback path.
"""

import ctypes
import os
from dataclasses import dataclass

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmi355am.so")

F32, BF16 = 0, 1
MEAN_VALID, SUM = 0, 1
K_GEMM_FWD, K_GEMM_BWD_DATA, K_GEMM_BWD_WGT, K_LSTM_FWD, K_LSTM_BWD = 0, 1, 2, 3, 4
K_CE, K_ENCODE, K_DECODE, K_SGD, K_MISC, K_BMUF = 5, 6, 7, 8, 9, 10
KERNEL_CLASSES = ["gemm_fwd", "gemm_bwd_data", "gemm_bwd_wgt", "lstm_fwd", "lstm_bwd",
                  "soft_ce", "encode", "decode", "sgd", "misc", "bmuf"]


OK, EINVAL, ECAPACITY, EUNSUPPORTED, EHIP, EWORKSPACE, ETIMEOUT = 0, -1, -2, -3, -4, -5, -6
PATH_XCD, PATH_DEVICE, PATH_STEP = 1, 2, 3


class AmError(RuntimeError):
    """A non-OK am_status (``status``), with the library's message."""

    def __init__(self, msg, status=None):
        super().__init__(msg)
        self.status = status


class _Model(ctypes.Structure):
    _fields_ = [("layers", ctypes.c_int32), ("input_dim", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("classes", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]


@dataclass(frozen=True)
class Model:
    layers: int
    input_dim: int
    hidden: int
    classes: int
    dtype: int = BF16

    def c(self):
        return _Model(self.layers, self.input_dim, self.hidden, self.classes, self.dtype)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == BF16 else torch.float32


_lib = None
_P, _I32, _I64, _F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
_PROTOS = {
    "am_param_count": (_I64, [_P]),
    "am_param_offsets": (_I32, [_P, _P]),
    "am_workspace_bytes": (_I64, [_P, _I32, _I32, _I64]),
    "am_ce_workspace_bytes": (_I64, [_I64]),
    "am_encode_workspace_bytes": (_I64, [_I64]),
    "am_status_string": (ctypes.c_char_p, [_I32]),
    "am_recurrence_path": (_I32, [_P, _I32, _I32, _I32, _I32]),
    "am_last_error": (ctypes.c_char_p, []),
    "lstm_am_forward": (_I32, [_P, _P, _P, _P, _P, _P, _I32, _I32, _P, _P, _P, _P, _I64, _P]),
    "sparse_soft_ce": (_I32, [_I64, _I32, _I32, _P, _P, _P, _P, _I32, _P, _P, _I32, _P, _I64, _P]),
    "lstm_am_backward": (_I32, [_P, _P, _P, _P, _I32, _I32, _P, _P, _I64, _P, _P]),
    "grad_threshold_encode": (_I32, [_I64, _P, _P, _F32, _P, _I64, _P, _P, _I64, _P]),
    "grad_threshold_encode_noalloc": (_I32, [_I64, _P, _P, _F32, _P, _I64, _P, _P]),
    "grad_threshold_decode": (_I32, [_P, _P, _I64, _F32, _I64, _P, _I32, _P]),
    "grad_threshold_decode_sgd": (_I32, [_P, _P, _I64, _F32, _I64, _F32, _P, _P, _P]),
    "sgd_apply": (_I32, [_I64, _P, _P, _P, _F32, _P]),
    "am_decode_multi_workspace_bytes": (_I64, [_I32, _I64]),
    "grad_threshold_decode_multi": (_I32, [_I32, _P, _I64, _P, _F32, _I64, _P, _I32, _P, _I64, _P]),
    "bmuf_block_update": (_I32, [_I64, _I32, _I32, _P, _I64, _P, _P, _F32, _F32, _F32, _P, _P, _P]),
    "am_lfr_frames": (_I32, [_I32, _I32, _I32, _I32]),
    "am_teacher_param_count": (_I64, [_P]),
    "am_teacher_param_offsets": (_I32, [_P, _P]),
    "am_teacher_workspace_bytes": (_I64, [_P, _I32, _I32, _I64]),
    "blstm_teacher_forward": (_I32, [_P, _P, _P, _P, _I32, _I32, _P, _P, _I64, _P]),
    "kbest_logits": (_I32, [_I64, _I32, _I32, _P, _P, _P, _P]),
    "kbest_posteriors": (_I32, [_I64, _I32, _P, _P, _P]),
    "lfr_features": (_I32, [_I32, _P, _P, _I32, _I32, _I32, _I32, _P, _P, _P, _I32, _P]),
    "delay_targets": (_I32, [_I32, _I32, _P, _I32, _I32, _P, _P, _P, _P, _P, _P]),
    "am_cast_f32_to_bf16": (_I32, [_I64, _P, _P, _P]),
    "am_workspace_check": (_I32, [_P, _I64, _P]),
    "am_profile_begin": (_I32, [ctypes.c_uint32]),
    "am_profile_end": (_I32, []),
    "am_profile_sample_every": (_I32, [_I32]),
    "am_profile_get": (_I32, [_I32, _P, _P, _P, _P]),
}


def lib():
    """The loaded native library (loads it on first use)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise AmError(f"native library missing: {LIB_PATH} "
                          "(build it with `python -m paper_1904_10584_amd.build`)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _PROTOS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def exported_symbols():
    return list(_PROTOS)


def _check(status):
    if status != 0:
        L = lib()
        raise AmError(f"{L.am_status_string(status).decode()} ({status}): "
                      f"{L.am_last_error().decode()}", status)


def _dev(t, name, dtype=None):
    """Device pointer of a contiguous GPU tensor, or None."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise AmError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise AmError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise AmError(f"{name} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _host_i32(a):
    if a is None:
        return None, None
    import numpy as np
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


# ----------------------------------------------------------------- queries --

def param_count(m: Model) -> int:
    n = lib().am_param_count(ctypes.byref(m.c()))
    if n < 0:
        _check(-1)
    return int(n)


def param_offsets(m: Model):
    out = (ctypes.c_int64 * (3 * m.layers + 2))()
    _check(lib().am_param_offsets(ctypes.byref(m.c()), out))
    return list(out)


def workspace_bytes(m: Model, T, B, N) -> int:
    n = lib().am_workspace_bytes(ctypes.byref(m.c()), T, B, N)
    if n < 0:
        raise AmError("invalid model or batch for workspace query")
    return int(n)


def recurrence_path(m: Model, T, B, varlen=False, forward=True) -> int:
    """PATH_XCD, PATH_DEVICE or PATH_STEP: the kernels a layer's recurrence
    takes for this batch shape (see am_recurrence_path)."""
    p = lib().am_recurrence_path(ctypes.byref(m.c()), T, B, 1 if varlen else 0, 1 if forward else 0)
    if p < 0:
        raise AmError("invalid model or batch for the recurrence-path query", EINVAL)
    return int(p)


def ce_workspace_bytes(N) -> int:
    return int(lib().am_ce_workspace_bytes(N))


def encode_workspace_bytes(n) -> int:
    return int(lib().am_encode_workspace_bytes(n))


# ------------------------------------------------------------- entry points --

def lstm_am_forward(m: Model, params, x, T, B, logits, ws, lengths=None, h0=None, c0=None,
                    hT=None, cT=None, stream=None):
    dt = m.torch_dtype
    arr, lp = _host_i32(lengths)  # arr keeps the host array alive during the call
    _check(lib().lstm_am_forward(
        ctypes.byref(m.c()), _dev(params, "params", dt), _dev(x, "x", dt), lp,
        _dev(h0, "h0", torch.float32), _dev(c0, "c0", torch.float32), T, B,
        _dev(logits, "logits", torch.float32), _dev(hT, "hT", torch.float32),
        _dev(cT, "cT", torch.float32), _dev(ws, "ws"), ws.numel() * ws.element_size(),
        _stream(stream)))


def lstm_am_backward(m: Model, params, x, T, B, dlogits, ws, grads, lengths=None, stream=None):
    dt = m.torch_dtype
    arr, lp = _host_i32(lengths)
    _check(lib().lstm_am_backward(
        ctypes.byref(m.c()), _dev(params, "params", dt), _dev(x, "x", dt), lp, T, B,
        _dev(dlogits, "dlogits", dt), _dev(ws, "ws"), ws.numel() * ws.element_size(),
        _dev(grads, "grads", torch.float32), _stream(stream)))


def sparse_soft_ce(logits, idx, prob, loss, dlogits, ws, mask=None, reduction=MEAN_VALID,
                   stream=None):
    N, C = logits.shape
    K = idx.shape[1]
    dt = BF16 if dlogits.dtype == torch.bfloat16 else F32
    _check(lib().sparse_soft_ce(
        N, C, K, _dev(logits, "logits", torch.float32), _dev(idx, "idx", torch.int32),
        _dev(prob, "prob", torch.float32), _dev(mask, "mask", torch.uint8), reduction,
        _dev(loss, "loss", torch.float32), _dev(dlogits, "dlogits"), dt, _dev(ws, "ws"),
        ws.numel() * ws.element_size(), _stream(stream)))


def workspace_check(ws, stream=None):
    """Synchronise the stream; raise AmError if a step barrier of the last
    forward/backward pass on `ws` timed out (its outputs are then invalid)."""
    _check(lib().am_workspace_check(_dev(ws, "ws"), ws.numel() * ws.element_size(),
                                    _stream(stream)))


def grad_threshold_encode(grad, residual, tau, words, count, ws, stream=None):
    n = grad.numel()
    _check(lib().grad_threshold_encode(
        n, _dev(grad, "grad", torch.float32), _dev(residual, "residual", torch.float32),
        float(tau), _dev(words, "words", torch.int32), words.numel(),
        _dev(count, "count", torch.int64), _dev(ws, "ws"), ws.numel() * ws.element_size(),
        _stream(stream)))


ENCODE_NOALLOC_MAX_N = 1 << 25


def grad_threshold_encode_noalloc(grad, residual, tau, words, count, stream=None):
    """grad_threshold_encode without a workspace (library-owned scratch)."""
    n = grad.numel()
    _check(lib().grad_threshold_encode_noalloc(
        n, _dev(grad, "grad", torch.float32), _dev(residual, "residual", torch.float32),
        float(tau), _dev(words, "words", torch.int32), words.numel(),
        _dev(count, "count", torch.int64), _stream(stream)))


def grad_threshold_decode(words, count, tau, dense, accumulate=False, stream=None):
    _check(lib().grad_threshold_decode(
        _dev(words, "words", torch.int32), _dev(count, "count", torch.int64), words.numel(),
        float(tau), dense.numel(), _dev(dense, "dense", torch.float32), int(bool(accumulate)),
        _stream(stream)))


def grad_threshold_decode_sgd(words, count, tau, master, lr, weights_bf16=None, stream=None):
    """The decode of one stream and the SGD step on its update in one pass
    (the dense update is not materialised)."""
    _check(lib().grad_threshold_decode_sgd(
        _dev(words, "words", torch.int32), _dev(count, "count", torch.int64), words.numel(),
        float(tau), master.numel(), float(lr), _dev(master, "master", torch.float32),
        _dev(weights_bf16, "weights_bf16", torch.bfloat16), _stream(stream)))


def decode_multi_workspace_bytes(streams, n) -> int:
    return int(lib().am_decode_multi_workspace_bytes(streams, n))


def grad_threshold_decode_multi(words, counts, tau, dense, ws, accumulate=False, stream=None):
    """words: [streams][capacity] int32 GPU tensor; counts: [streams] int64."""
    if words.dim() != 2:
        raise AmError("words must be [streams][capacity]")
    S, cap = words.shape
    _check(lib().grad_threshold_decode_multi(
        S, _dev(words, "words", torch.int32), cap, _dev(counts, "counts", torch.int64),
        float(tau), dense.numel(), _dev(dense, "dense", torch.float32), int(bool(accumulate)),
        _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))


def bmuf_block_update(models, workers, global_model, delta, eta, eta_next, zeta,
                      local_master=None, local_bf16=None, stream=None):
    """models: [count][n] (or [n]) fp32 GPU tensor of the average's addends."""
    m2 = models if models.dim() == 2 else models.view(1, -1)
    count, n = m2.shape
    if global_model.numel() != n or delta.numel() != n:
        raise AmError("global_model and delta must hold n elements")
    _check(lib().bmuf_block_update(
        n, count, int(workers), _dev(m2, "models", torch.float32), n,
        _dev(global_model, "global_model", torch.float32), _dev(delta, "delta", torch.float32),
        float(eta), float(eta_next), float(zeta),
        _dev(local_master, "local_master", torch.float32),
        _dev(local_bf16, "local_bf16", torch.bfloat16), _stream(stream)))


def lfr_frames(raw_frames, stack=3, skip=3, offset=0) -> int:
    return int(lib().am_lfr_frames(raw_frames, stack, skip, offset))


def lfr_features(raw_lengths, raw, mean, std, x, stack=3, skip=3, offset=0, stream=None):
    """raw: [sum raw_lengths][raw_dim] fp32 GPU tensor; x: packed model input."""
    arr, lp = _host_i32(raw_lengths)
    dt = BF16 if x.dtype == torch.bfloat16 else F32
    _check(lib().lfr_features(
        len(raw_lengths), lp, _dev(raw, "raw", torch.float32), raw.shape[1], stack, skip, offset,
        _dev(mean, "mean", torch.float32), _dev(std, "std", torch.float32), _dev(x, "x"), dt,
        _stream(stream)))


def delay_targets(T, B, idx, prob, idx_out, prob_out, mask_out, delay, lengths=None, stream=None):
    arr, lp = _host_i32(lengths)
    _check(lib().delay_targets(
        T, B, lp, idx.shape[1], delay, _dev(idx, "idx", torch.int32), _dev(prob, "prob", torch.float32),
        _dev(idx_out, "idx_out", torch.int32), _dev(prob_out, "prob_out", torch.float32),
        _dev(mask_out, "mask_out", torch.uint8), _stream(stream)))


def teacher_param_count(m: Model) -> int:
    n = lib().am_teacher_param_count(ctypes.byref(m.c()))
    if n < 0:
        _check(-1)
    return int(n)


def teacher_param_offsets(m: Model):
    out = (ctypes.c_int64 * (6 * m.layers + 2))()
    _check(lib().am_teacher_param_offsets(ctypes.byref(m.c()), out))
    return list(out)


def teacher_workspace_bytes(m: Model, T, B, N) -> int:
    n = lib().am_teacher_workspace_bytes(ctypes.byref(m.c()), T, B, N)
    if n < 0:
        raise AmError("invalid model or batch for workspace query")
    return int(n)


def blstm_teacher_forward(m: Model, params, x, T, B, logits, ws, lengths=None, stream=None):
    dt = m.torch_dtype
    arr, lp = _host_i32(lengths)
    _check(lib().blstm_teacher_forward(
        ctypes.byref(m.c()), _dev(params, "params", dt), _dev(x, "x", dt), lp, T, B,
        _dev(logits, "logits", torch.float32), _dev(ws, "ws"), ws.numel() * ws.element_size(),
        _stream(stream)))


def kbest_logits(logits, idx, val, stream=None):
    N, C = logits.shape
    _check(lib().kbest_logits(N, C, idx.shape[1], _dev(logits, "logits", torch.float32),
                              _dev(idx, "idx", torch.int32), _dev(val, "val", torch.float32),
                              _stream(stream)))


def kbest_posteriors(val, prob, stream=None):
    N, K = val.shape
    _check(lib().kbest_posteriors(N, K, _dev(val, "val", torch.float32),
                                  _dev(prob, "prob", torch.float32), _stream(stream)))


def sgd_apply(master, update, lr, weights_bf16=None, stream=None):
    _check(lib().sgd_apply(
        master.numel(), _dev(master, "master", torch.float32),
        _dev(weights_bf16, "weights_bf16", torch.bfloat16),
        _dev(update, "update", torch.float32), float(lr), _stream(stream)))


def cast_f32_to_bf16(src, dst, stream=None):
    _check(lib().am_cast_f32_to_bf16(
        src.numel(), _dev(src, "src", torch.float32), _dev(dst, "dst", torch.bfloat16),
        _stream(stream)))


# ------------------------------------------------------------------ timing --

def profile_begin(classes, every=1):
    """Brackets the launches of `classes` with HIP events; with every > 1
    only every n-th launch of each class is bracketed."""
    mask = 0
    for k in classes:
        mask |= 1 << k
    _check(lib().am_profile_sample_every(int(every)))
    _check(lib().am_profile_begin(mask))


def profile_end():
    _check(lib().am_profile_end())


def profile_get(kernel_class):
    n = ctypes.c_int64()
    ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib().am_profile_get(kernel_class, ctypes.byref(n), ctypes.byref(ms),
                                ctypes.byref(fl), ctypes.byref(by)))
    return {"launches": n.value, "ms": ms.value, "flops": fl.value, "bytes": by.value}
