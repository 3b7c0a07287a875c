"""ctypes binding of libadpsgd_blstm.so: one Python function per C entry
point, same names, argument marshalling only.  Device buffers are torch
tensors (torch supplies memory and streams); every computation runs in the
library's HIP kernels.  The library must have been built
(``__graft_entry__.build()``); loading fails loudly otherwise."""

from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libadpsgd_blstm.so")

BLSTM_FP32 = 0
BLSTM_BF16 = 1
ADPSGD_ORDER_EQ7 = 1
ADPSGD_WRITE_PEER = 2
BLSTM_EINVAL = -1
BLSTM_EUNSUPPORTED = -2
BLSTM_EHIP = -3
HEAD_STATIC_SCRATCH_BYTES = 64 << 20   # the static head workspace (adpsgd_blstm.h)

EXPORTED = ("blstm_param_count", "blstm_workspace_bytes", "blstm_pack_params", "blstm_fwd",
            "softmax_ce_fwd_bwd", "softmax_ce_fwd_bwd_static", "blstm_bwd", "replica_grad_reduce", "adpsgd_step",
            "blstm_recurrence_ok", "blstm_last_error", "blstm_timing_begin", "blstm_timing_end")


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("L", "D", "H", "P", "K", "T", "B", "precision")]


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


class BlstmError(RuntimeError):
    def __init__(self, fn, code, msg):
        super().__init__(f"{fn} failed ({code}): {msg}")
        self.code = code


_lib = None


def lib():
    """Load the library once (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        DP = ctypes.POINTER(Dims)
        S = ctypes.c_size_t
        L.blstm_param_count.argtypes = [DP]
        L.blstm_param_count.restype = ctypes.c_int64
        L.blstm_workspace_bytes.argtypes = [DP, ctypes.POINTER(S), ctypes.POINTER(S),
                                            ctypes.POINTER(S), ctypes.POINTER(S)]
        L.blstm_pack_params.argtypes = [DP, P, P, P]
        L.blstm_fwd.argtypes = [DP, P, P, P, P, P, P]
        L.softmax_ce_fwd_bwd.argtypes = [DP, P, P, P, P, ctypes.c_float, P, P, P, P, P]
        L.softmax_ce_fwd_bwd_static.argtypes = [DP, P, P, P, P, ctypes.c_float, P, P, P, P]
        L.blstm_bwd.argtypes = [DP, P, P, P, P, P, P, P]
        L.blstm_recurrence_ok.argtypes = [DP, P, P]
        L.replica_grad_reduce.argtypes = [ctypes.POINTER(P), ctypes.c_int32, ctypes.c_int64,
                                          ctypes.c_float, P, P]
        L.adpsgd_step.argtypes = [P, P, ctypes.POINTER(P), ctypes.c_int32, ctypes.c_float,
                                  ctypes.c_int64, ctypes.c_float, ctypes.c_uint32, P, P]
        L.blstm_last_error.restype = ctypes.c_char_p
        L.blstm_timing_begin.argtypes = [ctypes.c_char_p]
        L.blstm_timing_end.argtypes = [ctypes.POINTER(KernelTime), ctypes.c_int32,
                                       ctypes.POINTER(ctypes.c_int32)]
        for name in ("blstm_workspace_bytes", "blstm_pack_params", "blstm_fwd", "softmax_ce_fwd_bwd",
                     "softmax_ce_fwd_bwd_static",
                     "blstm_bwd", "replica_grad_reduce", "adpsgd_step", "blstm_timing_begin",
                     "blstm_timing_end"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def make_dims(L, D, H, P, K, T, B, precision):
    if isinstance(precision, str):
        precision = {"fp32": BLSTM_FP32, "bf16": BLSTM_BF16}[precision]
    return Dims(L, D, H, P, K, T, B, precision)


def _check(fn, rc):
    if rc != 0:
        raise BlstmError(fn, rc, lib().blstm_last_error().decode())
    return rc


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def blstm_param_count(dims: Dims) -> int:
    n = lib().blstm_param_count(ctypes.byref(dims))
    if n < 0:
        raise BlstmError("blstm_param_count", n, lib().blstm_last_error().decode())
    return n


def blstm_workspace_bytes(dims: Dims) -> dict:
    vals = [ctypes.c_size_t() for _ in range(4)]
    _check("blstm_workspace_bytes",
           lib().blstm_workspace_bytes(ctypes.byref(dims), *[ctypes.byref(v) for v in vals]))
    return dict(zip(("act_ws", "head_ws", "theta_lp", "y_top"), (v.value for v in vals)))


def blstm_pack_params(dims, theta, theta_lp, stream=None):
    return _check("blstm_pack_params", lib().blstm_pack_params(
        ctypes.byref(dims), _ptr(theta), _ptr(theta_lp), _stream(stream)))


def blstm_fwd(dims, theta, theta_lp, x, act_ws, y_top, stream=None):
    return _check("blstm_fwd", lib().blstm_fwd(
        ctypes.byref(dims), _ptr(theta), _ptr(theta_lp), _ptr(x), _ptr(act_ws), _ptr(y_top),
        _stream(stream)))


def softmax_ce_fwd_bwd(dims, theta, theta_lp, y_top, labels, loss_scale, loss, dy_top, grad,
                       head_ws, stream=None):
    return _check("softmax_ce_fwd_bwd", lib().softmax_ce_fwd_bwd(
        ctypes.byref(dims), _ptr(theta), _ptr(theta_lp), _ptr(y_top), _ptr(labels),
        ctypes.c_float(loss_scale), _ptr(loss), _ptr(dy_top), _ptr(grad), _ptr(head_ws),
        _stream(stream)))


def softmax_ce_fwd_bwd_static(dims, theta, theta_lp, y_top, labels, loss_scale, loss, dy_top, grad, stream=None):
    return _check("softmax_ce_fwd_bwd_static", lib().softmax_ce_fwd_bwd_static(
        ctypes.byref(dims), _ptr(theta), _ptr(theta_lp), _ptr(y_top), _ptr(labels),
        ctypes.c_float(loss_scale), _ptr(loss), _ptr(dy_top), _ptr(grad), _stream(stream)))


def blstm_bwd(dims, theta, theta_lp, act_ws, y_top, dy_top, grad, stream=None):
    return _check("blstm_bwd", lib().blstm_bwd(
        ctypes.byref(dims), _ptr(theta), _ptr(theta_lp), _ptr(act_ws), _ptr(y_top), _ptr(dy_top),
        _ptr(grad), _stream(stream)))


def blstm_recurrence_ok(dims, act_ws, stream=None):
    return _check("blstm_recurrence_ok", lib().blstm_recurrence_ok(ctypes.byref(dims), _ptr(act_ws),
                                                                   _stream(stream)))


def _ptr_array(tensors):
    arr = (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])
    return ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)), arr


def replica_grad_reduce(grads, scale, out, stream=None):
    ptrs, keep = _ptr_array(grads)
    n = grads[0].numel()
    return _check("replica_grad_reduce", lib().replica_grad_reduce(
        ptrs, len(grads), n, ctypes.c_float(scale), _ptr(out), _stream(stream)))


def adpsgd_step(theta, theta_peer, grads, scale, lr, flags=0, theta_lp=None, stream=None):
    ptrs, keep = _ptr_array(grads)
    return _check("adpsgd_step", lib().adpsgd_step(
        _ptr(theta), _ptr(theta_peer), ptrs, len(grads), ctypes.c_float(scale), theta.numel(),
        ctypes.c_float(lr), flags, _ptr(theta_lp), _stream(stream)))


def blstm_timing_begin(prefix: str = ""):
    return _check("blstm_timing_begin", lib().blstm_timing_begin(prefix.encode()))


def blstm_timing_end(cap: int = 64) -> dict:
    buf = (KernelTime * cap)()
    count = ctypes.c_int32()
    _check("blstm_timing_end", lib().blstm_timing_end(buf, cap, ctypes.byref(count)))
    return {buf[i].name.decode(): (buf[i].launches, buf[i].total_ms) for i in range(min(count.value, cap))}
