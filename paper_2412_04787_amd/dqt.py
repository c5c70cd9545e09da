"""ctypes binding of libdqt.so: the C ABI of include/dqt.h, one Python function
per entry point with the same name.  Argument marshalling only: torch tensors
are passed as device pointers on torch's current stream, every step of the
path runs in the library's HIP kernels, and a missing or unloadable library
raises immediately (there is no fallback).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdqt.so")

# dqt_status
DQT_OK, DQT_ERR_NULL, DQT_ERR_SHAPE, DQT_ERR_ALIGN, DQT_ERR_DTYPE = 0, 1, 2, 3, 4
DQT_ERR_RANGE, DQT_ERR_WORKSPACE, DQT_ERR_UNSUPPORTED, DQT_ERR_HIP = 5, 6, 7, 8
# dqt_dtype
DQT_F32, DQT_BF16, DQT_I8, DQT_FP8E4M3, DQT_TERNARY2, DQT_INT4, DQT_INT3 = 0, 1, 2, 3, 4, 5, 6

EXPORTS = (
    "dqt_act_quant", "dqt_act_quant_batch", "dqt_linear_fwd_workspace", "dqt_linear_fwd", "dqt_linear_bwd_workspace",
    "dqt_linear_bwd", "dqt_linear_fwd_batch_workspace", "dqt_linear_fwd_batch",
    "dqt_linear_bwd_batch_workspace", "dqt_linear_bwd_batch", "dqt_linear_bwd_sr_batch",
    "dqt_linear_fwd_batch_noalloc", "dqt_sr_table_bytes", "dqt_sr_table_build",
    "dqt_sr_update_table", "dqt_rmsnorm_act_quant", "dqt_rmsnorm_backward", "dqt_absmax_requant_workspace",
    "dqt_absmax_requant_batch",
    "dqt_sr_update_batch", "dqt_adamw_sr_update", "dqt_adamw_sr_update_batch",
    "dqt_update_variant_workspace", "dqt_update_variant_batch",
    "dqt_sr_update", "dqt_debug_rng", "dqt_absmean_init", "dqt_pack_ternary",
    "dqt_unpack_ternary", "dqt_pack_int4", "dqt_unpack_int4", "dqt_pack_int3", "dqt_unpack_int3", "dqt_launch_timer_start", "dqt_launch_timer_stop", "dqt_read_stream",
    "dqt_status_string", "dqt_version",
)


class DqtWeight(ctypes.Structure):
    _fields_ = [
        ("d_out", ctypes.c_int32), ("d_in", ctypes.c_int32), ("wfmt", ctypes.c_int32),
        ("qmin", ctypes.c_int32), ("qmax", ctypes.c_int32), ("alpha", ctypes.c_float),
        ("tensor_id", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
    ]


MAX_BATCH = 8


class DqtLinearIO(ctypes.Structure):
    _fields_ = [
        ("w", ctypes.POINTER(DqtWeight)), ("Wq", ctypes.c_void_p), ("Xq", ctypes.c_void_p),
        ("xdq", ctypes.c_void_p), ("Y", ctypes.c_void_p), ("dY", ctypes.c_void_p),
        ("dX", ctypes.c_void_p), ("dW", ctypes.c_void_p),
    ]


class DqtActIO(ctypes.Structure):
    _fields_ = [("X", ctypes.c_void_p), ("Xq", ctypes.c_void_p), ("xdq", ctypes.c_void_p),
                ("K", ctypes.c_int32), ("reserved", ctypes.c_int32)]


def weight(d_out: int, d_in: int, wfmt: int, qmin: int, qmax: int, alpha: float,
           tensor_id: int = 0) -> DqtWeight:
    return DqtWeight(d_out, d_in, wfmt, qmin, qmax, float(alpha), tensor_id, 0)


class DqtError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {status_string(status)}")


_lib = None

_vp, _i32, _i64, _u32, _u64, _f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                     ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float)
_wp = ctypes.POINTER(DqtWeight)

_SIGS = {
    "dqt_act_quant": (_i32, [_vp, _i32, _i64, _i32, _i32, _vp, _vp, _vp]),
    "dqt_act_quant_batch": (_i32, [_i32, _vp, _i32, _i64, _i32, _vp]),
    "dqt_rmsnorm_act_quant": (_i32, [_vp, _i32, _vp, _f32, _i64, _i32, _i32, _vp, _vp, _vp, _vp]),
    "dqt_rmsnorm_backward": (_i32, [_i32, _vp, _vp, _i32, _vp, _vp, _i64, _i32, _vp, _vp, _i32, _vp]),
    "dqt_linear_fwd_workspace": (ctypes.c_size_t, [_wp]),
    "dqt_linear_fwd": (_i32, [_wp, _vp, _vp, _i32, _i64, _i32, _vp, _vp, _vp, _i32, _vp,
                              ctypes.c_size_t, _vp]),
    "dqt_linear_bwd_workspace": (ctypes.c_size_t, [_wp, _i64]),
    "dqt_linear_bwd": (_i32, [_wp, _vp, _vp, _i32, _vp, _vp, _i32, _i64, _i32, _vp, _i32, _vp,
                              _vp, ctypes.c_size_t, _vp]),
    "dqt_sr_update": (_i32, [_wp, _vp, _vp, _f32, _u64, _u32, _vp, _vp]),
    "dqt_linear_fwd_batch_workspace": (ctypes.c_size_t, [_i32, _vp]),
    "dqt_linear_fwd_batch": (_i32, [_i32, _vp, _i64, _i32, _i32, _vp, ctypes.c_size_t, _vp]),
    "dqt_linear_fwd_batch_noalloc": (_i32, [_i32, _vp, _i64, _i32, _i32, _vp]),
    "dqt_linear_bwd_batch_workspace": (ctypes.c_size_t, [_i32, _vp, _i64]),
    "dqt_linear_bwd_batch": (_i32, [_i32, _vp, _i64, _i32, _i32, _i32, _i32, _vp,
                                    ctypes.c_size_t, _vp]),
    "dqt_linear_bwd_sr_batch": (_i32, [_i32, _vp, _i64, _i32, _i32, _i32, _i32, _f32, _u64, _u32,
                                       _vp, _vp, ctypes.c_size_t, _vp]),
    "dqt_sr_update_batch": (_i32, [_i32, _vp, _f32, _u64, _u32, _vp, _vp]),
    "dqt_sr_table_bytes": (ctypes.c_size_t, [_i32]),
    "dqt_sr_table_build": (_i32, [_i32, _vp, _vp, ctypes.c_size_t]),
    "dqt_sr_update_table": (_i32, [_i32, _vp, _vp, _f32, _u64, _u32, _vp, _vp, _vp]),
    "dqt_update_variant_workspace": (ctypes.c_size_t, [_i32]),
    "dqt_absmax_requant_workspace": (ctypes.c_size_t, [_i32]),
    "dqt_absmax_requant_batch": (_i32, [_i32, _vp, _f32, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "dqt_update_variant_batch": (_i32, [_i32, _vp, _f32, _u64, _u32, _i32, _f32, _vp, _vp,
                                        ctypes.c_size_t, _vp]),
    "dqt_adamw_sr_update": (_i32, [_wp, _vp, _vp, _vp, _vp, _vp, _u64, _u32, _vp, _vp]),
    "dqt_adamw_sr_update_batch": (_i32, [_i32, _vp, _vp, _vp, _vp, _u64, _u32, _vp, _vp]),
    "dqt_debug_rng": (_i32, [_u64, _u32, _u32, _u64, _i64, _vp, _vp]),
    "dqt_absmean_init": (_i32, [_vp, _i64, _i32, _i32, _vp, _vp]),
    "dqt_pack_ternary": (_i32, [_vp, _i64, _i64, _vp]),
    "dqt_unpack_ternary": (_i32, [_vp, _i64, _i64, _vp]),
    "dqt_pack_int4": (_i32, [_vp, _i64, _i64, _vp]),
    "dqt_unpack_int4": (_i32, [_vp, _i64, _i64, _vp]),
    "dqt_pack_int3": (_i32, [_vp, _i64, _i64, _vp]),
    "dqt_unpack_int3": (_i32, [_vp, _i64, _i64, _vp]),
    "dqt_launch_timer_start": (_i32, [_i32]),
    "dqt_launch_timer_stop": (_i32, [_vp, _i32, _vp]),
    "dqt_read_stream": (_i32, [_vp, ctypes.c_size_t, _vp, _vp]),
    "dqt_status_string": (ctypes.c_char_p, [_i32]),
    "dqt_version": (_i32, []),
}


def load(path: str = LIB_PATH):
    """Load libdqt.so (once).  Raises if it is missing: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2412_04787_amd.build_lib`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(fn: str, st: int):
    if st != DQT_OK:
        raise DqtError(fn, st)


def status_string(st: int) -> str:
    return load().dqt_status_string(st).decode()


def version() -> int:
    return load().dqt_version()


# ----------------------------------------------------------------- tensors

def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def dtype_code(t) -> int:
    torch = _torch()
    return {torch.float32: DQT_F32, torch.bfloat16: DQT_BF16, torch.int8: DQT_I8,
            torch.float8_e4m3fn: DQT_FP8E4M3, torch.uint8: DQT_FP8E4M3}[t.dtype]


def dqt_act_quant(X, act_q: int, Xq, xdq, stream=None):
    M, K = X.shape
    _check("dqt_act_quant", load().dqt_act_quant(_ptr(X), dtype_code(X), M, K, act_q, _ptr(Xq),
                                                 _ptr(xdq), _stream(stream)))


def dqt_rmsnorm_act_quant(X, gamma, eps: float, act_q: int, Xq, xdq, rinv=None, stream=None):
    M, K = X.shape
    _check("dqt_rmsnorm_act_quant",
           load().dqt_rmsnorm_act_quant(_ptr(X), dtype_code(X), _ptr(gamma), eps, M, K, act_q,
                                        _ptr(Xq), _ptr(xdq), _ptr(rinv), _stream(stream)))


def dqt_rmsnorm_backward(dYs, X, gamma, rinv, dX, gpart, stream=None):
    """dYs: list of 1..4 [M, K] bf16 tensors; gpart: [blocks, K] fp32."""
    M, K = X.shape
    ptrs = (ctypes.c_void_p * len(dYs))(*[t.data_ptr() for t in dYs])
    _check("dqt_rmsnorm_backward",
           load().dqt_rmsnorm_backward(len(dYs), ptrs, _ptr(X), dtype_code(X), _ptr(gamma),
                                       _ptr(rinv), M, K, _ptr(dX), _ptr(gpart), gpart.shape[0],
                                       _stream(stream)))


def dqt_linear_fwd_workspace(w: DqtWeight) -> int:
    return int(load().dqt_linear_fwd_workspace(ctypes.byref(w)))


def dqt_linear_fwd(w: DqtWeight, Wq, X, M: int, act_q: int, Xq, xdq, Y, ws=None, stream=None,
                   x_t: int | None = None):
    """X may be None when Xq / xdq already hold the quantised input."""
    if x_t is None:
        x_t = dtype_code(X) if X is not None else DQT_F32
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("dqt_linear_fwd", load().dqt_linear_fwd(ctypes.byref(w), _ptr(Wq), _ptr(X), x_t, M,
                                                   act_q, _ptr(Xq), _ptr(xdq), _ptr(Y),
                                                   dtype_code(Y), _ptr(ws), ws_bytes,
                                                   _stream(stream)))


def workspace(nbytes: int, device="cuda:0"):
    """A zero-filled device buffer of at least nbytes (16-byte aligned), or
    None for 0.  (The library does not depend on a workspace's contents; the
    zero fill only makes unused bytes deterministic.)"""
    if nbytes == 0:
        return None
    torch = _torch()
    return torch.zeros(((nbytes + 15) // 16 * 4,), dtype=torch.float32, device=device)


def dqt_linear_bwd_workspace(w: DqtWeight, M: int) -> int:
    return int(load().dqt_linear_bwd_workspace(ctypes.byref(w), M))


def dqt_linear_bwd(w: DqtWeight, Wq, Xq, act_q: int, xdq, dY, M: int, xt_t: int, dX, dW,
                   ws=None, stream=None, dy_t: int | None = None, dx_t: int | None = None):
    dy_t = dtype_code(dY) if dy_t is None else dy_t
    dx_t = (dtype_code(dX) if dX is not None else DQT_F32) if dx_t is None else dx_t
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("dqt_linear_bwd", load().dqt_linear_bwd(ctypes.byref(w), _ptr(Wq), _ptr(Xq), act_q,
                                                   _ptr(xdq), _ptr(dY), dy_t, M, xt_t, _ptr(dX),
                                                   dx_t, _ptr(dW), _ptr(ws), ws_bytes,
                                                   _stream(stream)))


def dqt_sr_update(w: DqtWeight, Wq, dW, lr: float, seed: int, step: int, counters=None,
                  stream=None):
    _check("dqt_sr_update", load().dqt_sr_update(ctypes.byref(w), _ptr(Wq), _ptr(dW), lr, seed,
                                                 step, _ptr(counters), _stream(stream)))


def dqt_debug_rng(seed: int, step: int, tensor_id: int, i0: int, out, stream=None):
    _check("dqt_debug_rng", load().dqt_debug_rng(seed, step, tensor_id, i0, out.numel(),
                                                 _ptr(out), _stream(stream)))


def dqt_launch_timer_start(max_launches: int):
    _check("dqt_launch_timer_start", load().dqt_launch_timer_start(max_launches))


def dqt_launch_timer_stop(max_launches: int):
    """Durations (ms) of the GEMM kernel launches timed since the start, in
    issue order, and how many launches were timed."""
    ms = (ctypes.c_float * max(1, max_launches))()
    count = ctypes.c_int32(0)
    _check("dqt_launch_timer_stop", load().dqt_launch_timer_stop(ms, max_launches, ctypes.byref(count)))
    return [float(ms[k]) for k in range(min(count.value, max_launches))], count.value


READ_STREAM_SINK_WORDS = 32768


def dqt_read_stream(src, sink, stream=None):
    """One streaming read of the device tensor src (all its bytes); sink: a
    device int32/uint32 tensor of READ_STREAM_SINK_WORDS words."""
    nbytes = src.numel() * src.element_size()
    assert sink.numel() * sink.element_size() >= 4 * READ_STREAM_SINK_WORDS
    _check("dqt_read_stream", load().dqt_read_stream(_ptr(src), nbytes, _ptr(sink), _stream(stream)))


# ----------------------------------------------------------------- batches

def linear_io(entries):
    """entries: list of dicts with keys w (DqtWeight), Wq, Xq, xdq, Y, dY, dX, dW
    (tensors or None).  Returns a ctypes array of dqt_linear_io; the weight
    descriptors and the tensors are kept alive on the array (it holds raw
    device pointers)."""
    arr = (DqtLinearIO * len(entries))()
    keep = []
    for k, e in enumerate(entries):
        w = e["w"]
        keep.append(w)
        arr[k].w = ctypes.pointer(w)
        for f in ("Wq", "Xq", "xdq", "Y", "dY", "dX", "dW"):
            t = e.get(f)
            setattr(arr[k], f, None if t is None else t.data_ptr())
            if t is not None:
                keep.append(t)
    arr._keep = keep
    return arr


def act_io(entries):
    """entries: list of (X, Xq, xdq) tensors with X [M, K].  Returns a ctypes
    array of dqt_act_io."""
    arr = (DqtActIO * len(entries))()
    for k, (X, Xq, xdq) in enumerate(entries):
        arr[k].X = X.data_ptr()
        arr[k].Xq = Xq.data_ptr()
        arr[k].xdq = xdq.data_ptr()
        arr[k].K = X.shape[1]
        arr[k].reserved = 0
    return arr


def dqt_act_quant_batch(io, x_t: int, M: int, act_q: int, stream=None):
    _check("dqt_act_quant_batch", load().dqt_act_quant_batch(len(io), io, x_t, M, act_q,
                                                             _stream(stream)))


def dqt_linear_fwd_batch_workspace(io) -> int:
    return int(load().dqt_linear_fwd_batch_workspace(len(io), io))


def dqt_linear_fwd_batch(io, M: int, act_q: int, y_t: int, ws=None, stream=None):
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("dqt_linear_fwd_batch", load().dqt_linear_fwd_batch(len(io), io, M, act_q, y_t, _ptr(ws),
                                                               ws_bytes, _stream(stream)))


NOALLOC_SCRATCH_BYTES = 32 << 20


def dqt_linear_fwd_batch_noalloc(io, M: int, act_q: int, y_t: int, stream=None):
    """dqt_linear_fwd_batch with the library's static per-GPU scratch instead
    of a workspace (the call allocates nothing)."""
    _check("dqt_linear_fwd_batch_noalloc",
           load().dqt_linear_fwd_batch_noalloc(len(io), io, M, act_q, y_t, _stream(stream)))


def dqt_linear_bwd_batch_workspace(io, M: int) -> int:
    return int(load().dqt_linear_bwd_batch_workspace(len(io), io, M))


def dqt_linear_bwd_batch(io, M: int, act_q: int, dy_t: int, xt_t: int, dx_t: int, ws=None,
                         stream=None):
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("dqt_linear_bwd_batch", load().dqt_linear_bwd_batch(len(io), io, M, act_q, dy_t, xt_t,
                                                               dx_t, _ptr(ws), ws_bytes,
                                                               _stream(stream)))


def dqt_linear_bwd_sr_batch(io, M: int, act_q: int, dy_t: int, xt_t: int, dx_t: int, lr: float,
                            seed: int, step: int, counters=None, ws=None, stream=None):
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("dqt_linear_bwd_sr_batch",
           load().dqt_linear_bwd_sr_batch(len(io), io, M, act_q, dy_t, xt_t, dx_t, lr, seed, step,
                                          _ptr(counters), _ptr(ws), ws_bytes, _stream(stream)))


DQT_UPD_SR, DQT_UPD_NEAREST, DQT_UPD_FORCE_REMAIN, DQT_UPD_FORCE_CHANGE = 0, 1, 2, 3


def dqt_update_variant_workspace(n: int) -> int:
    return int(load().dqt_update_variant_workspace(n))


def dqt_update_variant_batch(io, lr: float, seed: int, step: int, mode: int, frac: float = 0.2,
                             counters=None, ws=None, stream=None):
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("dqt_update_variant_batch",
           load().dqt_update_variant_batch(len(io), io, lr, seed, step, mode, frac, _ptr(counters),
                                           _ptr(ws), ws_bytes, _stream(stream)))


def dqt_absmax_requant_batch(io, lr: float, alpha_out, counters=None, ws=None, stream=None):
    """alpha_out: device fp32 [len(io)], receives each tensor's new scale."""
    if ws is None:
        ws = workspace(int(load().dqt_absmax_requant_workspace(len(io))))
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("dqt_absmax_requant_batch",
           load().dqt_absmax_requant_batch(len(io), io, lr, _ptr(alpha_out), _ptr(counters),
                                           _ptr(ws), ws_bytes, _stream(stream)))


class DqtAdamW(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float)]


def adamw(lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
          weight_decay: float = 0.0) -> DqtAdamW:
    return DqtAdamW(lr, beta1, beta2, eps, weight_decay)


def dqt_adamw_sr_update(w, Wq, dW, m, v, hp: DqtAdamW, seed: int, step: int, counters=None,
                        stream=None):
    _check("dqt_adamw_sr_update",
           load().dqt_adamw_sr_update(ctypes.byref(w), _ptr(Wq), _ptr(dW), _ptr(m), _ptr(v),
                                      ctypes.byref(hp), seed, step, _ptr(counters),
                                      _stream(stream)))


def dqt_adamw_sr_update_batch(io, ms, vs, hp: DqtAdamW, seed: int, step: int, counters=None,
                              stream=None):
    """ms, vs: lists of fp32 device tensors (the moments of each entry of io)."""
    n = len(io)
    mp = (ctypes.c_void_p * n)(*[t.data_ptr() for t in ms])
    vp = (ctypes.c_void_p * n)(*[t.data_ptr() for t in vs])
    _check("dqt_adamw_sr_update_batch",
           load().dqt_adamw_sr_update_batch(n, io, mp, vp, ctypes.byref(hp), seed, step,
                                            _ptr(counters), _stream(stream)))


def dqt_sr_update_batch(io, lr: float, seed: int, step: int, counters=None, stream=None):
    _check("dqt_sr_update_batch", load().dqt_sr_update_batch(len(io), io, lr, seed, step,
                                                             _ptr(counters), _stream(stream)))


def dqt_sr_table_bytes(n: int) -> int:
    return int(load().dqt_sr_table_bytes(n))


def dqt_sr_table_build(io) -> np.ndarray:
    """The update table of the entries of io, as host bytes (copy them to the
    device once, e.g. torch.from_numpy(t).to(device))."""
    n = len(io)
    table = np.zeros(max(dqt_sr_table_bytes(n), 1), dtype=np.uint8)
    _check("dqt_sr_table_build", load().dqt_sr_table_build(n, io, table.ctypes.data, table.size))
    return table


def dqt_sr_update_table(io, table, lr: float, seed: int, step: int, counters=None,
                        per_tensor=None, stream=None):
    """table: the device copy of dqt_sr_table_build(io)."""
    _check("dqt_sr_update_table",
           load().dqt_sr_update_table(len(io), io, _ptr(table), lr, seed, step, _ptr(counters),
                                      _ptr(per_tensor), _stream(stream)))


# ----------------------------------------------------------------- host helpers

def dqt_absmean_init(W0: np.ndarray, qmin: int, qmax: int):
    W0 = np.ascontiguousarray(W0, dtype=np.float32)
    q = np.empty(W0.shape, dtype=np.int8)
    alpha = ctypes.c_float()
    _check("dqt_absmean_init", load().dqt_absmean_init(W0.ctypes.data, W0.size, qmin, qmax,
                                                       q.ctypes.data, ctypes.byref(alpha)))
    return q, np.float32(alpha.value)


def dqt_pack_int4(q: np.ndarray) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.int8)
    rows, cols = q.shape
    packed = np.empty((rows, cols // 2), dtype=np.uint8)
    _check("dqt_pack_int4", load().dqt_pack_int4(q.ctypes.data, rows, cols, packed.ctypes.data))
    return packed


def dqt_unpack_int4(packed: np.ndarray, cols: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    rows = packed.shape[0]
    q = np.empty((rows, cols), dtype=np.int8)
    _check("dqt_unpack_int4", load().dqt_unpack_int4(packed.ctypes.data, rows, cols, q.ctypes.data))
    return q


def dqt_pack_int3(q: np.ndarray) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.int8)
    rows, cols = q.shape
    packed = np.empty((rows, 3 * cols // 8), dtype=np.uint8)
    _check("dqt_pack_int3", load().dqt_pack_int3(q.ctypes.data, rows, cols, packed.ctypes.data))
    return packed


def dqt_unpack_int3(packed: np.ndarray, cols: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    rows = packed.shape[0]
    q = np.empty((rows, cols), dtype=np.int8)
    _check("dqt_unpack_int3", load().dqt_unpack_int3(packed.ctypes.data, rows, cols, q.ctypes.data))
    return q


def dqt_pack_ternary(q: np.ndarray) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.int8)
    rows, cols = q.shape
    packed = np.empty((rows, cols // 4), dtype=np.uint8)
    _check("dqt_pack_ternary", load().dqt_pack_ternary(q.ctypes.data, rows, cols,
                                                       packed.ctypes.data))
    return packed


def dqt_unpack_ternary(packed: np.ndarray, cols: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    rows = packed.shape[0]
    q = np.empty((rows, cols), dtype=np.int8)
    _check("dqt_unpack_ternary", load().dqt_unpack_ternary(packed.ctypes.data, rows, cols,
                                                           q.ctypes.data))
    return q
