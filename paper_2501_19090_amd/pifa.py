"""Thin ctypes binding of libpifa (include/pifa.h).

Argument marshalling only: every function has the name of the C entry point
it calls, takes torch tensors for device buffers (or numpy arrays for host
index arrays) and raises :class:`PifaError` on a non-OK status.  All compute
runs in the HIP library; if it is missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os
import re
import threading

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpifa.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "pifa.h")

PIFA_F32 = 0
PIFA_BF16 = 1

PIFA_OK = 0
PIFA_ERR_INVALID_ARG = -1
PIFA_ERR_BAD_INDEX = -2
PIFA_ERR_UNSUPPORTED = -3
PIFA_ERR_HIP = -4
PIFA_ERR_OOM = -5
PIFA_ERR_NOT_RANK_R = -6
PIFA_ERR_NOT_SPD = -7
PIFA_ERR_WRONG_DEVICE = -8
PIFA_ERR_TOO_LARGE = -9


class pifa_dims(ctypes.Structure):
    _fields_ = [("d_in", ctypes.c_int64), ("d_out", ctypes.c_int64), ("r", ctypes.c_int64)]


class PifaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__("%s failed: %s" % (fn, pifa_status_string(status)))


_lock = threading.Lock()
_lib = None

_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32p = ctypes.POINTER(ctypes.c_int32)
_st = ctypes.c_int

_SIGNATURES = {
    "pifa_status_string": (ctypes.c_char_p, [_st]),
    "pifa_validate_partition": (_st, [_i32p, _i32p, pifa_dims]),
    "pifa_gemm_plan": (_st, [_i64, _i64, _i64, ctypes.c_int, ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                             ctypes.POINTER(_i64)]),
    "pifa_layer_create": (_st, [_vp, _vp, _i32p, _i32p, pifa_dims, ctypes.c_int, ctypes.POINTER(_vp)]),
    "pifa_layer_destroy": (_st, [_vp]),
    "pifa_layer_reserve": (_st, [_vp, _i64]),
    "pifa_forward": (_st, [_vp, _vp, _vp, _i64, _vp]),
    "pifa_forward_noalloc": (_st, [_vp, _vp, _vp, _i64, _vp]),
    "pifa_layer_weight_bytes": (ctypes.c_size_t, [_vp]),
    "pifa_layer_set_intermediate_scale": (_st, [_vp, ctypes.c_int]),
    "pifa_layer_overflow_count": (_st, [_vp, ctypes.POINTER(_i64)]),
    "dense_forward": (_st, [_vp, _vp, _vp, _i64, _i64, _i64, ctypes.c_int, _vp]),
    "dense_layer_create": (_st, [_vp, _i64, _i64, ctypes.c_int, ctypes.POINTER(_vp)]),
    "dense_layer_forward": (_st, [_vp, _vp, _vp, _i64, _vp]),
    "dense_layer_destroy": (_st, [_vp]),
    "dense_layer_reserve": (_st, [_vp, _i64]),
    "lowrank_uv_forward": (_st, [_vp, _vp, _vp, _vp, _i64, pifa_dims, ctypes.c_int, _vp]),
    "lowrank_layer_create": (_st, [_vp, _vp, pifa_dims, ctypes.c_int, ctypes.POINTER(_vp)]),
    "lowrank_layer_forward": (_st, [_vp, _vp, _vp, _i64, _vp]),
    "lowrank_layer_reserve": (_st, [_vp, _i64]),
    "lowrank_layer_destroy": (_st, [_vp]),
    "pifa_layer_backward": (_st, [_vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp]),
    "pifa_group_create": (_st, [ctypes.c_int, ctypes.POINTER(_vp), ctypes.POINTER(_vp), ctypes.POINTER(_i32p),
                                ctypes.POINTER(_i32p), ctypes.POINTER(pifa_dims), ctypes.c_int,
                                ctypes.POINTER(_vp)]),
    "pifa_group_destroy": (_st, [_vp]),
    "pifa_group_reserve": (_st, [_vp, _i64]),
    "pifa_group_forward": (_st, [_vp, _vp, _vp, _i64, _vp]),
    "pifa_group_weight_bytes": (ctypes.c_size_t, [_vp]),
    "pifa_group_set_intermediate_scale": (_st, [_vp, ctypes.c_int]),
    "pifa_group_overflow_count": (_st, [_vp, ctypes.POINTER(_i64)]),
    "pifa_calib_create": (_st, [_i64, ctypes.POINTER(_vp)]),
    "pifa_calib_destroy": (_st, [_vp]),
    "pifa_calib_reset": (_st, [_vp, _vp]),
    "pifa_calib_accumulate": (_st, [_vp, _vp, _vp, _i64, _vp]),
    "pifa_calib_read": (_st, [_vp, _vp, _vp, _vp]),
    "pifa_calib_reconstruct": (_st, [_vp, _vp, _i64, _vp, _i64, ctypes.c_double, ctypes.c_double, _vp, _vp, _vp]),
    "pifa_build_f64": (_st, [_vp, pifa_dims, _vp, _vp, _i32p, _i32p, ctypes.POINTER(ctypes.c_double), _vp]),
    "pifa_probe_mfma": (_st, [_i64, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), _vp]),
    "pifa_probe_mfma_random": (_st, [_i64, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), _vp]),
    "pifa_probe_hbm_read": (_st, [_vp, _i64, ctypes.c_int, ctypes.POINTER(ctypes.c_double), _vp]),
    "pifa_profile_enable": (_st, [ctypes.c_int]),
    "pifa_profile_reset": (_st, []),
    "pifa_profile_read": (_st, [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(_i64),
                                ctypes.POINTER(ctypes.c_double), ctypes.c_int, ctypes.POINTER(ctypes.c_int)]),
}


def lib():
    """Open libpifa.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError("libpifa.so not built: run `python -m paper_2501_19090_amd.build`")
            handle = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in _SIGNATURES.items():
                fn = getattr(handle, name)
                fn.restype = res
                fn.argtypes = args
            _lib = handle
        return _lib


def declared_symbols(header: str = HEADER_PATH):
    """Function names declared in include/pifa.h."""
    with open(header) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) - {"defined"})


# ---------------------------------------------------------------- marshalling
def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return PIFA_BF16
    if t.dtype == torch.float32:
        return PIFA_F32
    raise TypeError("unsupported dtype %s (bf16 or fp32)" % t.dtype)


def _dev_ptr(t, name: str) -> int | None:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t.data_ptr()


# Dimensions of the live handles created through this module.  The library
# takes raw pointers and cannot see how large a tensor is, so the calls below
# check that each buffer holds the bytes the call will read or write (a short
# buffer would be accessed past its end on the GPU).  Handles created
# elsewhere are passed through unchecked.
_dims: dict = {}
_dims_lock = threading.Lock()


def _esize(dt: int) -> int:
    return 2 if dt == PIFA_BF16 else 4


def _need(t, nbytes: int, name: str) -> None:
    if t is not None and t.numel() * t.element_size() < nbytes:
        raise ValueError("%s holds %d bytes, the call needs %d" % (name, t.numel() * t.element_size(), nbytes))


def _torch_dtype(dt: int):
    import torch
    return {PIFA_BF16: torch.bfloat16, PIFA_F32: torch.float32}.get(dt, torch.float64 if dt == "f64" else None)


def _same(t, name: str, dt, device=None) -> None:
    """t (if given) has element type dt (PIFA_BF16, PIFA_F32 or "f64") and lives
    on the given device index: the library reads raw bytes, so a tensor of
    another type or on another GPU would be misread, not rejected."""
    if t is None:
        return
    want = _torch_dtype(dt)
    if want is not None and t.dtype != want:
        raise TypeError("%s is %s, the call expects %s" % (name, t.dtype, want))
    if device is not None and t.is_cuda and t.device.index != device:
        raise ValueError("%s is on cuda:%d, the handle on cuda:%d" % (name, t.device.index, device))


def _device_of(t):
    return t.device.index if (t is not None and t.is_cuda) else None


def _remember(handle: int, **dims) -> int:
    with _dims_lock:
        _dims[handle] = dims
    return handle


def _recall(handle: int):
    with _dims_lock:
        return _dims.get(handle)


def _forget(handle: int) -> None:
    with _dims_lock:
        _dims.pop(handle, None)


def _check_io(handle: int, X, Y, M: int) -> None:
    d = _recall(handle)
    if d is not None:
        _same(X, "X", d["dt"], d.get("dev"))
        _same(Y, "Y", d["dt"], d.get("dev"))
    if d is not None and M > 0:
        _need(X, M * d["d_in"] * _esize(d["dt"]), "X")
        _need(Y, M * d["d_out"] * _esize(d["dt"]), "Y")


def _host_i32(a):
    if a is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(a), dtype=np.int32)
    return arr, arr.ctypes.data_as(_i32p)


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return int(getattr(stream, "cuda_stream", stream))


def _check(fn: str, status: int):
    if status != PIFA_OK:
        raise PifaError(fn, status)


# ---------------------------------------------------------------- entry points
def pifa_status_string(status: int) -> str:
    return lib().pifa_status_string(int(status)).decode()


def pifa_gemm_plan(M: int, N: int, K: int, wide_epilogue: bool = True):
    """(tile_m, tile_n, k_splits) of a prefill product of M x N outputs over K
    (host only).  Raises on an invalid size."""
    tm, tn, ks = _i64(), _i64(), _i64()
    _check("pifa_gemm_plan", lib().pifa_gemm_plan(int(M), int(N), int(K), int(bool(wide_epilogue)), ctypes.byref(tm),
                                                  ctypes.byref(tn), ctypes.byref(ks)))
    return tm.value, tn.value, ks.value


def pifa_validate_partition(pivot_idx, nonpivot_idx, dims) -> int:
    """Returns the status code (no exception): PIFA_OK or the error."""
    piv, pp = _host_i32(pivot_idx)
    npv, npp = _host_i32(nonpivot_idx)
    return int(lib().pifa_validate_partition(pp, npp, pifa_dims(*dims)))


def pifa_layer_create(W_p, C, pivot_idx, nonpivot_idx, dims, dtype: int | None = None) -> int:
    """dims = (d_in, d_out, r); returns an opaque handle."""
    dt = _dtype_code(W_p) if dtype is None else int(dtype)
    piv, pp = _host_i32(pivot_idx)
    npv, npp = _host_i32(nonpivot_idx)
    d_in, d_out, r = (int(v) for v in dims)
    dev = _device_of(W_p)
    _same(W_p, "W_p", dt, dev)
    _same(C, "C", dt, dev)
    _need(W_p, r * d_in * _esize(dt), "W_p")
    _need(C, max(d_out - r, 0) * r * _esize(dt), "C")
    out = _vp()
    _check("pifa_layer_create", lib().pifa_layer_create(
        _dev_ptr(W_p, "W_p"), _dev_ptr(C, "C"), pp, npp, pifa_dims(*dims), dt, ctypes.byref(out)))
    return _remember(out.value, d_in=d_in, d_out=d_out, r=r, dt=dt, dev=dev)


def pifa_layer_destroy(handle: int) -> None:
    _forget(handle)
    _check("pifa_layer_destroy", lib().pifa_layer_destroy(handle))


def pifa_layer_reserve(handle: int, max_M: int) -> None:
    _check("pifa_layer_reserve", lib().pifa_layer_reserve(handle, int(max_M)))


def pifa_forward(handle: int, X, Y, M: int | None = None, stream=None) -> None:
    M = X.shape[0] if M is None else int(M)
    _check_io(handle, X, Y, M)
    _check("pifa_forward", lib().pifa_forward(handle, _dev_ptr(X, "X"), _dev_ptr(Y, "Y"), M,
                                              _stream(stream)))


def pifa_forward_noalloc(handle: int, X, Y, M: int | None = None, stream=None) -> None:
    """pifa_forward with the library's fixed per-GPU scratch as workspace (no
    allocation; calls on one GPU must not overlap)."""
    M = X.shape[0] if M is None else int(M)
    _check_io(handle, X, Y, M)
    _check("pifa_forward_noalloc", lib().pifa_forward_noalloc(handle, _dev_ptr(X, "X"), _dev_ptr(Y, "Y"), M,
                                                              _stream(stream)))


def pifa_layer_weight_bytes(handle: int) -> int:
    return int(lib().pifa_layer_weight_bytes(handle))


def pifa_layer_set_intermediate_scale(handle: int, log2_scale: int) -> None:
    _check("pifa_layer_set_intermediate_scale",
           lib().pifa_layer_set_intermediate_scale(handle, int(log2_scale)))


def pifa_layer_overflow_count(handle: int) -> int:
    out = _i64()
    _check("pifa_layer_overflow_count", lib().pifa_layer_overflow_count(handle, ctypes.byref(out)))
    return int(out.value)


def pifa_layer_backward(handle: int, X, Y, dY, dX=None, dW_p=None, dC=None, M: int | None = None,
                        stream=None) -> None:
    """Gradients of the layer: dX (bf16 M x d_in), dW_p (fp32 r x d_in), dC (fp32 (d_out-r) x r);
    each output may be None to skip it."""
    M = dY.shape[0] if M is None else int(M)
    d = _recall(handle)
    if d is not None:
        for t, name in ((X, "X"), (Y, "Y"), (dY, "dY"), (dX, "dX")):
            _same(t, name, PIFA_BF16, d.get("dev"))
        _same(dW_p, "dW_p", PIFA_F32, d.get("dev"))
        _same(dC, "dC", PIFA_F32, d.get("dev"))
    if d is not None and M > 0:  # bf16 activations and gradients, fp32 weight gradients
        for t, n, name in ((X, M * d["d_in"], "X"), (Y, M * d["d_out"], "Y"), (dY, M * d["d_out"], "dY"),
                           (dX, M * d["d_in"], "dX")):
            _need(t, 2 * n, name)
        _need(dW_p, 4 * d["r"] * d["d_in"], "dW_p")
        _need(dC, 4 * (d["d_out"] - d["r"]) * d["r"], "dC")
    _check("pifa_layer_backward", lib().pifa_layer_backward(
        handle, _dev_ptr(X, "X"), _dev_ptr(Y, "Y"), _dev_ptr(dY, "dY"), M, _dev_ptr(dX, "dX"),
        _dev_ptr(dW_p, "dW_p"), _dev_ptr(dC, "dC"), _stream(stream)))


def dense_forward(W, X, Y, M: int | None = None, d_in: int | None = None, d_out: int | None = None,
                  dtype: int | None = None, stream=None) -> None:
    M = X.shape[0] if M is None else int(M)
    d_in = W.shape[1] if d_in is None else int(d_in)
    d_out = W.shape[0] if d_out is None else int(d_out)
    dt = _dtype_code(W) if dtype is None else int(dtype)
    for t, name in ((W, "W"), (X, "X"), (Y, "Y")):
        _same(t, name, dt, _device_of(W))
    if M > 0:
        _need(W, d_out * d_in * _esize(dt), "W")
        _need(X, M * d_in * _esize(dt), "X")
        _need(Y, M * d_out * _esize(dt), "Y")
    _check("dense_forward", lib().dense_forward(_dev_ptr(W, "W"), _dev_ptr(X, "X"), _dev_ptr(Y, "Y"),
                                                M, d_in, d_out, dt, _stream(stream)))


def dense_layer_create(W, d_in: int | None = None, d_out: int | None = None,
                       dtype: int | None = None) -> int:
    d_in = W.shape[1] if d_in is None else int(d_in)
    d_out = W.shape[0] if d_out is None else int(d_out)
    dt = _dtype_code(W) if dtype is None else int(dtype)
    _same(W, "W", dt)
    _need(W, d_out * d_in * _esize(dt), "W")
    out = _vp()
    _check("dense_layer_create", lib().dense_layer_create(_dev_ptr(W, "W"), d_in, d_out, dt,
                                                          ctypes.byref(out)))
    return _remember(out.value, d_in=d_in, d_out=d_out, dt=dt, dev=_device_of(W))


def dense_layer_forward(handle: int, X, Y, M: int | None = None, stream=None) -> None:
    M = X.shape[0] if M is None else int(M)
    _check_io(handle, X, Y, M)
    _check("dense_layer_forward", lib().dense_layer_forward(handle, _dev_ptr(X, "X"), _dev_ptr(Y, "Y"), M,
                                                            _stream(stream)))


def dense_layer_reserve(handle: int, max_M: int) -> None:
    _check("dense_layer_reserve", lib().dense_layer_reserve(handle, int(max_M)))


def dense_layer_destroy(handle: int) -> None:
    _forget(handle)
    _check("dense_layer_destroy", lib().dense_layer_destroy(handle))


def lowrank_uv_forward(U, V, X, Y, M: int | None = None, dims=None, dtype: int | None = None,
                       stream=None) -> None:
    M = X.shape[0] if M is None else int(M)
    dims = (V.shape[1], U.shape[0], U.shape[1]) if dims is None else dims
    dt = _dtype_code(U) if dtype is None else int(dtype)
    d_in, d_out, r = (int(v) for v in dims)
    for t, name in ((U, "U"), (V, "V"), (X, "X"), (Y, "Y")):
        _same(t, name, dt, _device_of(U))
    if M > 0:
        _need(U, d_out * r * _esize(dt), "U")
        _need(V, r * d_in * _esize(dt), "V")
        _need(X, M * d_in * _esize(dt), "X")
        _need(Y, M * d_out * _esize(dt), "Y")
    _check("lowrank_uv_forward", lib().lowrank_uv_forward(
        _dev_ptr(U, "U"), _dev_ptr(V, "V"), _dev_ptr(X, "X"), _dev_ptr(Y, "Y"), M, pifa_dims(*dims),
        dt, _stream(stream)))


def lowrank_layer_create(U, V, dims=None, dtype: int | None = None) -> int:
    dims = (V.shape[1], U.shape[0], U.shape[1]) if dims is None else dims
    dt = _dtype_code(U) if dtype is None else int(dtype)
    d_in, d_out, r = (int(v) for v in dims)
    _same(U, "U", dt, _device_of(U))
    _same(V, "V", dt, _device_of(U))
    _need(U, d_out * r * _esize(dt), "U")
    _need(V, r * d_in * _esize(dt), "V")
    out = _vp()
    _check("lowrank_layer_create", lib().lowrank_layer_create(
        _dev_ptr(U, "U"), _dev_ptr(V, "V"), pifa_dims(*dims), dt, ctypes.byref(out)))
    return _remember(out.value, d_in=d_in, d_out=d_out, dt=dt, dev=_device_of(U))


def lowrank_layer_forward(handle: int, X, Y, M: int | None = None, stream=None) -> None:
    M = X.shape[0] if M is None else int(M)
    _check_io(handle, X, Y, M)
    _check("lowrank_layer_forward", lib().lowrank_layer_forward(
        handle, _dev_ptr(X, "X"), _dev_ptr(Y, "Y"), M, _stream(stream)))


def lowrank_layer_reserve(handle: int, max_M: int) -> None:
    _check("lowrank_layer_reserve", lib().lowrank_layer_reserve(handle, int(max_M)))


def lowrank_layer_destroy(handle: int) -> None:
    _forget(handle)
    _check("lowrank_layer_destroy", lib().lowrank_layer_destroy(handle))


def pifa_group_create(layers, dtype: int | None = None) -> int:
    """layers: sequence of (W_p, C, pivot_idx, nonpivot_idx, (d_in, d_out, r)) with one d_in;
    returns an opaque group handle."""
    n = len(layers)
    wp = (_vp * max(n, 1))()
    cc = (_vp * max(n, 1))()
    pp = (_i32p * max(n, 1))()
    npp = (_i32p * max(n, 1))()
    dims = (pifa_dims * max(n, 1))()
    keep = []
    dt = (_dtype_code(layers[0][0]) if n else PIFA_BF16) if dtype is None else int(dtype)
    dev = _device_of(layers[0][0]) if n else None
    for i, (W_p, C, piv, npiv, d) in enumerate(layers):
        if dt == PIFA_BF16:  # the only group dtype; the library rejects the others
            _same(W_p, "W_p", dt, dev)
            _same(C, "C", dt, dev)
            _need(W_p, int(d[2]) * int(d[0]) * 2, "W_p")
            _need(C, max(int(d[1]) - int(d[2]), 0) * int(d[2]) * 2, "C")
        wp[i] = _dev_ptr(W_p, "W_p")
        cc[i] = _dev_ptr(C, "C")
        a, ap = _host_i32(piv)
        b, bp = _host_i32(npiv)
        keep += [a, b]
        pp[i] = ap
        npp[i] = bp
        dims[i] = pifa_dims(*d)
    out = _vp()
    _check("pifa_group_create", lib().pifa_group_create(n, wp, cc, pp, npp, dims, dt, ctypes.byref(out)))
    return _remember(out.value, d_in=int(layers[0][4][0]), d_out=sum(int(l[4][1]) for l in layers), dt=dt,
                     dev=dev)


def pifa_group_destroy(handle: int) -> None:
    _forget(handle)
    _check("pifa_group_destroy", lib().pifa_group_destroy(handle))


def pifa_group_reserve(handle: int, max_M: int) -> None:
    _check("pifa_group_reserve", lib().pifa_group_reserve(handle, int(max_M)))


def pifa_group_forward(handle: int, X, Y, M: int | None = None, stream=None) -> None:
    M = X.shape[0] if M is None else int(M)
    _check_io(handle, X, Y, M)
    _check("pifa_group_forward", lib().pifa_group_forward(handle, _dev_ptr(X, "X"), _dev_ptr(Y, "Y"), M,
                                                          _stream(stream)))


def pifa_group_weight_bytes(handle: int) -> int:
    return int(lib().pifa_group_weight_bytes(handle))


def pifa_group_set_intermediate_scale(handle: int, log2_scale: int) -> None:
    _check("pifa_group_set_intermediate_scale",
           lib().pifa_group_set_intermediate_scale(handle, int(log2_scale)))


def pifa_group_overflow_count(handle: int) -> int:
    out = _i64()
    _check("pifa_group_overflow_count", lib().pifa_group_overflow_count(handle, ctypes.byref(out)))
    return int(out.value)


def pifa_calib_create(d_in: int) -> int:
    out = _vp()
    _check("pifa_calib_create", lib().pifa_calib_create(int(d_in), ctypes.byref(out)))
    return _remember(out.value, n=int(d_in))


def pifa_calib_destroy(handle: int) -> None:
    _forget(handle)
    _check("pifa_calib_destroy", lib().pifa_calib_destroy(handle))


def pifa_calib_reset(handle: int, stream=None) -> None:
    _check("pifa_calib_reset", lib().pifa_calib_reset(handle, _stream(stream)))


def pifa_calib_accumulate(handle: int, X_o, X_u, B: int | None = None, stream=None) -> None:
    B = X_u.shape[0] if B is None else int(B)
    d = _recall(handle)
    if d is not None:
        _same(X_o, "X_o", PIFA_BF16)
        _same(X_u, "X_u", PIFA_BF16)
    if d is not None and B > 0:
        _need(X_o, 2 * B * d["n"], "X_o")
        _need(X_u, 2 * B * d["n"], "X_u")
    _check("pifa_calib_accumulate", lib().pifa_calib_accumulate(handle, _dev_ptr(X_o, "X_o"), _dev_ptr(X_u, "X_u"),
                                                                B, _stream(stream)))


def pifa_calib_read(handle: int, S=None, P=None, stream=None) -> None:
    d = _recall(handle)
    _same(S, "S", "f64")
    _same(P, "P", "f64")
    if d is not None:
        _need(S, 8 * d["n"] * d["n"], "S")
        _need(P, 8 * d["n"] * d["n"], "P")
    _check("pifa_calib_read", lib().pifa_calib_read(handle, _dev_ptr(S, "S"), _dev_ptr(P, "P"), _stream(stream)))


def pifa_calib_reconstruct(handle: int, W, Vt, lam: float, alpha: float, U_r=None, Vt_r=None, stream=None):
    """Returns (U_r, Vt_r) as device fp64 tensors (allocated when not given)."""
    import torch
    d_out, d_in = W.shape
    r = Vt.shape[0]
    if U_r is None:
        U_r = torch.empty((d_out, r), dtype=torch.float64, device=W.device)
    if Vt_r is None:
        Vt_r = torch.empty((r, d_in), dtype=torch.float64, device=W.device)
    for t, name in ((W, "W"), (Vt, "Vt"), (U_r, "U_r"), (Vt_r, "Vt_r")):
        _same(t, name, "f64", _device_of(W))
    d = _recall(handle)
    if d is not None:
        n = d["n"]
        for t, nb, name in ((W, d_out * n, "W"), (Vt, r * n, "Vt"), (U_r, d_out * r, "U_r"), (Vt_r, r * n, "Vt_r")):
            _need(t, 8 * nb, name)
    _check("pifa_calib_reconstruct", lib().pifa_calib_reconstruct(
        handle, _dev_ptr(W, "W"), int(d_out), _dev_ptr(Vt, "Vt"), int(r), float(lam), float(alpha),
        _dev_ptr(U_r, "U_r"), _dev_ptr(Vt_r, "Vt_r"), _stream(stream)))
    return U_r, Vt_r


def pifa_build_f64(W, r: int, stream=None):
    """Algorithm "Pivoting Factorization" on the GPU for a device fp64 W'
    (d_out x d_in).  Returns (pivot_idx, nonpivot_idx, W_p, C, report) with
    sorted numpy index arrays, device fp64 W_p / C, and the 4-entry report."""
    import torch
    if W.dtype != torch.float64:
        raise TypeError("W must be float64")
    d_out, d_in = W.shape
    r = int(r)
    Wp = torch.empty((r, d_in), dtype=torch.float64, device=W.device)
    C = torch.empty((d_out - r, r), dtype=torch.float64, device=W.device)
    piv = np.zeros(r, np.int32)
    npiv = np.zeros(max(d_out - r, 0), np.int32)
    report = (ctypes.c_double * 4)()
    npp = npiv.ctypes.data_as(_i32p) if npiv.size else None
    _check("pifa_build_f64", lib().pifa_build_f64(
        _dev_ptr(W, "W"), pifa_dims(d_in, d_out, r), _dev_ptr(Wp, "W_p"), C.data_ptr() if C.numel() else None,
        piv.ctypes.data_as(_i32p), npp, report, _stream(stream)))
    return piv, npiv, Wp, C, np.array(list(report))


def pifa_probe_mfma(iters: int = 20000, stream=None):
    """(dense bf16 MFMA TFLOP/s, shader clock in MHz) of an MFMA-only kernel."""
    tf, mhz = ctypes.c_double(), ctypes.c_double()
    _check("pifa_probe_mfma", lib().pifa_probe_mfma(int(iters), ctypes.byref(tf), ctypes.byref(mhz),
                                                    _stream(stream)))
    return tf.value, mhz.value


def pifa_probe_mfma_random(iters: int = 20000, stream=None):
    """(dense bf16 MFMA TFLOP/s, shader clock in MHz) of an MFMA-only kernel
    whose operands change with every MFMA (random bf16 values)."""
    tf, mhz = ctypes.c_double(), ctypes.c_double()
    _check("pifa_probe_mfma_random", lib().pifa_probe_mfma_random(int(iters), ctypes.byref(tf), ctypes.byref(mhz),
                                                                  _stream(stream)))
    return tf.value, mhz.value


def pifa_probe_hbm_read(buf, reps: int = 5, stream=None) -> float:
    """GB/s of `reps` streaming reads of the device tensor `buf`."""
    nbytes = (buf.numel() * buf.element_size()) // 16 * 16
    out = ctypes.c_double()
    _check("pifa_probe_hbm_read", lib().pifa_probe_hbm_read(_dev_ptr(buf, "buf"), nbytes, int(reps),
                                                            ctypes.byref(out), _stream(stream)))
    return out.value


def pifa_profile_enable(on: bool) -> None:
    _check("pifa_profile_enable", lib().pifa_profile_enable(1 if on else 0))


def pifa_profile_reset() -> None:
    _check("pifa_profile_reset", lib().pifa_profile_reset())


def pifa_profile_read(max_sites: int = 32) -> dict:
    """{site name: (launches, total milliseconds)} since the last reset."""
    names = (ctypes.c_char_p * max_sites)()
    launches = (_i64 * max_sites)()
    ms = (ctypes.c_double * max_sites)()
    n = ctypes.c_int()
    _check("pifa_profile_read", lib().pifa_profile_read(names, launches, ms, max_sites, ctypes.byref(n)))
    return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(n.value)}


# ---------------------------------------------------------------- convenience
class PifaLayer:
    """Owns a pifa_handle; ``layer(X)`` allocates Y and runs pifa_forward."""

    def __init__(self, W_p, C, pivot_idx, nonpivot_idx, d_out: int):
        self.d_in = int(W_p.shape[1])
        self.r = int(W_p.shape[0])
        self.d_out = int(d_out)
        self.dtype = W_p.dtype
        self.handle = pifa_layer_create(W_p, C, pivot_idx, nonpivot_idx, (self.d_in, self.d_out, self.r))

    def __call__(self, X, Y=None, stream=None):
        import torch
        if Y is None:
            Y = torch.empty((X.shape[0], self.d_out), dtype=X.dtype, device=X.device)
        pifa_forward(self.handle, X, Y, X.shape[0], stream)
        return Y

    def close(self):
        if self.handle:
            pifa_layer_destroy(self.handle)
            self.handle = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
