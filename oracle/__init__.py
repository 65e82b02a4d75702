"""PIFA oracle -- TEST INFRASTRUCTURE ONLY.

Plain fp64 CPU implementation of Pivoting Factorization (arXiv 2501.19090):
the build of Algorithm "Pivoting Factorization" (Sec. 3.2) and the forward
pass of Algorithm "PIFA Layer", plus the dense and low-rank layers of
Sec. 3.3.  The arithmetic lives in ``pifa_oracle.c`` (plain loops, OpenMP
only across independent rows/columns); this module only marshals numpy
arrays to it.

Only ``tests/``, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU library never calls it, and it never calls the
GPU library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pifa_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

ORACLE_OK = 0
ORACLE_NOT_RANK_R = 1


def compile_oracle(force: bool = False) -> str:
    """Compile ``pifa_oracle.c`` into ``liboracle.so`` with gcc (-O2, OpenMP)."""
    stale = (not os.path.exists(_LIB_PATH)
             or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC))
    if force or stale:
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        compile_oracle()
        lib = ctypes.CDLL(_LIB_PATH)
        i64, i32p, f64p = ctypes.c_int64, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)
        lib.oracle_pifa_build.restype = ctypes.c_int
        lib.oracle_pifa_build.argtypes = [f64p, i64, i64, i64, ctypes.c_int, i32p, i32p,
                                          f64p, f64p, i32p, f64p]
        lib.oracle_pifa_forward.restype = None
        lib.oracle_pifa_forward.argtypes = [f64p, i64, i64, i64, i64, i32p, i32p, f64p, f64p,
                                            f64p, ctypes.c_int]
        lib.oracle_dense_forward.restype = None
        lib.oracle_dense_forward.argtypes = [f64p, f64p, i64, i64, i64, f64p, ctypes.c_int]
        lib.oracle_lowrank_forward.restype = None
        lib.oracle_lowrank_forward.argtypes = [f64p, f64p, f64p, i64, i64, i64, i64, f64p,
                                               ctypes.c_int]
        lib.oracle_pifa_backward.restype = None
        lib.oracle_pifa_backward.argtypes = [f64p, f64p, i64, i64, i64, i64, i32p, i32p, f64p, f64p, f64p,
                                             f64p, f64p, ctypes.c_int]
        lib.oracle_reconstruction_error.restype = ctypes.c_double
        lib.oracle_reconstruction_error.argtypes = [f64p, i64, i64, i64, i32p, i32p, f64p, f64p,
                                                    ctypes.c_int]
        lib.oracle_set_progress.restype = None
        lib.oracle_set_progress.argtypes = [i64]
        lib.oracle_max_threads.restype = ctypes.c_int
        lib.oracle_max_threads.argtypes = []
        _lib = lib
        return lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _p(a, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


def default_threads() -> int:
    """Threads the oracle uses when none are given (OpenMP's default)."""
    return int(_load().oracle_max_threads())


class OracleRankError(ValueError):
    """The input W' does not have numerical rank exactly r."""


def build_pifa(W, r: int, threads: int | None = None, progress: int = 0) -> dict:
    """Pivoting Factorization of a rank-r matrix W' (d_out x d_in).

    Returns a dict with ``pivot_idx`` (sorted I), ``nonpivot_idx`` (sorted
    I^c), ``Wp`` = W'[I, :], ``C`` with W'[I^c, :] = C W_p, ``select_order``
    (pivots in QRCP selection order) and ``report`` (|R_00|, |R_{r-1,r-1}|,
    largest residual norm after r steps, certification flag).
    Raises OracleRankError if W' is not numerically of rank r.
    progress > 0 prints a line to stderr every `progress` pivoting steps
    (long builds); it does not change the result.
    """
    lib = _load()
    W = _f64(W)
    d_out, d_in = W.shape
    r = int(r)
    piv = np.zeros(r, np.int32)
    npiv = np.zeros(max(d_out - r, 0), np.int32)
    Wp = np.zeros((r, d_in), np.float64)
    C = np.zeros((max(d_out - r, 0), r), np.float64)
    order = np.zeros(r, np.int32)
    report = np.zeros(4, np.float64)
    nt = threads if threads is not None else default_threads()
    # a 1-element dummy keeps the pointer valid when C is empty
    Cbuf = C if C.size else np.zeros(1, np.float64)
    npbuf = npiv if npiv.size else np.zeros(1, np.int32)
    with _lock:
        lib.oracle_set_progress(int(progress))
        try:
            st = lib.oracle_pifa_build(_p(W, ctypes.c_double), d_out, d_in, r, int(nt),
                                       _p(piv, ctypes.c_int32), _p(npbuf, ctypes.c_int32),
                                       _p(Wp, ctypes.c_double), _p(Cbuf, ctypes.c_double),
                                       _p(order, ctypes.c_int32), _p(report, ctypes.c_double))
        finally:
            lib.oracle_set_progress(0)
    if st == ORACLE_NOT_RANK_R:
        raise OracleRankError("input is not numerically of rank %d (report=%s)" % (r, report))
    if st != ORACLE_OK:
        raise ValueError("oracle_pifa_build failed with status %d" % st)
    return {"pivot_idx": piv, "nonpivot_idx": npiv, "Wp": Wp, "C": C,
            "select_order": order, "report": report}


def pifa_forward(X, pivot_idx, nonpivot_idx, Wp, C, d_out: int | None = None,
                 threads: int | None = None) -> np.ndarray:
    """Algorithm "PIFA Layer" in fp64 for row-major X (M x d_in) -> Y (M x d_out)."""
    lib = _load()
    X, Wp = _f64(X), _f64(Wp)
    piv, npiv = _i32(pivot_idx), _i32(nonpivot_idx)
    M, d_in = X.shape
    r = Wp.shape[0]
    d_out = r + npiv.size if d_out is None else int(d_out)
    C = _f64(C).reshape(d_out - r, r)
    Y = np.zeros((M, d_out), np.float64)
    nt = threads if threads is not None else default_threads()
    Cbuf = C if C.size else np.zeros(1, np.float64)
    npbuf = npiv if npiv.size else np.zeros(1, np.int32)
    lib.oracle_pifa_forward(_p(X, ctypes.c_double), M, d_in, d_out, r,
                            _p(piv, ctypes.c_int32), _p(npbuf, ctypes.c_int32),
                            _p(Wp, ctypes.c_double), _p(Cbuf, ctypes.c_double),
                            _p(Y, ctypes.c_double), int(nt))
    return Y


def group_forward(X, layers, threads: int | None = None) -> np.ndarray:
    """Layers that read the same X, their outputs side by side: the block
    [Y_1 | Y_2 | ...] with Y_i = Algorithm "PIFA Layer" of layer i.
    layers: sequence of (pivot_idx, nonpivot_idx, Wp, C)."""
    outs = [pifa_forward(X, piv, npiv, Wp, C, threads=threads) for piv, npiv, Wp, C in layers]
    return np.concatenate(outs, axis=1) if outs else np.zeros((np.shape(X)[0], 0))


def pifa_backward(X, G, pivot_idx, nonpivot_idx, Wp, C, threads: int | None = None):
    """Gradients of Algorithm "PIFA Layer" for G = dL/dY: returns (dX, dWp, dC)."""
    lib = _load()
    X, G, Wp = _f64(X), _f64(G), _f64(Wp)
    piv, npiv = _i32(pivot_idx), _i32(nonpivot_idx)
    M, d_in = X.shape
    r = Wp.shape[0]
    d_out = G.shape[1]
    C = _f64(C).reshape(d_out - r, r)
    dX = np.zeros((M, d_in), np.float64)
    dWp = np.zeros((r, d_in), np.float64)
    dC = np.zeros((d_out - r, r), np.float64)
    nt = threads if threads is not None else default_threads()
    Cbuf = C if C.size else np.zeros(1, np.float64)
    dCbuf = dC if dC.size else np.zeros(1, np.float64)
    npbuf = npiv if npiv.size else np.zeros(1, np.int32)
    lib.oracle_pifa_backward(_p(X, ctypes.c_double), _p(G, ctypes.c_double), M, d_in, d_out, r,
                             _p(piv, ctypes.c_int32), _p(npbuf, ctypes.c_int32), _p(Wp, ctypes.c_double),
                             _p(Cbuf, ctypes.c_double), _p(dX, ctypes.c_double), _p(dWp, ctypes.c_double),
                             _p(dCbuf, ctypes.c_double), int(nt))
    return dX, dWp, dC


def dense_forward(X, W, threads: int | None = None) -> np.ndarray:
    """Dense layer Y = X W^T in fp64."""
    lib = _load()
    X, W = _f64(X), _f64(W)
    M, d_in = X.shape
    d_out = W.shape[0]
    Y = np.zeros((M, d_out), np.float64)
    nt = threads if threads is not None else default_threads()
    lib.oracle_dense_forward(_p(X, ctypes.c_double), _p(W, ctypes.c_double), M, d_in, d_out,
                             _p(Y, ctypes.c_double), int(nt))
    return Y


def lowrank_forward(X, U, V, threads: int | None = None) -> np.ndarray:
    """Low-rank layer Y = (X V^T) U^T in fp64; U is d_out x r, V is r x d_in."""
    lib = _load()
    X, U, V = _f64(X), _f64(U), _f64(V)
    M, d_in = X.shape
    d_out, r = U.shape
    Y = np.zeros((M, d_out), np.float64)
    nt = threads if threads is not None else default_threads()
    lib.oracle_lowrank_forward(_p(X, ctypes.c_double), _p(U, ctypes.c_double),
                               _p(V, ctypes.c_double), M, d_in, d_out, r,
                               _p(Y, ctypes.c_double), int(nt))
    return Y


def reconstruction_error(W, pivot_idx, nonpivot_idx, Wp, C, threads: int | None = None) -> float:
    """|| P[W_p; C W_p] - W ||_F / ||W||_F for a PIFA layer of W."""
    lib = _load()
    W, Wp = _f64(W), _f64(Wp)
    piv, npiv = _i32(pivot_idx), _i32(nonpivot_idx)
    d_out, d_in = W.shape
    r = Wp.shape[0]
    C = _f64(C).reshape(d_out - r, r)
    nt = threads if threads is not None else default_threads()
    Cbuf = C if C.size else np.zeros(1, np.float64)
    npbuf = npiv if npiv.size else np.zeros(1, np.int32)
    return float(lib.oracle_reconstruction_error(
        _p(W, ctypes.c_double), d_out, d_in, r, _p(piv, ctypes.c_int32),
        _p(npbuf, ctypes.c_int32), _p(Wp, ctypes.c_double), _p(Cbuf, ctypes.c_double), int(nt)))
