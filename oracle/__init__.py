"""fp64 CPU oracle for the CoLA layer -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU product path never does, and
the two share no code: this package wraps ``cola_oracle.c`` (plain C loops in
fp64) with ctypes, nothing else.

Functions follow the paper's statement of the layer (Sec. 3.2, Eq. main-fwd),
its gradient rule (Sec. 3.4) and CoLA-M's saved set (Sec. 4.2, App. C).
All arrays are token-major (one token per row), fp64, C-contiguous.
"""
import ctypes
import os

import numpy as np

from .build import LIB, SRC, build

_lib = None
_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.c_int64


def _load(path=None):
    global _lib
    if _lib is not None and path is None:
        return _lib
    if path is None:
        path = LIB
        # (re)build when missing or older than its source
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(SRC):
            build()
    lib = ctypes.CDLL(path)
    i64, d, c_int = _I64, _D, ctypes.c_int
    lib.oracle_sigma.argtypes = [c_int, ctypes.c_double]
    lib.oracle_sigma.restype = ctypes.c_double
    lib.oracle_sigma_prime.argtypes = [c_int, ctypes.c_double]
    lib.oracle_sigma_prime.restype = ctypes.c_double
    lib.oracle_reset_macs.argtypes = []
    lib.oracle_macs.restype = ctypes.c_int64
    lib.oracle_num_threads.restype = c_int
    lib.oracle_set_threads.argtypes = [c_int]
    lib.oracle_cola_fwd.argtypes = [i64, i64, i64, i64, c_int, d, d, d, d, d, d]
    lib.oracle_cola_bwd.argtypes = [i64, i64, i64, i64, c_int, d, d, d, d, d,
                                    d, d, d, d, d]
    lib.oracle_cola_fwd_outer.argtypes = [i64, i64, i64, i64, c_int, c_int, d, d, d, d, d, d, d]
    lib.oracle_cola_bwd_outer.argtypes = [i64, i64, i64, i64, c_int, c_int, d, d, d, d, d, d,
                                          d, d, d, d, d, d]
    lib.oracle_dense_fwd.argtypes = [i64, i64, i64, d, d, d]
    lib.oracle_dense_bwd.argtypes = [i64, i64, i64, d, d, d, d, d]
    lib.oracle_cola_rows.argtypes = [i64, i64, i64, i64, c_int, d, d, d, d,
                                     i64, ctypes.POINTER(ctypes.c_int64),
                                     d, d, d, d, d]
    lib.oracle_cola_wgrad_cols.argtypes = [i64, i64, i64, i64, c_int, d, d, d, d,
                                           i64, ctypes.POINTER(ctypes.c_int64), d, d]
    lib.oracle_cola_wgrad_cols.restype = c_int
    lib.oracle_cola_up_from_z.argtypes = [i64, i64, i64, c_int, d, d, d, d]
    lib.oracle_dense_rows.argtypes = [i64, i64, i64, d, d, d, i64, ctypes.POINTER(ctypes.c_int64), d, d]
    lib.oracle_dense_wgrad_rows.argtypes = [i64, i64, i64, d, d, i64, ctypes.POINTER(ctypes.c_int64), d]
    _lib = lib
    return lib


def use_library(path=None):
    """Point the wrapper at another build of cola_oracle.c (the mutation tests
    load deliberately broken copies); ``None`` restores the real oracle."""
    global _lib
    _lib = None
    if path is not None:
        _load(path)


ACT = {"identity": 0, "silu": 1, "gelu": 2}


def _act(act):
    return ACT[act] if isinstance(act, str) else int(act)


def _f64(a, shape=None):
    a = np.ascontiguousarray(a, dtype=np.float64)
    if shape is not None and a.shape != tuple(shape):
        raise ValueError(f"expected shape {tuple(shape)}, got {a.shape}")
    return a


def _p(a):
    return a.ctypes.data_as(_D)


def sigma(act, z):
    return _load().oracle_sigma(_act(act), float(z))


def sigma_prime(act, z):
    return _load().oracle_sigma_prime(_act(act), float(z))


def reset_macs():
    _load().oracle_reset_macs()


def macs():
    return int(_load().oracle_macs())


def num_threads():
    return int(_load().oracle_num_threads())


def set_threads(n):
    _load().oracle_set_threads(int(n))


def cola_fwd(X, A, B, act="silu"):
    """Z = X A^T, H = sigma(Z), Y = H B^T.  Returns (Z, H, Y)."""
    X = _f64(X); A = _f64(A); B = _f64(B)
    T, d_in = X.shape
    r = A.shape[0]
    d_out = B.shape[0]
    _f64(A, (r, d_in)); _f64(B, (d_out, r))
    Z = np.empty((T, r)); H = np.empty((T, r)); Y = np.empty((T, d_out))
    _load().oracle_cola_fwd(T, d_in, d_out, r, _act(act), _p(X), _p(A), _p(B),
                            _p(Z), _p(H), _p(Y))
    return Z, H, Y


def cola_bwd(X, Z, A, B, dY, act="silu"):
    """Gradients from the saved pre-activation Z.  Returns (dZ, dX, dA, dB)."""
    X = _f64(X); Z = _f64(Z); A = _f64(A); B = _f64(B); dY = _f64(dY)
    T, d_in = X.shape
    r = A.shape[0]
    d_out = B.shape[0]
    _f64(Z, (T, r)); _f64(dY, (T, d_out))
    dZ = np.empty((T, r)); dX = np.empty((T, d_in))
    dA = np.empty((r, d_in)); dB = np.empty((d_out, r))
    scratch = np.empty(2 * T * r)
    _load().oracle_cola_bwd(T, d_in, d_out, r, _act(act), _p(X), _p(Z), _p(A), _p(B),
                            _p(dY), _p(dZ), _p(dX), _p(dA), _p(dB), _p(scratch))
    return dZ, dX, dA, dB


def cola_fwd_outer(X, A, B, act="silu", outer="silu"):
    """The "both sigma" variant: Y = sigma_out(H B^T).  Returns (Z, H, P, Y),
    P = H B^T the output before sigma_out."""
    X = _f64(X); A = _f64(A); B = _f64(B)
    T, d_in = X.shape
    r = A.shape[0]
    d_out = B.shape[0]
    _f64(A, (r, d_in)); _f64(B, (d_out, r))
    Z = np.empty((T, r)); H = np.empty((T, r)); P = np.empty((T, d_out)); Y = np.empty((T, d_out))
    _load().oracle_cola_fwd_outer(T, d_in, d_out, r, _act(act), _act(outer), _p(X), _p(A), _p(B),
                                  _p(Z), _p(H), _p(P), _p(Y))
    return Z, H, P, Y


def cola_bwd_outer(X, Z, P, A, B, dY, act="silu", outer="silu"):
    """Gradients of the "both sigma" variant from the saved Z and P.
    Returns (dP, dZ, dX, dA, dB), dP = dY * sigma_out'(P)."""
    X = _f64(X); Z = _f64(Z); P = _f64(P); A = _f64(A); B = _f64(B); dY = _f64(dY)
    T, d_in = X.shape
    r = A.shape[0]
    d_out = B.shape[0]
    _f64(Z, (T, r)); _f64(P, (T, d_out)); _f64(dY, (T, d_out))
    dP = np.empty((T, d_out)); dZ = np.empty((T, r)); dX = np.empty((T, d_in))
    dA = np.empty((r, d_in)); dB = np.empty((d_out, r))
    scratch = np.empty(2 * T * r + T * d_out)
    _load().oracle_cola_bwd_outer(T, d_in, d_out, r, _act(act), _act(outer), _p(X), _p(Z), _p(P), _p(A),
                                  _p(B), _p(dY), _p(dP), _p(dZ), _p(dX), _p(dA), _p(dB), _p(scratch))
    return dP, dZ, dX, dA, dB


def dense_fwd(X, W):
    X = _f64(X); W = _f64(W)
    T, d_in = X.shape
    d_out = W.shape[0]
    _f64(W, (d_out, d_in))
    Y = np.empty((T, d_out))
    _load().oracle_dense_fwd(T, d_in, d_out, _p(X), _p(W), _p(Y))
    return Y


def dense_bwd(X, W, dY):
    X = _f64(X); W = _f64(W); dY = _f64(dY)
    T, d_in = X.shape
    d_out = W.shape[0]
    dX = np.empty((T, d_in)); dW = np.empty((d_out, d_in))
    _load().oracle_dense_bwd(T, d_in, d_out, _p(X), _p(W), _p(dY), _p(dX), _p(dW))
    return dX, dW


def cola_rows(X, A, B, dY, rows, act="silu"):
    """Z, H, Y, dZ, dX for the selected tokens only.  Returns a dict of [n][width]."""
    X = _f64(X); A = _f64(A); B = _f64(B); dY = _f64(dY)
    T, d_in = X.shape
    r = A.shape[0]
    d_out = B.shape[0]
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    if rows.size and (rows.min() < 0 or rows.max() >= T):
        raise ValueError("row index out of range")
    n = rows.size
    out = {k: np.empty((n, w)) for k, w in
           (("Z", r), ("H", r), ("Y", d_out), ("dZ", r), ("dX", d_in))}
    _load().oracle_cola_rows(T, d_in, d_out, r, _act(act), _p(X), _p(A), _p(B), _p(dY),
                             n, rows.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                             _p(out["Z"]), _p(out["H"]), _p(out["Y"]), _p(out["dZ"]),
                             _p(out["dX"]))
    return out


def cola_wgrad_cols(X, A, B, dY, cols, act="silu"):
    """Rows dA[j, :] and columns dB[:, j] for the selected rank indices j.
    Returns (dA_rows [n][d_in], dB_cols [n][d_out])."""
    X = _f64(X); A = _f64(A); B = _f64(B); dY = _f64(dY)
    T, d_in = X.shape
    r = A.shape[0]
    d_out = B.shape[0]
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    if cols.size and (cols.min() < 0 or cols.max() >= r):
        raise ValueError("rank index out of range")
    n = cols.size
    dA = np.empty((n, d_in)); dB = np.empty((n, d_out))
    rc = _load().oracle_cola_wgrad_cols(T, d_in, d_out, r, _act(act), _p(X), _p(A), _p(B),
                                        _p(dY), n,
                                        cols.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                        _p(dA), _p(dB))
    if rc != 0:
        raise MemoryError("oracle could not allocate its token columns")
    return dA, dB


def dense_rows(X, W, dY, rows):
    """Dense layer rows Y[t, :] and dX[t, :] for the selected tokens.
    Returns (Y_rows [n][d_out], dX_rows [n][d_in])."""
    X = _f64(X); W = _f64(W); dY = _f64(dY)
    T, d_in = X.shape
    d_out = W.shape[0]
    _f64(W, (d_out, d_in)); _f64(dY, (T, d_out))
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    if rows.size and (rows.min() < 0 or rows.max() >= T):
        raise ValueError("row index out of range")
    n = rows.size
    Y = np.empty((n, d_out)); dX = np.empty((n, d_in))
    _load().oracle_dense_rows(T, d_in, d_out, _p(X), _p(W), _p(dY), n,
                              rows.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _p(Y), _p(dX))
    return Y, dX


def dense_wgrad_rows(X, dY, outs):
    """Rows dW[o, :] = sum_t dY[t, o] X[t, :] for the selected output indices o."""
    X = _f64(X); dY = _f64(dY)
    T, d_in = X.shape
    d_out = dY.shape[1]
    outs = np.ascontiguousarray(outs, dtype=np.int64)
    if outs.size and (outs.min() < 0 or outs.max() >= d_out):
        raise ValueError("output index out of range")
    dW = np.empty((outs.size, d_in))
    _load().oracle_dense_wgrad_rows(T, d_in, d_out, _p(X), _p(dY), outs.size,
                                    outs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), _p(dW))
    return dW


def cola_up_from_z(Z, B, act="silu"):
    """CoLA-M's recompute from the saved pre-activation: H = sigma(Z), Y = H B^T.
    Returns (H, Y)."""
    Z = _f64(Z); B = _f64(B)
    T, r = Z.shape
    d_out = B.shape[0]
    _f64(B, (d_out, r))
    H = np.empty((T, r)); Y = np.empty((T, d_out))
    _load().oracle_cola_up_from_z(T, d_out, r, _act(act), _p(Z), _p(B), _p(H), _p(Y))
    return H, Y
