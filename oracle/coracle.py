"""ctypes binding of the C oracle (``libmdoracle.so``) -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use it.  Arrays are numpy, C-contiguous, limb-major.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build_oracle

_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)
_lp = ctypes.POINTER(ctypes.c_int64)
_i64 = ctypes.c_int64


def lib():
    """Load ``libmdoracle.so``, building it first if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(build_oracle.OUT):
            build_oracle.build()
        L = ctypes.CDLL(build_oracle.OUT)
        L.oracle_two_sum.argtypes = [_i64, _dp, _dp, _dp, _dp]
        L.oracle_fast_two_sum.argtypes = [_i64, _dp, _dp, _dp, _dp]
        L.oracle_two_prod.argtypes = [_i64, _dp, _dp, _dp, _dp]
        L.oracle_md_fma.argtypes = [ctypes.c_int, _i64, _dp, _dp, _dp, _dp]
        L.oracle_dd_add.argtypes = [_i64, _dp, _dp, _dp]
        L.oracle_dd_mul.argtypes = [_i64, _dp, _dp, _dp]
        L.oracle_classic_gemm.argtypes = [_i64, _i64, _i64, ctypes.c_int, _dp, _dp, _dp, _i64, _i64,
                                          ctypes.c_int, ctypes.c_int]
        L.oracle_classic_gemm.restype = ctypes.c_int
        L.oracle_exponents.argtypes = [_i64, _i64, ctypes.c_int, _dp, _ip]
        L.oracle_exponents.restype = ctypes.c_int
        L.oracle_split.argtypes = [_i64, _i64, ctypes.c_int, ctypes.c_int, ctypes.c_int, _dp, _ip, _dp]
        L.oracle_split.restype = ctypes.c_int
        L.oracle_split_bits.argtypes = [_i64, _i64, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, _dp, _ip,
                                        _dp]
        L.oracle_split_bits.restype = ctypes.c_int
        L.oracle_levels.argtypes = [_i64, _i64, _i64, ctypes.c_int, ctypes.c_int, ctypes.c_int, _dp, _dp, _lp]
        L.oracle_levels.restype = ctypes.c_int
        L.oracle_num_threads.restype = ctypes.c_int
        L.oracle_qr_dd.argtypes = [_i64, _i64, _dp, _dp]
        L.oracle_qr_dd.restype = ctypes.c_int
        L.oracle_qr_dd_check.argtypes = [_i64, _i64, _dp, _dp, _dp, _dp, _dp]
        L.oracle_taylor_dd.argtypes = [_i64, _i64, ctypes.c_int, _dp, _dp, _dp]
        L.oracle_taylor_dd.restype = ctypes.c_int
        L.oracle_qr_dd_check.restype = ctypes.c_int
        _lib = L
    return _lib


def _d(a):
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(_dp)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def two_sum(a, b):
    a, b = _f64(a).ravel(), _f64(b).ravel()
    s, e = np.empty_like(a), np.empty_like(a)
    lib().oracle_two_sum(a.size, _d(a), _d(b), _d(s), _d(e))
    return s, e


def fast_two_sum(a, b):
    a, b = _f64(a).ravel(), _f64(b).ravel()
    s, e = np.empty_like(a), np.empty_like(a)
    lib().oracle_fast_two_sum(a.size, _d(a), _d(b), _d(s), _d(e))
    return s, e


def two_prod(a, b):
    a, b = _f64(a).ravel(), _f64(b).ravel()
    p, e = np.empty_like(a), np.empty_like(a)
    lib().oracle_two_prod(a.size, _d(a), _d(b), _d(p), _d(e))
    return p, e


def md_fma(acc, a, b):
    """acc + a*b rounded to L limbs; arrays [L][n]."""
    acc, a, b = _f64(acc), _f64(a), _f64(b)
    L, n = a.shape
    out = np.empty_like(a)
    lib().oracle_md_fma(L, n, _d(acc), _d(a), _d(b), _d(out))
    return out


def dd_add(a, b):
    a, b = _f64(a), _f64(b)
    out = np.empty_like(a)
    lib().oracle_dd_add(a.shape[1], _d(a), _d(b), _d(out))
    return out


def dd_mul(a, b):
    a, b = _f64(a), _f64(b)
    out = np.empty_like(a)
    lib().oracle_dd_mul(a.shape[1], _d(a), _d(b), _d(out))
    return out


def classic_gemm(A, B, rows=None, variant=None, nthreads=0):
    """Classic multiple-double GEMM (one sequential inner product per element).

    Returns (C, threads_used); with ``rows=(r0, r1)`` only those rows of C are
    computed (the others are zero)."""
    A, B = _f64(A), _f64(B)
    L, m, k = A.shape
    n = B.shape[2]
    if variant is None:
        variant = 0 if L == 2 else 1
    r0, r1 = (0, m) if rows is None else rows
    C = np.zeros((L, m, n), dtype=np.float64)
    used = lib().oracle_classic_gemm(m, n, k, L, _d(A), _d(B), _d(C), r0, r1, variant, nthreads)
    if used < 0:
        raise ValueError(f"oracle_classic_gemm failed: {used}")
    return C, used


def exponents(X0, axis):
    X0 = _f64(X0)
    rows, cols = X0.shape
    E = np.empty(rows if axis == 0 else cols, dtype=np.int32)
    st = lib().oracle_exponents(rows, cols, axis, _d(X0), E.ctypes.data_as(_ip))
    if st:
        raise ValueError(st)
    return E


def split(X, E, S, axis, bits=13):
    """Digits [S][rows][cols] (float64, integer valued) of `bits` bits each."""
    X = _f64(X)
    L, rows, cols = X.shape
    E = np.ascontiguousarray(E, dtype=np.int32)
    D = np.empty((S, rows, cols), dtype=np.float64)
    if bits == 13:
        st = lib().oracle_split(rows, cols, L, S, axis, _d(X), E.ctypes.data_as(_ip), _d(D))
    else:
        st = lib().oracle_split_bits(rows, cols, L, S, bits, axis, _d(X), E.ctypes.data_as(_ip), _d(D))
    if st:
        raise ValueError(f"oracle_split failed: {st}")
    return D


def levels(DA, DB, T, per_pair=False):
    """Level products [T+1][m][n] (or pair products [S][S][m][n]) in int64."""
    DA, DB = _f64(DA), _f64(DB)
    S, m, k = DA.shape
    n = DB.shape[2]
    shape = (S, S, m, n) if per_pair else (T + 1, m, n)
    G = np.zeros(shape, dtype=np.int64)
    st = lib().oracle_levels(m, n, k, S, T, int(per_pair), _d(DA), _d(DB), G.ctypes.data_as(_lp))
    if st:
        raise ValueError(st)
    return G


def num_threads() -> int:
    return lib().oracle_num_threads()


def qr_dd(A):
    """Householder QR of a double-double matrix A [2][m][n] (m >= n) in classic
    double-double arithmetic: (QR [2][m][n] with R on and above the diagonal and
    the vectors below, tau [2][n])."""
    QR = np.array(A, dtype=np.float64, order="C", copy=True)
    _, m, n = QR.shape
    tau = np.zeros((2, n), dtype=np.float64)
    st = lib().oracle_qr_dd(m, n, _d(QR), _d(tau))
    if st:
        raise ValueError(f"oracle_qr_dd failed: {st}")
    return QR, tau


def qr_dd_check(A0, QR, tau):
    """(max |A0 - Q R| / max |A0|, max |Q^T Q - I|, Q [2][m][n]) of a factorization
    stored as qr_dd leaves it, every entry formed in double-double."""
    A0, QR, tau = _f64(A0), _f64(QR), _f64(tau)
    _, m, n = A0.shape
    out = np.zeros(2, dtype=np.float64)
    Q = np.zeros((2, m, n), dtype=np.float64)
    st = lib().oracle_qr_dd_check(m, n, _d(A0), _d(QR), _d(tau), _d(out), _d(Q))
    if st:
        raise ValueError(f"oracle_qr_dd_check failed: {st}")
    return float(out[0]), float(out[1]), Q


def taylor_dd(A, B):
    """X [d+1][2][n][r]: the Taylor coefficients of the solution of A(t) X(t) = B(t)
    modulo t^(d+1) (A [d+1][2][n][n], B [d+1][2][n][r]), each X_k from
    A_0 X_k = B_k - sum_{i=1..k} A_i X_{k-i} by the QR of A_0, in double-double."""
    A, B = _f64(A), _f64(B)
    nd, _, n, _ = A.shape
    r = B.shape[3]
    X = np.zeros((nd, 2, n, r), dtype=np.float64)
    st = lib().oracle_taylor_dd(n, r, nd - 1, _d(A), _d(B), _d(X))
    if st:
        raise ValueError(f"oracle_taylor_dd failed: {st}")
    return X
