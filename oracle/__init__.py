"""ctypes wrapper over the fp64 CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: the product path never imports this package.
Inputs are converted to float64 C-contiguous numpy arrays; outputs are numpy
float64 arrays.  See oracle.c for what is computed and which passages of the
paper each step follows.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None
_D = ctypes.POINTER(ctypes.c_double)
_U8 = ctypes.POINTER(ctypes.c_uint8)
_I64 = ctypes.POINTER(ctypes.c_int64)

STARTING, ENDING = 0, 1


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _LIB = load(_build.LIB)
    return _LIB


def load(path):
    """Load an oracle shared library from path and declare its signatures."""
    lib = ctypes.CDLL(path)
    i64, dbl, ci = ctypes.c_int64, ctypes.c_double, ctypes.c_int
    lib.oracle_fwd.argtypes = [ci, i64, i64, i64, dbl, _D, _D, _D, _D, _D, _U8, _D, _D,
                               _I64, i64]
    lib.oracle_fwd.restype = None
    lib.oracle_bwd.argtypes = [ci, i64, i64, i64, dbl, _D, _D, _D, _D, _D, _U8, _D,
                               _D, _D, _D, _D, _D, _I64, i64, _I64, i64]
    lib.oracle_bwd.restype = None
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = ctypes.c_int
    return lib


def max_threads() -> int:
    """OpenMP threads the oracle runs on."""
    return int(_lib().oracle_max_threads())


def use_library(lib):
    """Swap the loaded library (returns the previous one).  The mutation
    tests use this to run the pins against deliberately broken builds."""
    global _LIB
    prev, _LIB = _LIB, lib
    return prev


def _f64(x):
    if hasattr(x, "detach"):  # torch tensor -> exact float64 copy
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a, t=_D):
    return a.ctypes.data_as(t) if a is not None else None


def _mask(mask, n):
    if mask is None:
        return None
    if hasattr(mask, "detach"):
        mask = mask.detach().to("cpu").numpy()
    m = np.ascontiguousarray(np.asarray(mask) != 0, dtype=np.uint8)
    assert m.shape == (n, n)
    return m


def _list(lst):
    if lst is None:
        return None, 0
    a = np.ascontiguousarray(np.asarray(lst, dtype=np.int64))
    return a, int(a.size)


def fwd(node, q, k, v, g, bias, mask=None, scale=None, rows=None, out=None, lse=None):
    """Forward: returns (out [n,n,h,d], lse [n,n,h]) in float64.

    rows restricts the work to those rows (entries of other rows are NaN
    unless out/lse arrays are passed in)."""
    q, k, v, g, bias = (_f64(t) for t in (q, k, v, g, bias))
    n, _, h, d = q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    m = _mask(mask, n)
    if out is None:
        out = np.full((n, n, h, d), np.nan)
    if lse is None:
        lse = np.full((n, n, h), np.nan)
    rl, nr = _list(rows)
    _lib().oracle_fwd(int(node), n, h, d, float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                      _ptr(bias), _ptr(m, _U8), _ptr(out), _ptr(lse), _ptr(rl, _I64), nr)
    return out, lse


def bwd(node, q, k, v, g, bias, dout, mask=None, scale=None, rows=None, db_queries=None):
    """Backward of sum(dout * out): returns dq, dk, dv, dg [n,n,h,d] and
    db [n,n,h] in float64.  rows restricts dq/dk/dv/dg to those rows;
    db_queries restricts db to those query indices (other entries NaN)."""
    q, k, v, g, bias, dout = (_f64(t) for t in (q, k, v, g, bias, dout))
    n, _, h, d = q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    m = _mask(mask, n)
    dq, dk, dv, dg = (np.full((n, n, h, d), np.nan) for _ in range(4))
    db = np.full((n, n, h), np.nan)
    rl, nr = _list(rows)
    ql, nq = _list(db_queries)
    _lib().oracle_bwd(int(node), n, h, d, float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                      _ptr(bias), _ptr(m, _U8), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv),
                      _ptr(dg), _ptr(db), _ptr(rl, _I64), nr, _ptr(ql, _I64), nq)
    return dq, dk, dv, dg, db


# ---- fused layer-norm + linear projection (ln_linear.c) ----------------------------

def _lnl_decl(lib):
    i64, dbl = ctypes.c_int64, ctypes.c_double
    lib.oracle_lnl_fwd.argtypes = [i64, i64, i64, dbl, _D, _D, _D, _D, _D, _D, _D, _I64, i64]
    lib.oracle_lnl_fwd.restype = None
    lib.oracle_lnl_bwd.argtypes = [i64, i64, i64, dbl, _D, _D, _D, _D, _D, _D, _D, _D, _D,
                                   _I64, i64]
    lib.oracle_lnl_bwd.restype = None
    return lib


def lnl_fwd(x, gamma, beta, w, eps=1e-5, rows=None):
    """Layer-norm over the last axis of x [M, K], then o2 = o1 W (W [K, N]).
    Returns (o2 [M, N], mean [M], rstd [M]) in float64; rows restricts the
    work to those rows (other entries NaN)."""
    x, gamma, beta, w = (_f64(t) for t in (x, gamma, beta, w))
    M, K = x.shape
    N = w.shape[1]
    o2 = np.full((M, N), np.nan)
    mean = np.full(M, np.nan)
    rstd = np.full(M, np.nan)
    rl, nr = _list(rows)
    _lnl_decl(_lib()).oracle_lnl_fwd(M, K, N, float(eps), _ptr(x), _ptr(gamma), _ptr(beta),
                                     _ptr(w), _ptr(o2), _ptr(mean), _ptr(rstd), _ptr(rl, _I64), nr)
    return o2, mean, rstd


def lnl_bwd(x, gamma, beta, w, do2, eps=1e-5, rows=None, sums=True):
    """Backward of sum(do2 * o2): returns (dx [M, K], dw [K, N], dgamma [K],
    dbeta [K]) in float64.  rows restricts dx to those rows; sums=False skips
    the sums over rows (dw, dgamma, dbeta are then None)."""
    x, gamma, beta, w, do2 = (_f64(t) for t in (x, gamma, beta, w, do2))
    M, K = x.shape
    N = w.shape[1]
    dx = np.full((M, K), np.nan)
    dw = np.full((K, N), np.nan) if sums else None
    dgamma = np.full(K, np.nan) if sums else None
    dbeta = np.full(K, np.nan) if sums else None
    rl, nr = _list(rows)
    _lnl_decl(_lib()).oracle_lnl_bwd(M, K, N, float(eps), _ptr(x), _ptr(gamma), _ptr(beta),
                                     _ptr(w), _ptr(do2), _ptr(dx), _ptr(dw), _ptr(dgamma),
                                     _ptr(dbeta), _ptr(rl, _I64), nr)
    return dx, dw, dgamma, dbeta
