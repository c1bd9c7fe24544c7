"""fp64 dictionary-of-keys oracle for the sparse-gradient path (ctypes wrapper).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg.  The library itself never imports it.

Every arithmetic step lives in nsd_oracle.c; this module only marshals numpy
arrays.  fp32 inputs are promoted to fp64 exactly before they reach C.
Outputs come in (value, mag) pairs: mag is the expression evaluated on the
absolute values of its terms and bounds the rounding error of any fp
evaluation order (|got - ref| <= c * u * mag).
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_i64, _f64 = C.c_int64, C.c_double
_p = C.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = C.CDLL(_LIB_PATH)
    sig = {
        "orc_dok_build2": (_p, [_i64, _i64, _i64, _p, _p, _p]),
        "orc_dok_build3": (_p, [_i64, _i64, _i64, _i64, _p, _p, _p, _p]),
        "orc_dok_free": (None, [_p]),
        "orc_dok_nkeys": (_i64, [_p]),
        "orc_dok_lookup2": (None, [_p, _i64, _p, _p, _p, _p]),
        "orc_coo_to_csr": (_i64, [_p, _p, _p, _p, _p]),
        "orc_stable_sort_by_key": (None, [_i64, _p, _i64, _p, _p, _p]),
        "orc_spmm": (None, [_p, _p, _p, _i64, _i64, _p, _p, _p]),
        "orc_spmm_t": (None, [_p, _p, _p, _i64, _f64, _i64, _p, _p, _p]),
        "orc_sddmm": (None, [_p, _p, _p, _p, _p, _i64, _f64, _i64, _p, _p, _p, _p]),
        "orc_loss_sum_spmv": (None, [_p, _p, _p, _p]),
        "orc_loss_half_sq": (None, [_i64, _p, _p, _p, _p]),
        "orc_loss_bilinear": (None, [_p, _p, _p, _i64, _p, _p]),
        "orc_mf_loss": (None, [_p, _p, _p, _i64, _p, _p]),
        "orc_mf_resid": (None, [_p, _p, _p, _i64, _i64, _p, _p, _p, _p]),
        "orc_mf_grad": (None, [_p, _p, _p, _i64, C.c_int, _i64, _p, _p, _p]),
        "orc_cp_loss": (None, [_p, _p, _p, _p, _i64, _p, _p]),
        "orc_cp_resid": (None, [_p, _p, _p, _p, _i64, _i64, _p, _p, _p, _p, _p]),
        "orc_cp_grad": (None, [_p, _p, _p, _p, _i64, C.c_int, _i64, _p, _p, _p]),
        "orc_ttv": (_i64, [_p, _p, _p, _p, _p, _p]),
        "orc_ttv_vjp": (None, [_p, _p, _p, _i64, _p, _p, _p, _p, _p, _p, _p]),
        "orc_ttm": (_i64, [_p, _p, C.c_int32, _p, _p, _p, _p]),
        "orc_ttm_vjp": (None, [_p, _p, C.c_int32, _p, _i64, _p, _p, _p, _p, _p, _p, _p]),
        "orc_ttmn": (_i64, [_p, C.c_int32, _p, C.c_int32, _p, _p, _p]),
        "orc_ttmn_vjp": (None, [_p, C.c_int32, _p, C.c_int32, _p, _i64, _p, _p, _p, _p, _p]),
        "orc_batax_jacobian": (_i64, [_p, _f64, _i64, _p, _p, _p, _p]),
        "orc_spmm_jvp": (None, [_p, _p, _p, _p, _i64, _p, _p, _p, _p]),
        "orc_dok_buildn": (_p, [C.c_int32, _p, _i64, _p, _p]),
        "orc_cpn_loss": (None, [_p, _p, _i64, _p, _p]),
        "orc_cpn_resid": (None, [_p, _p, _i64, _i64, _p, _p, _p]),
        "orc_cpn_grad": (None, [_p, _p, _i64, C.c_int, _i64, _p, _p, _p]),
        "orc_set_threads": (None, [C.c_int]),
        "orc_max_threads": (C.c_int, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def set_threads(n: int):
    """OpenMP threads of the oracle's loss scans and gradient loops, for
    calls made from the calling thread.  The gradient loops split their
    outputs by owner, so every thread count gives bitwise the same result."""
    _load().orc_set_threads(n)


def max_threads() -> int:
    return _load().orc_max_threads()


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f64a(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _sel(sel):
    return (0, None) if sel is None else (len(sel), _i32(sel))


class Dok:
    """A sparse matrix (order 2) or tensor (order 3 to 6) held as a DOK.

    Duplicate coordinates are summed on insert (semi-ring insert)."""

    def __init__(self, dims, coords, val=None):
        lib = _load()
        self.dims = tuple(int(d) for d in dims)
        self._keep = [_i32(c) for c in coords]
        v = None if val is None else np.ascontiguousarray(val, dtype=np.float32)
        n = len(self._keep[0])
        if len(self.dims) == 2:
            self.h = lib.orc_dok_build2(self.dims[0], self.dims[1], n,
                                        _ptr(self._keep[0]), _ptr(self._keep[1]), _ptr(v))
        elif len(self.dims) == 3:
            self.h = lib.orc_dok_build3(self.dims[0], self.dims[1], self.dims[2], n,
                                        *[_ptr(c) for c in self._keep], _ptr(v))
        else:
            dims = np.asarray(self.dims, dtype=np.int64)
            ptrs = (C.c_void_p * len(self.dims))(*[_ptr(c) for c in self._keep])
            self.h = lib.orc_dok_buildn(len(self.dims), _ptr(dims), n, ptrs, _ptr(v))
        self._keep = None

    @classmethod
    def from_csr(cls, nrows, ncols, rowptr, colind, val=None):
        rowptr = np.asarray(rowptr, dtype=np.int64)
        row = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
        return cls((nrows, ncols), (row, colind), val)

    @property
    def nkeys(self):
        return _load().orc_dok_nkeys(self.h)

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.orc_dok_free(self.h)
            self.h = None

    def lookup(self, qi, qj):
        qi, qj = _i32(qi), _i32(qj)
        out = np.empty(len(qi))
        pres = np.empty(len(qi), dtype=np.int8)
        _load().orc_dok_lookup2(self.h, len(qi), _ptr(qi), _ptr(qj), _ptr(out), _ptr(pres))
        return out, pres.astype(bool)


# -------------------------------------------------------------- formats

def coo_to_csr(A: Dok):
    """(rowptr, colind, val fp64, first-occurrence index) of the stored keys."""
    n = A.nkeys
    rowptr = np.empty(A.dims[0] + 1, dtype=np.int32)
    colind = np.empty(n, dtype=np.int32)
    val = np.empty(n)
    first = np.empty(n, dtype=np.int64)
    _load().orc_coo_to_csr(A.h, _ptr(rowptr), _ptr(colind), _ptr(val), _ptr(first))
    return rowptr, colind, val, first


def stable_sort_by_key(key, nkeys):
    """(segptr, sorted_key, perm): positions stably sorted by key."""
    key = _i32(key)
    n = len(key)
    segptr = np.empty(nkeys + 1, dtype=np.int32)
    skey = np.empty(n, dtype=np.int32)
    perm = np.empty(n, dtype=np.int32)
    _load().orc_stable_sort_by_key(n, _ptr(key), nkeys, _ptr(segptr), _ptr(skey), _ptr(perm))
    return segptr, skey, perm


# ------------------------------------------------------------- products

def spmm(A: Dok, B, k, rows=None, Bmag=None):
    """C = A B (B None: ones), for the selected rows; returns (C, Cmag)."""
    B, Bmag = _f64a(B), _f64a(Bmag)
    nsel, sel = _sel(rows)
    m = nsel if rows is not None else A.dims[0]
    out, mag = np.empty((m, k)), np.empty((m, k))
    _load().orc_spmm(A.h, _ptr(B), _ptr(Bmag), k, nsel, _ptr(sel), _ptr(out), _ptr(mag))
    return out, mag


def spmm_t(A: Dok, G, k, alpha=1.0, cols=None, Gmag=None):
    """alpha * A^T G (G None: ones), for the selected columns."""
    G, Gmag = _f64a(G), _f64a(Gmag)
    nsel, sel = _sel(cols)
    m = nsel if cols is not None else A.dims[1]
    out, mag = np.empty((m, k)), np.empty((m, k))
    _load().orc_spmm_t(A.h, _ptr(G), _ptr(Gmag), k, alpha, nsel, _ptr(sel), _ptr(out), _ptr(mag))
    return out, mag


def sddmm(A: Dok, X, Y, k, qi, qj, alpha=1.0, Xmag=None, Ymag=None):
    """alpha * <X_i, Y_j> at each queried stored key (0 elsewhere)."""
    X, Xmag, Y, Ymag = _f64a(X), _f64a(Xmag), _f64a(Y), _f64a(Ymag)
    qi, qj = _i32(qi), _i32(qj)
    out, mag = np.empty(len(qi)), np.empty(len(qi))
    _load().orc_sddmm(A.h, _ptr(X), _ptr(Xmag), _ptr(Y), _ptr(Ymag), k, alpha, len(qi),
                      _ptr(qi), _ptr(qj), _ptr(out), _ptr(mag))
    return out, mag


# ---------------------------------------------------------------- losses

def _two():
    return C.c_double(0.0), C.c_double(0.0)


def loss_sum_spmv(A: Dok, x):
    x = _f64a(x)
    L, M = _two()
    _load().orc_loss_sum_spmv(A.h, _ptr(x), C.byref(L), C.byref(M))
    return L.value, M.value


def loss_half_sq(Cd, Cmag):
    Cd, Cmag = _f64a(Cd), _f64a(Cmag)
    L, M = _two()
    _load().orc_loss_half_sq(Cd.size, _ptr(Cd), _ptr(Cmag), C.byref(L), C.byref(M))
    return L.value, M.value


def loss_bilinear(A: Dok, G, H, k):
    G, H = _f64a(G), _f64a(H)
    L, M = _two()
    _load().orc_loss_bilinear(A.h, _ptr(G), _ptr(H), k, C.byref(L), C.byref(M))
    return L.value, M.value


def mf_loss(A: Dok, U, V, k):
    U, V = _f64a(U), _f64a(V)
    L, M = _two()
    _load().orc_mf_loss(A.h, _ptr(U), _ptr(V), k, C.byref(L), C.byref(M))
    return L.value, M.value


def mf_resid(A: Dok, U, V, k, qi, qj):
    U, V, qi, qj = _f64a(U), _f64a(V), _i32(qi), _i32(qj)
    r, m = np.empty(len(qi)), np.empty(len(qi))
    _load().orc_mf_resid(A.h, _ptr(U), _ptr(V), k, len(qi), _ptr(qi), _ptr(qj), _ptr(r), _ptr(m))
    return r, m


def mf_grad(A: Dok, U, V, k, mode, sel=None):
    U, V = _f64a(U), _f64a(V)
    nsel, s = _sel(sel)
    m = nsel if sel is not None else A.dims[mode]
    out, mag = np.empty((m, k)), np.empty((m, k))
    _load().orc_mf_grad(A.h, _ptr(U), _ptr(V), k, mode, nsel, _ptr(s), _ptr(out), _ptr(mag))
    return out, mag


def cp_loss(X: Dok, F1, F2, F3, R):
    F1, F2, F3 = _f64a(F1), _f64a(F2), _f64a(F3)
    L, M = _two()
    _load().orc_cp_loss(X.h, _ptr(F1), _ptr(F2), _ptr(F3), R, C.byref(L), C.byref(M))
    return L.value, M.value


def cp_resid(X: Dok, F1, F2, F3, R, qi, qj, ql):
    F1, F2, F3 = _f64a(F1), _f64a(F2), _f64a(F3)
    qi, qj, ql = _i32(qi), _i32(qj), _i32(ql)
    r, m = np.empty(len(qi)), np.empty(len(qi))
    _load().orc_cp_resid(X.h, _ptr(F1), _ptr(F2), _ptr(F3), R, len(qi), _ptr(qi), _ptr(qj),
                         _ptr(ql), _ptr(r), _ptr(m))
    return r, m


def cp_grad(X: Dok, F1, F2, F3, R, mode, sel=None):
    F1, F2, F3 = _f64a(F1), _f64a(F2), _f64a(F3)
    nsel, s = _sel(sel)
    m = nsel if sel is not None else X.dims[mode]
    out, mag = np.empty((m, R)), np.empty((m, R))
    _load().orc_cp_grad(X.h, _ptr(F1), _ptr(F2), _ptr(F3), R, mode, nsel, _ptr(s), _ptr(out),
                        _ptr(mag))
    return out, mag


def ttv(X: Dok, v):
    """Y = X x_3 v on the projected (i, j) keys: (yi, yj, y, ymag) in (i, j) order."""
    v = _f64a(v)
    cap = X.nkeys
    yi, yj = np.empty(cap, dtype=np.int32), np.empty(cap, dtype=np.int32)
    y, ym = np.empty(cap), np.empty(cap)
    n = _load().orc_ttv(X.h, _ptr(v), _ptr(yi), _ptr(yj), _ptr(y), _ptr(ym))
    return yi[:n], yj[:n], y[:n], ym[:n]


def ttv_vjp(X: Dok, v, gY: Dok, qi, qj, ql):
    """(dX at queries, dXmag, dv, dvmag) for the upstream gY."""
    v = _f64a(v)
    qi, qj, ql = _i32(qi), _i32(qj), _i32(ql)
    dX, dXm = np.empty(len(qi)), np.empty(len(qi))
    dv, dvm = np.empty(X.dims[2]), np.empty(X.dims[2])
    _load().orc_ttv_vjp(X.h, _ptr(v), gY.h, len(qi), _ptr(qi), _ptr(qj), _ptr(ql), _ptr(dX),
                        _ptr(dXm), _ptr(dv), _ptr(dvm))
    return dX, dXm, dv, dvm


def ttm(X: Dok, U, R):
    """Y = X x_3 U (U [dims[2] x R]) on the projected (i, j) keys:
    (yi, yj, y [ny x R], ymag) in (i, j) order."""
    U = _f64a(U)
    cap = X.nkeys
    yi, yj = np.empty(cap, dtype=np.int32), np.empty(cap, dtype=np.int32)
    y, ym = np.empty(max(cap, 1) * R), np.empty(max(cap, 1) * R)
    n = _load().orc_ttm(X.h, _ptr(U), R, _ptr(yi), _ptr(yj), _ptr(y), _ptr(ym))
    return yi[:n], yj[:n], y[: n * R].reshape(n, R), ym[: n * R].reshape(n, R)


def ttm_vjp(X: Dok, U, R, gY, qi, qj, ql):
    """(dX at queries, dXmag, dU [dims[2] x R], dUmag) for the upstream gY
    [ny x R] on Y's keys in (i, j) order."""
    U, gY = _f64a(U), _f64a(gY)
    qi, qj, ql = _i32(qi), _i32(qj), _i32(ql)
    dX, dXm = np.empty(len(qi)), np.empty(len(qi))
    dU, dUm = np.empty(X.dims[2] * R), np.empty(X.dims[2] * R)
    _load().orc_ttm_vjp(X.h, _ptr(U), R, _ptr(gY), len(qi), _ptr(qi), _ptr(qj), _ptr(ql),
                        _ptr(dX), _ptr(dXm), _ptr(dU), _ptr(dUm))
    return dX, dXm, dU.reshape(X.dims[2], R), dUm.reshape(X.dims[2], R)


def ttmn(X: Dok, mode, U, R):
    """Mode-`mode` product Y = X x_mode U (U [dims[mode] x R]) of an order-N
    DOK on its projected keys: (keys, y [ny x R], ymag), keys a list of the
    N - 1 coordinate arrays of the other modes, in lexicographic order."""
    U = _f64a(U)
    cap = max(X.nkeys, 1)
    keys = [np.empty(cap, dtype=np.int32) for _ in range(len(X.dims) - 1)]
    kp = (C.c_void_p * len(keys))(*[_ptr(k) for k in keys])
    y, ym = np.empty(cap * R), np.empty(cap * R)
    n = _load().orc_ttmn(X.h, int(mode), _ptr(U), R, kp, _ptr(y), _ptr(ym))
    return [k[:n] for k in keys], y[: n * R].reshape(n, R), ym[: n * R].reshape(n, R)


def ttmn_vjp(X: Dok, mode, U, R, gY, coords):
    """(dX at the queried keys, dXmag, dU [dims[mode] x R], dUmag) of the
    mode product for the upstream gY [ny x R] on Y's keys in lexicographic
    order; coords: N arrays of query coordinates."""
    U, gY = _f64a(U), _f64a(gY)
    qs = [_i32(c) for c in coords]
    qp = (C.c_void_p * len(qs))(*[_ptr(c) for c in qs])
    n = len(qs[0])
    dX, dXm = np.empty(n), np.empty(n)
    nl = X.dims[mode]
    dU, dUm = np.empty(nl * R), np.empty(nl * R)
    _load().orc_ttmn_vjp(X.h, int(mode), _ptr(U), R, _ptr(gY), n, qp, _ptr(dX), _ptr(dXm),
                         _ptr(dU), _ptr(dUm))
    return dX, dXm, dU.reshape(nl, R), dUm.reshape(nl, R)


def batax_jacobian(A: Dok, beta):
    """J = beta A^T A of the BATAX kernel as an n x n CSR (rowptr, colind,
    val, mag), n = columns of A; keys are the pairs of stored keys sharing a
    row of A."""
    rowptr_a, _, _, _ = coo_to_csr(A)
    cap = int(np.sum(np.diff(rowptr_a).astype(np.int64) ** 2))
    n = A.dims[1]
    rowptr = np.empty(n + 1, dtype=np.int32)
    colind = np.empty(max(cap, 1), dtype=np.int32)
    val, mag = np.empty(max(cap, 1)), np.empty(max(cap, 1))
    nk = _load().orc_batax_jacobian(A.h, float(beta), cap, _ptr(rowptr), _ptr(colind), _ptr(val),
                                    _ptr(mag))
    assert nk <= cap
    return rowptr, colind[:nk], val[:nk], mag[:nk]


def spmm_jvp(A: Dok, dA: Dok, B, dB, k):
    """(C, Cmag, dC, dCmag) of C = A B with tangents dA (on A's keys) and dB."""
    B, dB = _f64a(B), _f64a(dB)
    m = A.dims[0]
    C, Cm, dC, dCm = (np.empty((m, k)) for _ in range(4))
    _load().orc_spmm_jvp(A.h, dA.h, _ptr(B), _ptr(dB), k, _ptr(C), _ptr(Cm), _ptr(dC), _ptr(dCm))
    return C, Cm, dC, dCm


def _fptrs(F):
    Fs = [_f64a(f) for f in F]
    return Fs, (C.c_void_p * len(Fs))(*[_ptr(f) for f in Fs])


def cpn_loss(X: Dok, F, R):
    """Order-N CP loss 1/2 sum (x - m)^2 (and its mag); F = [F_1 .. F_N]."""
    Fs, fp = _fptrs(F)
    L, M = _two()
    _load().orc_cpn_loss(X.h, fp, R, C.byref(L), C.byref(M))
    return L.value, M.value


def cpn_resid(X: Dok, F, R, coords):
    """Residual x - m at the queried keys (coords: N arrays)."""
    Fs, fp = _fptrs(F)
    qs = [_i32(c) for c in coords]
    qp = (C.c_void_p * len(qs))(*[_ptr(c) for c in qs])
    n = len(qs[0])
    r, m = np.empty(n), np.empty(n)
    _load().orc_cpn_resid(X.h, fp, R, n, qp, _ptr(r), _ptr(m))
    return r, m


def cpn_grad(X: Dok, F, R, mode, sel=None):
    """dF_mode, the negated mode MTTKRP of the residual (selected rows)."""
    Fs, fp = _fptrs(F)
    nsel, s = _sel(sel)
    m = nsel if sel is not None else X.dims[mode]
    out, mag = np.empty((m, R)), np.empty((m, R))
    _load().orc_cpn_grad(X.h, fp, R, mode, nsel, _ptr(s), _ptr(out), _ptr(mag))
    return out, mag
