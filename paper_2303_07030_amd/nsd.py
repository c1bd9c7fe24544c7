"""ctypes binding of libnsd (include/nsd.h), argument marshalling only.

Every function has the name of the C entry point it calls and takes torch
tensors (device memory owned by the caller), which are passed as raw
pointers; `None` passes NULL.  A status other than NSD_OK raises NsdError.
No arithmetic of the method happens here: every step runs in the HIP
library, and importing this module fails loudly when the library is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import torch  # noqa: F401  (loads the HIP runtime libnsd links against)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libnsd.so")

NSD_OK = 0
NSD_ERR_INVALID_ARG = 1
NSD_ERR_BAD_FORMAT = 2
NSD_ERR_DUPLICATE = 3
NSD_ERR_TOO_LARGE = 4
NSD_ERR_WORKSPACE = 5
NSD_ERR_UNSUPPORTED = 6
NSD_ERR_HIP = 7
NSD_DUP_SUM = 0
NSD_DUP_ERROR = 1
KERNEL_IDS = {"sgr_main": 1, "sgr_fix": 2, "sddmm": 3, "frob_row": 4, "frob_col": 5, "mf": 6,
              "cp": 7, "loss": 8, "ttv": 9, "dual": 10, "sort": 11, "jvp": 12, "cpn": 13,
              "perm": 14, "batax_rows": 15}


class NsdError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        super().__init__(f"{func}: {status_name(status)}: {msg}")
        self.status = status


class nsd_perm_plan(C.Structure):
    _fields_ = [("n", C.c_int32), ("tile", C.c_int32), ("stage", C.c_void_p),
                ("src_local", C.c_void_p), ("dst_local", C.c_void_p)]


class nsd_plan(C.Structure):
    _fields_ = [("item_len", C.c_int32), ("nitems", C.c_int32), ("nlong", C.c_int32),
                ("nhuge", C.c_int32), ("nchunks", C.c_int32), ("nempty", C.c_int32),
                ("item_ptr", C.c_void_p), ("long_seg", C.c_void_p), ("long_first", C.c_void_p),
                ("huge_idx", C.c_void_p), ("chunk_item", C.c_void_p), ("chunk_ord", C.c_void_p),
                ("empty_seg", C.c_void_p),
                ("longest_chunks", C.c_int32)]


class nsd_csr(C.Structure):
    _fields_ = [("nrows", C.c_int32), ("ncols", C.c_int32), ("nnz", C.c_int32),
                ("rowptr", C.c_void_p), ("rowidx", C.c_void_p), ("colind", C.c_void_p),
                ("val", C.c_void_p), ("plan", nsd_plan)]


class nsd_csc(C.Structure):
    _fields_ = [("nrows", C.c_int32), ("ncols", C.c_int32), ("nnz", C.c_int32),
                ("colptr", C.c_void_p), ("colidx", C.c_void_p), ("rowind", C.c_void_p),
                ("perm", C.c_void_p), ("plan", nsd_plan), ("to_csc", nsd_perm_plan),
                ("to_csr", nsd_perm_plan)]


class nsd_coo3_mode(C.Structure):
    _fields_ = [("mode", C.c_int32), ("segptr", C.c_void_p), ("segidx", C.c_void_p),
                ("idx_a", C.c_void_p), ("idx_b", C.c_void_p), ("val", C.c_void_p),
                ("perm", C.c_void_p), ("plan", nsd_plan)]


class nsd_coo3(C.Structure):
    _fields_ = [("dims", C.c_int32 * 3), ("nnz", C.c_int32), ("mode", nsd_coo3_mode * 3)]


MAX_ORDER = 6


class nsd_coon_mode(C.Structure):
    _fields_ = [("mode", C.c_int32), ("segptr", C.c_void_p), ("segidx", C.c_void_p),
                ("idx", C.c_void_p * (MAX_ORDER - 1)), ("val", C.c_void_p),
                ("perm", C.c_void_p), ("plan", nsd_plan), ("fiber", C.c_int32)]


class nsd_coon(C.Structure):
    _fields_ = [("order", C.c_int32), ("dims", C.c_int32 * MAX_ORDER), ("nnz", C.c_int32),
                ("mode", nsd_coon_mode * MAX_ORDER)]


class nsd_ttv_plan(C.Structure):
    _fields_ = [("order", C.c_int32), ("mode", C.c_int32), ("dims", C.c_int32 * MAX_ORDER),
                ("nnz", C.c_int32), ("ny", C.c_int32),
                ("ykey", C.c_void_p * (MAX_ORDER - 1)), ("yptr", C.c_void_p),
                ("yseg", C.c_void_p), ("yperm", C.c_void_p), ("ykidx", C.c_void_p),
                ("yplan", nsd_plan), ("lptr", C.c_void_p), ("lseg", C.c_void_p),
                ("lperm", C.c_void_p), ("lpair", C.c_void_p), ("lplan", nsd_plan)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"libnsd.so is not built ({LIB_PATH}); run "
                      "`python -m paper_2303_07030_amd.build` first")
_lib = C.CDLL(LIB_PATH)

_P = C.c_void_p
_I = C.c_int32
_SZ = C.c_size_t
_CSR = C.POINTER(nsd_csr)
_CSC = C.POINTER(nsd_csc)
_COO3 = C.POINTER(nsd_coo3)
_TTV = C.POINTER(nsd_ttv_plan)

_SIGS = {
    "nsd_status_string": (C.c_char_p, [C.c_int]),
    "nsd_last_error": (C.c_char_p, []),
    "nsd_version": (C.c_int, []),
    "nsd_probe_set": (C.c_int, [C.c_int, C.POINTER(_P), C.POINTER(_P), _I]),
    "nsd_probe_count": (C.c_int, [C.POINTER(_I)]),
    "nsd_probe_clear": (C.c_int, []),
    "nsd_workspace_size": (C.c_int, [_CSR, _CSC, _I, C.POINTER(_SZ)]),
    "nsd_plan_item_len": (C.c_int, [_I, _I, C.POINTER(_I)]),
    "nsd_plan_bounds": (C.c_int, [_I, _I, _I, C.POINTER(_I), C.POINTER(_I), C.POINTER(_I),
                                  C.POINTER(_SZ)]),
    "nsd_plan_build": (C.c_int, [_I, _I, _P, _I, _P, _P, _P, _P, _P, _P, _P,
                                 C.POINTER(nsd_plan), _P, _SZ, _P]),
    "nsd_build_workspace_size": (C.c_int, [_I, _I, C.POINTER(_SZ)]),
    "nsd_perm_plan_workspace_size": (C.c_int, [_I, C.POINTER(_SZ)]),
    "nsd_perm_plan_build": (C.c_int, [_I, _P, C.c_int, _P, _P, _P, C.POINTER(nsd_perm_plan),
                                      _P, _SZ, _P]),
    "nsd_permute_f32": (C.c_int, [C.POINTER(nsd_perm_plan), _P, _P, _P, _P]),
    "nsd_csr_expand_rows": (C.c_int, [_I, _I, _P, _P, _P]),
    "nsd_coo_to_csr": (C.c_int, [_I, _I, _I, _P, _P, _P, C.c_int, _P, _P, _P, _P, _P,
                                 C.POINTER(_I), _P, _SZ, _P]),
    "nsd_csr_to_csc": (C.c_int, [_CSR, _P, _P, _P, _P, _P, _SZ, _P]),
    "nsd_coo_mode_index": (C.c_int, [_I, _I, _P, _P, _P, _P, _P, _SZ, _P]),
    "nsd_gather_f32": (C.c_int, [_I, _P, _P, _P, _P]),
    "nsd_gather_i32": (C.c_int, [_I, _P, _P, _P, _P]),
    "nsd_validate_csr": (C.c_int, [_CSR, C.c_int, _P, _SZ, _P]),
    "nsd_spmv": (C.c_int, [_CSR, _P, _P, _P, _SZ, _P]),
    "nsd_spmm": (C.c_int, [_CSR, _P, _I, _P, _P, _SZ, _P]),
    "nsd_sddmm": (C.c_int, [_CSR, _P, _P, _I, C.c_float, _P, _P]),
    "nsd_spmm_t": (C.c_int, [_CSR, _CSC, _P, _I, C.c_float, _P, _P, _SZ, _P]),
    "nsd_loss_sum_spmv": (C.c_int, [_CSR, _CSC, _P, C.c_float, _P, _P, _P, _P, _SZ, _P]),
    "nsd_loss_frob_spmm": (C.c_int, [_CSR, _CSC, _P, _I, C.c_float, _P, _P, _P, _P, _P, _SZ,
                                     _P]),
    "nsd_loss_bilinear": (C.c_int, [_CSR, _CSC, _P, _P, _I, C.c_float, _P, _P, _P, _P, _SZ,
                                    _P]),
    "nsd_loss_bilinear_noalloc": (C.c_int, [_CSR, _CSC, _P, _P, _I, C.c_float, _P, _P, _P,
                                            _P]),
    "nsd_loss_mf": (C.c_int, [_CSR, _CSC, _P, _P, _P, _I, C.c_float, _P, _P, _P, _P, _SZ, _P]),
    "nsd_cp_workspace_size": (C.c_int, [_COO3, _I, C.POINTER(_SZ)]),
    "nsd_ttv_build_workspace_size": (C.c_int, [_I, C.POINTER(_I), _I, C.POINTER(_SZ)]),
    "nsd_ttv_build": (C.c_int, [_I, C.POINTER(_I), _I, C.POINTER(_P), _I, C.POINTER(_P),
                                _P, _P, _P, _P, _P, _P, _P, _P,
                                C.POINTER(_I), _P, _SZ, _P]),
    "nsd_ttv_workspace_size": (C.c_int, [_TTV, C.POINTER(_SZ)]),
    "nsd_ttv": (C.c_int, [_TTV, _P, _P, _P, _P, _SZ, _P]),
    "nsd_ttv_vjp": (C.c_int, [_TTV, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "nsd_ttm_workspace_size": (C.c_int, [_TTV, _I, C.POINTER(_SZ)]),
    "nsd_ttm": (C.c_int, [_TTV, _P, _P, _I, _P, _P, _SZ, _P]),
    "nsd_ttm_vjp": (C.c_int, [_TTV, _P, _P, _I, _P, _P, _P, _P, _SZ, _P]),
    "nsd_dot": (C.c_int, [C.c_int64, _P, _P, C.c_double, C.c_int, _P, _P, _SZ, _P]),
    "nsd_spmm_vjp": (C.c_int, [C.POINTER(nsd_csr), C.POINTER(nsd_csc), _P, _P, _I, _P, _P, _P,
                               _SZ, _P]),
    "nsd_spmv_vjp": (C.c_int, [C.POINTER(nsd_csr), C.POINTER(nsd_csc), _P, _P, _P, _P, _P, _SZ,
                               _P]),
    "nsd_validate_coo_workspace_size": (C.c_int, [_I, _P, _I, C.POINTER(_SZ)]),
    "nsd_validate_coo": (C.c_int, [_I, _P, _I, _P, C.c_int, _P, _SZ, _P]),
    "nsd_axpby": (C.c_int, [C.c_int64, C.c_float, _P, C.c_float, _P, _P]),
    "nsd_diag_keys": (C.c_int, [_CSR, C.c_float, _P, _P]),
    "nsd_cpn_workspace_size": (C.c_int, [C.POINTER(nsd_coon), _I, C.POINTER(_SZ)]),
    "nsd_loss_cpn": (C.c_int, [C.POINTER(nsd_coon), C.POINTER(_P), _I, C.c_float, _P, _P,
                               C.POINTER(_P), _P, _SZ, _P]),
    "nsd_spmm_jvp": (C.c_int, [_CSR, _P, _P, _P, _I, _P, _P, _P, _SZ, _P]),
    "nsd_spmm_jvp_batch_workspace_size": (C.c_int, [_CSR, _I, C.POINTER(_SZ)]),
    "nsd_spmm_jvp_batch": (C.c_int, [_CSR, _I, _P, _P, _P, _I, _P, _P, _P, _SZ, _P]),
    "nsd_scale": (C.c_int, [C.c_int64, C.c_double, _P, _P, _P, _P, _P, C.c_float, _P, _P, _P]),
    "nsd_scale_real": (C.c_int, [C.c_double, _P, _P, _P, C.c_double, _P, _P]),
    "nsd_batax_pairs": (C.c_int, [_CSR, C.POINTER(C.c_int64), _P, _SZ, _P]),
    "nsd_batax_workspace_size": (C.c_int, [_CSR, C.c_int64, C.POINTER(_SZ)]),
    "nsd_batax_jacobian": (C.c_int, [_CSR, C.c_float, C.c_int64, _P, _P, _P, C.POINTER(_I), _P,
                                     _SZ, _P]),
    "nsd_loss_cp": (C.c_int, [_COO3, _P, _P, _P, _I, C.c_float, _P, _P, _P, _P, _P, _P, _SZ,
                              _P]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_SIGS)


def status_name(status: int) -> str:
    return _lib.nsd_status_string(status).decode()


def _p(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def _stream(s):
    if s is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    return s if isinstance(s, int) else s.cuda_stream


def _check(status: int, func: str):
    if status != NSD_OK:
        raise NsdError(status, func, _lib.nsd_last_error().decode())


# ------------------------------------------------------------------ info

def nsd_status_string(status: int) -> str:
    return status_name(status)


def nsd_last_error() -> str:
    return _lib.nsd_last_error().decode()


def nsd_version() -> int:
    return _lib.nsd_version()


def nsd_probe_set(kernel_id: int, start_events, stop_events):
    """start_events / stop_events: raw hipEvent_t handles (ints)."""
    n = len(start_events)
    sa = (_P * n)(*start_events)
    so = (_P * n)(*stop_events)
    _check(_lib.nsd_probe_set(kernel_id, sa, so, n), "nsd_probe_set")


def nsd_probe_count() -> int:
    c = _I(0)
    _check(_lib.nsd_probe_count(C.byref(c)), "nsd_probe_count")
    return c.value


def nsd_probe_clear():
    _check(_lib.nsd_probe_clear(), "nsd_probe_clear")


def nsd_workspace_size(A: nsd_csr, At, k: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_workspace_size(C.byref(A), None if At is None else C.byref(At), k,
                                   C.byref(b)), "nsd_workspace_size")
    return b.value


def nsd_plan_item_len(nnz: int, k: int) -> int:
    L = _I(0)
    _check(_lib.nsd_plan_item_len(nnz, k, C.byref(L)), "nsd_plan_item_len")
    return L.value


def nsd_plan_bounds(nseg: int, nnz: int, item_len: int):
    """(max_items, max_long, max_chunks, workspace bytes) for nsd_plan_build."""
    mi, ml, mc, wb = _I(0), _I(0), _I(0), _SZ(0)
    _check(_lib.nsd_plan_bounds(nseg, nnz, item_len, C.byref(mi), C.byref(ml), C.byref(mc),
                                C.byref(wb)), "nsd_plan_bounds")
    return mi.value, ml.value, mc.value, wb.value


def nsd_plan_build(nseg, nnz, segptr, item_len, item_ptr, long_seg, long_first, huge_idx,
                   chunk_item, chunk_ord, empty_seg, ws, stream=None) -> nsd_plan:
    plan = nsd_plan()
    _check(_lib.nsd_plan_build(nseg, nnz, _p(segptr), item_len, _p(item_ptr), _p(long_seg),
                               _p(long_first), _p(huge_idx), _p(chunk_item), _p(chunk_ord),
                               _p(empty_seg), C.byref(plan), _p(ws), _nbytes(ws),
                               _stream(stream)),
           "nsd_plan_build")
    plan._keep = dict(item_ptr=item_ptr, long_seg=long_seg, long_first=long_first,
                      huge_idx=huge_idx, chunk_item=chunk_item, chunk_ord=chunk_ord,
                      empty_seg=empty_seg)
    return plan


def nsd_perm_plan_workspace_size(n: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_perm_plan_workspace_size(n, C.byref(b)), "nsd_perm_plan_workspace_size")
    return b.value


def nsd_perm_plan_build(n, perm, inverse, stage, src_local, dst_local, ws,
                        stream=None) -> nsd_perm_plan:
    plan = nsd_perm_plan()
    _check(_lib.nsd_perm_plan_build(n, _p(perm), int(inverse), _p(stage), _p(src_local),
                                    _p(dst_local), C.byref(plan), _p(ws), _nbytes(ws),
                                    _stream(stream)),
           "nsd_perm_plan_build")
    plan._keep = dict(stage=stage, src_local=src_local, dst_local=dst_local)
    return plan


def nsd_permute_f32(plan: nsd_perm_plan, src, dst, staging, stream=None):
    _check(_lib.nsd_permute_f32(C.byref(plan), _p(src), _p(dst), _p(staging), _stream(stream)),
           "nsd_permute_f32")


def nsd_build_workspace_size(n: int, max_key: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_build_workspace_size(n, max_key, C.byref(b)), "nsd_build_workspace_size")
    return b.value


# ------------------------------------------------------------ descriptors

def csr_desc(nrows, ncols, rowptr, rowidx, colind, val) -> nsd_csr:
    nnz = 0 if colind is None else colind.numel()
    d = nsd_csr(nrows, ncols, nnz, _p(rowptr), _p(rowidx), _p(colind), _p(val))
    d._keep = (rowptr, rowidx, colind, val)
    return d


def csc_desc(nrows, ncols, colptr, colidx, rowind, perm) -> nsd_csc:
    nnz = 0 if rowind is None else rowind.numel()
    d = nsd_csc(nrows, ncols, nnz, _p(colptr), _p(colidx), _p(rowind), _p(perm))
    d._keep = (colptr, colidx, rowind, perm)
    return d


# -------------------------------------------------------------- builders

def nsd_csr_expand_rows(nrows, nnz, rowptr, rowidx, stream=None):
    _check(_lib.nsd_csr_expand_rows(nrows, nnz, _p(rowptr), _p(rowidx), _stream(stream)),
           "nsd_csr_expand_rows")


def nsd_coo_to_csr(nrows, ncols, nnz, row, col, val, policy, rowptr, rowidx, colind, val_out,
                   perm, ws, stream=None) -> int:
    out = _I(0)
    _check(_lib.nsd_coo_to_csr(nrows, ncols, nnz, _p(row), _p(col), _p(val), policy, _p(rowptr),
                               _p(rowidx), _p(colind), _p(val_out), _p(perm), C.byref(out),
                               _p(ws), _nbytes(ws), _stream(stream)), "nsd_coo_to_csr")
    return out.value


def nsd_csr_to_csc(A: nsd_csr, colptr, colidx, rowind, perm, ws, stream=None):
    _check(_lib.nsd_csr_to_csc(C.byref(A), _p(colptr), _p(colidx), _p(rowind), _p(perm), _p(ws),
                               _nbytes(ws), _stream(stream)), "nsd_csr_to_csc")


def nsd_coo_mode_index(nnz, dim, key, segptr, segidx, perm, ws, stream=None):
    _check(_lib.nsd_coo_mode_index(nnz, dim, _p(key), _p(segptr), _p(segidx), _p(perm), _p(ws),
                                   _nbytes(ws), _stream(stream)), "nsd_coo_mode_index")


def nsd_gather_f32(n, perm, src, dst, stream=None):
    _check(_lib.nsd_gather_f32(n, _p(perm), _p(src), _p(dst), _stream(stream)), "nsd_gather_f32")


def nsd_gather_i32(n, perm, src, dst, stream=None):
    _check(_lib.nsd_gather_i32(n, _p(perm), _p(src), _p(dst), _stream(stream)), "nsd_gather_i32")


def nsd_validate_csr(A: nsd_csr, check_sorted, ws, stream=None):
    _check(_lib.nsd_validate_csr(C.byref(A), int(check_sorted), _p(ws), _nbytes(ws),
                                 _stream(stream)), "nsd_validate_csr")


# --------------------------------------------------------------- compute

def nsd_spmv(A: nsd_csr, x, y, ws, stream=None):
    _check(_lib.nsd_spmv(C.byref(A), _p(x), _p(y), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_spmv")


def nsd_spmm(A: nsd_csr, B, k, Cout, ws, stream=None):
    _check(_lib.nsd_spmm(C.byref(A), _p(B), k, _p(Cout), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_spmm")


def nsd_sddmm(A: nsd_csr, X, Y, k, alpha, out, stream=None):
    _check(_lib.nsd_sddmm(C.byref(A), _p(X), _p(Y), k, alpha, _p(out), _stream(stream)),
           "nsd_sddmm")


def nsd_spmm_t(A: nsd_csr, At: nsd_csc, G, k, alpha, out, ws, stream=None):
    _check(_lib.nsd_spmm_t(C.byref(A), C.byref(At), _p(G), k, alpha, _p(out), _p(ws), _nbytes(ws),
                           _stream(stream)), "nsd_spmm_t")


def nsd_loss_sum_spmv(A: nsd_csr, At: nsd_csc, x, seed, loss, dA, dx, ws, stream=None):
    _check(_lib.nsd_loss_sum_spmv(C.byref(A), C.byref(At), _p(x), seed, _p(loss), _p(dA), _p(dx),
                                  _p(ws), _nbytes(ws), _stream(stream)), "nsd_loss_sum_spmv")


def nsd_loss_frob_spmm(A: nsd_csr, At: nsd_csc, B, k, seed, Cout, loss, dA, dB, ws, stream=None):
    _check(_lib.nsd_loss_frob_spmm(C.byref(A), C.byref(At), _p(B), k, seed, _p(Cout), _p(loss),
                                   _p(dA), _p(dB), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_loss_frob_spmm")


def nsd_loss_bilinear(A: nsd_csr, At: nsd_csc, H, G, k, seed, loss, dA, dH, ws, stream=None):
    _check(_lib.nsd_loss_bilinear(C.byref(A), C.byref(At), _p(H), _p(G), k, seed, _p(loss),
                                  _p(dA), _p(dH), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_loss_bilinear")


def nsd_loss_bilinear_noalloc(A: nsd_csr, At: nsd_csc, H, G, k, seed, loss, dA, dH,
                              stream=None):
    _check(_lib.nsd_loss_bilinear_noalloc(C.byref(A), C.byref(At), _p(H), _p(G), k, seed,
                                          _p(loss), _p(dA), _p(dH), _stream(stream)),
           "nsd_loss_bilinear_noalloc")


def nsd_loss_mf(A: nsd_csr, At: nsd_csc, valT, U, V, k, seed, loss, dU, dV, ws, stream=None):
    _check(_lib.nsd_loss_mf(C.byref(A), C.byref(At), _p(valT), _p(U), _p(V), k, seed, _p(loss),
                            _p(dU), _p(dV), _p(ws), _nbytes(ws), _stream(stream)), "nsd_loss_mf")


def nsd_cp_workspace_size(X: nsd_coo3, rank: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_cp_workspace_size(C.byref(X), rank, C.byref(b)), "nsd_cp_workspace_size")
    return b.value


def nsd_loss_cp(X: nsd_coo3, F1, F2, F3, rank, seed, loss, dX, dF1, dF2, dF3, ws, stream=None):
    _check(_lib.nsd_loss_cp(C.byref(X), _p(F1), _p(F2), _p(F3), rank, seed, _p(loss), _p(dX),
                            _p(dF1), _p(dF2), _p(dF3), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_loss_cp")


def _dims3(dims):
    return (_I * 3)(*[int(x) for x in dims])


def _dimsn(dims):
    return (_I * len(dims))(*[int(x) for x in dims])


def _ptr_array(ts):
    return (_P * len(ts))(*[_p(t) for t in ts])


def nsd_ttv_build_workspace_size(order, dims, nnz) -> int:
    b = _SZ(0)
    _check(_lib.nsd_ttv_build_workspace_size(order, _dimsn(dims), nnz, C.byref(b)),
           "nsd_ttv_build_workspace_size")
    return b.value


def nsd_ttv_build(order, dims, nnz, coords, mode, ykey, yptr, yseg, yperm, ykidx, lptr, lseg,
                  lperm, lpair, ws, stream=None) -> int:
    """coords: `order` device tensors; ykey: order - 1 device tensors."""
    ny = _I(0)
    _check(_lib.nsd_ttv_build(order, _dimsn(dims), nnz, _ptr_array(coords), mode,
                              _ptr_array(ykey), _p(yptr), _p(yseg), _p(yperm), _p(ykidx),
                              _p(lptr), _p(lseg), _p(lperm), _p(lpair), C.byref(ny), _p(ws),
                              _nbytes(ws), _stream(stream)),
           "nsd_ttv_build")
    return ny.value


def nsd_ttv_workspace_size(T: nsd_ttv_plan) -> int:
    b = _SZ(0)
    _check(_lib.nsd_ttv_workspace_size(C.byref(T), C.byref(b)), "nsd_ttv_workspace_size")
    return b.value


def nsd_ttv(T: nsd_ttv_plan, x, v, y, ws, stream=None):
    _check(_lib.nsd_ttv(C.byref(T), _p(x), _p(v), _p(y), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_ttv")


def nsd_ttv_vjp(T: nsd_ttv_plan, x, v, gy, dx, dv, ws, stream=None):
    _check(_lib.nsd_ttv_vjp(C.byref(T), _p(x), _p(v), _p(gy), _p(dx), _p(dv), _p(ws), _nbytes(ws),
                            _stream(stream)), "nsd_ttv_vjp")


def nsd_ttm_workspace_size(T: nsd_ttv_plan, R: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_ttm_workspace_size(C.byref(T), R, C.byref(b)), "nsd_ttm_workspace_size")
    return b.value


def nsd_ttm(T: nsd_ttv_plan, x, U, R, Y, ws, stream=None):
    _check(_lib.nsd_ttm(C.byref(T), _p(x), _p(U), R, _p(Y), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_ttm")


def nsd_ttm_vjp(T: nsd_ttv_plan, x, U, R, gY, dx, dU, ws, stream=None):
    _check(_lib.nsd_ttm_vjp(C.byref(T), _p(x), _p(U), R, _p(gY), _p(dx), _p(dU), _p(ws),
                            _nbytes(ws), _stream(stream)), "nsd_ttm_vjp")


# ------------------------------------------------------------ BATAX Jacobian

def nsd_batax_pairs(A: nsd_csr, ws, stream=None) -> int:
    n = C.c_int64(0)
    _check(_lib.nsd_batax_pairs(C.byref(A), C.byref(n), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_batax_pairs")
    return n.value


def nsd_batax_workspace_size(A: nsd_csr, npairs: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_batax_workspace_size(C.byref(A), npairs, C.byref(b)),
           "nsd_batax_workspace_size")
    return b.value


def nsd_batax_jacobian(A: nsd_csr, beta, npairs, jrowptr, jcolind, jval, ws, stream=None) -> int:
    out = _I(0)
    _check(_lib.nsd_batax_jacobian(C.byref(A), beta, npairs, _p(jrowptr), _p(jcolind), _p(jval),
                                   C.byref(out), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_batax_jacobian")
    return out.value


# ------------------------------------------------------ forward-mode tangent

def nsd_spmm_jvp(A: nsd_csr, dAval, B, dB, k, C_out, dC, ws, stream=None):
    _check(_lib.nsd_spmm_jvp(C.byref(A), _p(dAval), _p(B), _p(dB), k, _p(C_out), _p(dC), _p(ws),
                             _nbytes(ws), _stream(stream)), "nsd_spmm_jvp")


def nsd_spmm_jvp_batch_workspace_size(A: nsd_csr, k: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_spmm_jvp_batch_workspace_size(C.byref(A), k, C.byref(b)),
           "nsd_spmm_jvp_batch_workspace_size")
    return b.value


def nsd_spmm_jvp_batch(A: nsd_csr, m, dAval, B, dB, k, C_out, dC, ws, stream=None):
    _check(_lib.nsd_spmm_jvp_batch(C.byref(A), m, _p(dAval), _p(B), _p(dB), k, _p(C_out),
                                   _p(dC), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_spmm_jvp_batch")


# --------------------------------------------------- order-N CP gradient

def nsd_cpn_workspace_size(X: nsd_coon, rank: int) -> int:
    b = _SZ(0)
    _check(_lib.nsd_cpn_workspace_size(C.byref(X), rank, C.byref(b)), "nsd_cpn_workspace_size")
    return b.value


def nsd_loss_cpn(X: nsd_coon, F, rank, seed, loss, dX, dF, ws, stream=None):
    """F, dF: sequences of `order` device tensors (passed as a host array of
    device pointers)."""
    fp = (_P * len(F))(*[_p(f) for f in F])
    dp = (_P * len(dF))(*[_p(t) for t in dF])
    _check(_lib.nsd_loss_cpn(C.byref(X), fp, rank, seed, _p(loss), _p(dX), dp, _p(ws),
                             _nbytes(ws), _stream(stream)), "nsd_loss_cpn")


def nsd_dot(n, x, y, alpha, accumulate, out, ws, stream=None):
    _check(_lib.nsd_dot(n, _p(x), _p(y), alpha, int(bool(accumulate)), _p(out), _p(ws),
                        _nbytes(ws), _stream(stream)), "nsd_dot")


def nsd_axpby(n, alpha, x, beta, y, stream=None):
    _check(_lib.nsd_axpby(n, alpha, _p(x), beta, _p(y), _stream(stream)), "nsd_axpby")


def nsd_scale(n, alpha, s1, s2, x1, x2, x2_idx, beta, y, y_idx=None, stream=None):
    _check(_lib.nsd_scale(n, alpha, _p(s1), _p(s2), _p(x1), _p(x2), _p(x2_idx), beta, _p(y),
                          _p(y_idx), _stream(stream)), "nsd_scale")


def nsd_scale_real(alpha, s1, s2, x, beta, y, stream=None):
    _check(_lib.nsd_scale_real(alpha, _p(s1), _p(s2), _p(x), beta, _p(y), _stream(stream)),
           "nsd_scale_real")


def nsd_diag_keys(A: nsd_csr, alpha, out, stream=None):
    _check(_lib.nsd_diag_keys(C.byref(A), alpha, _p(out), _stream(stream)), "nsd_diag_keys")


def nsd_spmm_vjp(A: nsd_csr, At: nsd_csc, X, G, k, dA, dX, ws, stream=None):
    _check(_lib.nsd_spmm_vjp(C.byref(A), C.byref(At), _p(X), _p(G), k, _p(dA), _p(dX), _p(ws),
                             _nbytes(ws), _stream(stream)), "nsd_spmm_vjp")


def nsd_spmv_vjp(A: nsd_csr, At: nsd_csc, x, gy, dA, dx, ws, stream=None):
    _check(_lib.nsd_spmv_vjp(C.byref(A), C.byref(At), _p(x), _p(gy), _p(dA), _p(dx), _p(ws),
                             _nbytes(ws), _stream(stream)), "nsd_spmv_vjp")


def _host_i32(vals):
    return (C.c_int32 * len(vals))(*[int(v) for v in vals])


def nsd_validate_coo_workspace_size(dims, nnz) -> int:
    out = _SZ(0)
    _check(_lib.nsd_validate_coo_workspace_size(len(dims), C.cast(_host_i32(dims), _P), nnz,
                                                C.byref(out)), "nsd_validate_coo_workspace_size")
    return out.value


def nsd_validate_coo(dims, nnz, coords, check_unique, ws, stream=None):
    ptrs = (C.c_void_p * len(coords))(*[_p(c) for c in coords])
    _check(_lib.nsd_validate_coo(len(dims), C.cast(_host_i32(dims), _P), nnz, C.cast(ptrs, _P),
                                 int(bool(check_unique)), _p(ws), _nbytes(ws), _stream(stream)),
           "nsd_validate_coo")
