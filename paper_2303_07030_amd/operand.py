"""Device-resident sparse operands for the hot path.

A DeviceCsr holds a CSR in HBM together with the arrays the gradient
kernels read: rowidx (the row of every stored entry), the work plan over the
rows, and the CSC of the same matrix (colptr, colidx, rowind, perm) with its
plan over the columns.  All of them are produced by the library's own
builders; this module only allocates torch tensors and calls the binding.
"""
from __future__ import annotations

import numpy as np
import torch

from . import nsd


def _dev(a, dtype, device):
    if isinstance(a, torch.Tensor):
        return a.to(device=device, dtype=dtype)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dtype)


def build_plan(nseg, nnz, segptr, item_len, device, stream=None):
    """Work plan of a segment pointer array (device tensors kept alive on it)."""
    max_items, max_long, max_chunks, wsb = nsd.nsd_plan_bounds(nseg, nnz, item_len)

    def arr(n):
        return torch.empty(max(n, 1), dtype=torch.int32, device=device)

    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device=device)
    return nsd.nsd_plan_build(nseg, nnz, segptr, item_len, arr(max_items + 1), arr(max_long),
                              arr(max_long), arr(max_long), arr(max_chunks), arr(max_items),
                              arr(nseg), ws, stream)


# Patterns with at least this many entries get the two-pass forms of their
# CSC permutation (nsd_perm_plan_build) unless asked otherwise: below it the
# two extra launches of a move cost more than the scattered 4-byte accesses
# they replace.
PERM_PLAN_MIN_NNZ = 4_000_000


def build_perm_plan(n, perm, inverse, device, stream=None):
    """Two-pass form of a permutation (device arrays kept alive on it)."""
    stage = torch.empty(max(n, 1), dtype=torch.int32, device=device)
    src_local = torch.empty(max(n, 1), dtype=torch.uint16, device=device)
    dst_local = torch.empty(max(n, 1), dtype=torch.uint16, device=device)
    ws = torch.empty(max(nsd.nsd_perm_plan_workspace_size(n), 256), dtype=torch.uint8,
                     device=device)
    return nsd.nsd_perm_plan_build(n, perm, inverse, stage, src_local, dst_local, ws, stream)


class DeviceCsr:
    def __init__(self, nrows: int, ncols: int, rowptr, colind, val, device="cuda",
                 build_csc: bool = True, stream=None, k_hint: int = 64, item_len=None,
                 rowidx=None, perm_plans=None):
        """perm_plans: build the two-pass forms of the CSC permutation (None:
        when nnz >= PERM_PLAN_MIN_NNZ)."""
        self.perm_plans = perm_plans
        self.nrows, self.ncols = int(nrows), int(ncols)
        self.rowptr = _dev(rowptr, torch.int32, device)
        self.colind = _dev(colind, torch.int32, device)
        self.val = _dev(val, torch.float32, device)
        self.nnz = int(self.colind.numel())
        if rowidx is None:
            self.rowidx = torch.empty(self.nnz, dtype=torch.int32, device=device)
            nsd.nsd_csr_expand_rows(self.nrows, self.nnz, self.rowptr, self.rowidx, stream)
        else:
            self.rowidx = rowidx
        self.desc = nsd.csr_desc(self.nrows, self.ncols, self.rowptr, self.rowidx, self.colind,
                                 self.val)
        self.item_len = item_len or nsd.nsd_plan_item_len(self.nnz, k_hint)
        self.row_plan = build_plan(self.nrows, self.nnz, self.rowptr, self.item_len, device,
                                   stream)
        self.desc.plan = self.row_plan
        self.csc = None
        if build_csc:
            self.build_csc(stream)

    def build_csc(self, stream=None):
        dev = self.rowptr.device
        self.colptr = torch.empty(self.ncols + 1, dtype=torch.int32, device=dev)
        self.colidx = torch.empty(self.nnz, dtype=torch.int32, device=dev)
        self.rowind = torch.empty(self.nnz, dtype=torch.int32, device=dev)
        self.perm = torch.empty(self.nnz, dtype=torch.int32, device=dev)
        ws = torch.empty(nsd.nsd_build_workspace_size(self.nnz, max(self.ncols, 1)),
                         dtype=torch.uint8, device=dev)
        nsd.nsd_csr_to_csc(self.desc, self.colptr, self.colidx, self.rowind, self.perm, ws, stream)
        self.csc = nsd.csc_desc(self.nrows, self.ncols, self.colptr, self.colidx, self.rowind,
                                self.perm)
        self.col_plan = build_plan(self.ncols, self.nnz, self.colptr, self.item_len, dev, stream)
        self.csc.plan = self.col_plan
        plans = self.perm_plans
        if plans is None:
            plans = self.nnz >= PERM_PLAN_MIN_NNZ
        if plans and self.nnz > 0:
            # the descriptor holds copies of the plans; their arrays live here
            self.to_csc = build_perm_plan(self.nnz, self.perm, 0, dev, stream)
            self.to_csr = build_perm_plan(self.nnz, self.perm, 1, dev, stream)
            self.csc.to_csc, self.csc.to_csr = self.to_csc, self.to_csr
        return self.csc

    def workspace(self, k: int):
        n = nsd.nsd_workspace_size(self.desc, self.csc, k)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.rowptr.device)

    @classmethod
    def from_coo(cls, nrows, ncols, row, col, val, device="cuda", policy=None, **kw):
        """CSR of a COO input built on the GPU by nsd_coo_to_csr; `coo_perm`
        maps every CSR slot to the input position of its first occurrence."""
        row = _dev(row, torch.int32, device)
        col = _dev(col, torch.int32, device)
        v = _dev(val, torch.float32, device)
        n = int(row.numel())
        rowptr = torch.empty(nrows + 1, dtype=torch.int32, device=device)
        rowidx = torch.empty(max(n, 1), dtype=torch.int32, device=device)
        colind = torch.empty(max(n, 1), dtype=torch.int32, device=device)
        vout = torch.empty(max(n, 1), dtype=torch.float32, device=device)
        perm = torch.empty(max(n, 1), dtype=torch.int32, device=device)
        ws = torch.empty(nsd.nsd_build_workspace_size(n, max(nrows, ncols, 1)), dtype=torch.uint8,
                         device=device)
        pol = nsd.NSD_DUP_SUM if policy is None else policy
        m = nsd.nsd_coo_to_csr(nrows, ncols, n, row, col, v, pol, rowptr, rowidx, colind, vout,
                               perm, ws)
        A = cls(nrows, ncols, rowptr, colind[:m], vout[:m], device=device, rowidx=rowidx[:m], **kw)
        A.coo_perm = perm[:m]
        return A

    def values_in_csc_order(self, stream=None):
        """A's values permuted into CSC order (an exact copy, nsd_gather_f32)."""
        valT = torch.empty(max(self.nnz, 1), dtype=torch.float32, device=self.val.device)
        nsd.nsd_gather_f32(self.nnz, self.perm, self.val, valT, stream)
        return valT[: self.nnz]


class DeviceSparseVec:
    """A sparse vector in HBM: its stored keys (int32, strictly increasing, in
    [0, n)) and their values.  The keys are checked by nsd_validate_csr on
    the 1 x n matrix they form (distinct keys are what lets a result be
    scattered into a dense vector with one write per key)."""

    def __init__(self, n: int, keys, val, device="cuda", stream=None):
        self.n = int(n)
        self.keys = _dev(keys, torch.int32, device).contiguous()
        self.val = _dev(val, torch.float32, device).contiguous()
        self.nnz = int(self.keys.numel())
        if self.val.numel() != self.nnz:
            raise ValueError(f"{self.nnz} keys and {self.val.numel()} values")
        rowptr = torch.tensor([0, self.nnz], dtype=torch.int32, device=device)
        ws = torch.empty(256, dtype=torch.uint8, device=device)
        nsd.nsd_validate_csr(nsd.csr_desc(1, self.n, rowptr, None, self.keys, self.val), True,
                             ws, stream)


def lex_order(coords, dims, ws, stream=None):
    """Permutation q -> input position that sorts COO entries by (c0, c1, ...)
    lexicographically: stable sorts by the last coordinate first, each one the
    library's mode index, composed by the library's gather."""
    n = int(coords[0].numel())
    dev = coords[0].device
    m_ = max(n, 1)
    perm = None
    for m in reversed(range(len(coords))):
        key = coords[m]
        if perm is not None:
            key = torch.empty(m_, dtype=torch.int32, device=dev)
            nsd.nsd_gather_i32(n, perm, coords[m], key, stream)
        segptr = torch.empty(int(dims[m]) + 1, dtype=torch.int32, device=dev)
        segidx = torch.empty(m_, dtype=torch.int32, device=dev)
        p = torch.empty(m_, dtype=torch.int32, device=dev)
        nsd.nsd_coo_mode_index(n, int(dims[m]), key, segptr, segidx, p, ws, stream)
        if perm is None:
            perm = p
        else:
            composed = torch.empty(m_, dtype=torch.int32, device=dev)
            nsd.nsd_gather_i32(n, p, perm, composed, stream)
            perm = composed
    return perm[:n]


def _stored_in_lex_order(coords, val, dims, ws, stream):
    """(coordinates, values, coo_perm) with the entries in lexicographic
    coordinate order; coo_perm[q] is the input position of stored entry q."""
    n = int(val.numel())
    perm = lex_order(coords, dims, ws, stream)
    out = []
    for c in coords:
        t = torch.empty(max(n, 1), dtype=torch.int32, device=val.device)
        nsd.nsd_gather_i32(n, perm, c, t, stream)
        out.append(t[:n])
    v = torch.empty(max(n, 1), dtype=torch.float32, device=val.device)
    nsd.nsd_gather_f32(n, perm, val, v, stream)
    return out, v[:n], perm


class DeviceCoo3:
    """A COO 3-tensor in HBM, stored in lexicographic (i, j, l) order (the
    order its first mode pass walks, so the residual on X's keys is written
    sequentially), and in its three mode orders: for every mode n the
    library's mode index (stable sort by the mode-n coordinate over the
    stored order), the other two coordinates and the values gathered into
    that order, and the work plan over the mode-n slices.  `coo_perm[q]` is
    the input position of stored entry q; gradients on X's keys come out in
    the stored order (as a CSR's values do)."""

    def __init__(self, dims, i, j, l, val, device="cuda", rank_hint=32, item_len=None,
                 stream=None):
        self.dims = tuple(int(d) for d in dims)
        coords = [_dev(c, torch.int32, device) for c in (i, j, l)]
        val = _dev(val, torch.float32, device)
        self.nnz = int(val.numel())
        # shorter items than the library's general choice: measured on
        # MI355X, 3/8 of it is best for the fused order-3 CP pass (24 entries
        # at 20M entries, rank 32: 1.05 ms per step against 1.08 at 16 and
        # 1.10 at 32)
        self.item_len = item_len or max(8, nsd.nsd_plan_item_len(self.nnz, rank_hint) * 3 // 8)
        self.desc = nsd.nsd_coo3()
        self.desc.dims[:] = self.dims
        self.desc.nnz = self.nnz
        self._keep = []
        ws = torch.empty(nsd.nsd_build_workspace_size(self.nnz, max(max(self.dims), 1)),
                         dtype=torch.uint8, device=device)
        coords, self.val, self.coo_perm = _stored_in_lex_order(coords, val, self.dims, ws,
                                                               stream)
        self.coords = coords
        n = max(self.nnz, 1)
        for m in range(3):
            segptr = torch.empty(self.dims[m] + 1, dtype=torch.int32, device=device)
            segidx = torch.empty(n, dtype=torch.int32, device=device)
            perm = torch.empty(n, dtype=torch.int32, device=device)
            nsd.nsd_coo_mode_index(self.nnz, self.dims[m], coords[m], segptr, segidx, perm, ws,
                                   stream)
            ia = torch.empty(n, dtype=torch.int32, device=device)
            ib = torch.empty(n, dtype=torch.int32, device=device)
            v = torch.empty(n, dtype=torch.float32, device=device)
            nsd.nsd_gather_i32(self.nnz, perm, coords[(m + 1) % 3], ia, stream)
            nsd.nsd_gather_i32(self.nnz, perm, coords[(m + 2) % 3], ib, stream)
            nsd.nsd_gather_f32(self.nnz, perm, self.val, v, stream)
            plan = build_plan(self.dims[m], self.nnz, segptr, self.item_len, device, stream)
            md = self.desc.mode[m]
            md.mode = m
            md.segptr, md.segidx, md.idx_a, md.idx_b = (segptr.data_ptr(), segidx.data_ptr(),
                                                        ia.data_ptr(), ib.data_ptr())
            md.val, md.perm = v.data_ptr(), perm.data_ptr()
            md.plan = plan
            self._keep += [segptr, segidx, perm, ia, ib, v, plan]

    def workspace(self, rank: int):
        n = nsd.nsd_cp_workspace_size(self.desc, rank)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.val.device)


class DeviceCooN:
    """A COO tensor of order 3 to 6 in HBM, stored in lexicographic
    coordinate order (`coo_perm[q]` is the input position of stored entry q;
    gradients on X's keys come out in the stored order), and in all its mode
    orders: for every mode n the library's mode index (stable sort by
    coordinate n), the other coordinates (modes n+1, n+2, ... mod order) and
    the values gathered into that order, and the work plan over the mode-n
    slices."""

    def __init__(self, dims, coords, val, device="cuda", rank_hint=32, item_len=None,
                 stream=None, fibers=False):
        """fibers: let the CP passes take each slice's runs of equal first
        other coordinate as fibers (the second level of a compressed-fiber
        tree); the lexicographic storage order makes them contiguous.  Off by
        default: with factor tables that stay in L2 the per-entry gather it
        saves is cheap, and the order-4 workload (1000^4, 20M entries, rank
        32, about 20 entries per fiber) measured 1.54 ms per launch with it
        against 1.52 without."""
        self.dims = tuple(int(d) for d in dims)
        N = self.order = len(self.dims)
        if not 3 <= N <= nsd.MAX_ORDER:
            raise ValueError(f"order {N} outside [3, {nsd.MAX_ORDER}]")
        coords = [_dev(c, torch.int32, device) for c in coords]
        val = _dev(val, torch.float32, device)
        self.nnz = int(val.numel())
        # 3/8 of the library's general item length, as for order 3: measured
        # best on MI355X for the order-4 CP pass (24 entries at 20M entries,
        # rank 32: 1.46 ms per step against 1.51 at 16 and 1.48 at 32)
        self.item_len = item_len or max(8, nsd.nsd_plan_item_len(self.nnz, rank_hint) * 3 // 8)
        self.desc = nsd.nsd_coon()
        self.desc.order = N
        for m in range(N):
            self.desc.dims[m] = self.dims[m]
        self.desc.nnz = self.nnz
        self._keep = []
        ws = torch.empty(nsd.nsd_build_workspace_size(self.nnz, max(max(self.dims), 1)),
                         dtype=torch.uint8, device=device)
        coords, self.val, self.coo_perm = _stored_in_lex_order(coords, val, self.dims, ws,
                                                               stream)
        self.coords = coords
        n = max(self.nnz, 1)
        self.modes = []
        for m in range(N):
            segptr = torch.empty(self.dims[m] + 1, dtype=torch.int32, device=device)
            segidx = torch.empty(n, dtype=torch.int32, device=device)
            perm = torch.empty(n, dtype=torch.int32, device=device)
            nsd.nsd_coo_mode_index(self.nnz, self.dims[m], coords[m], segptr, segidx, perm, ws,
                                   stream)
            others = []
            for o in range(N - 1):
                t = torch.empty(n, dtype=torch.int32, device=device)
                nsd.nsd_gather_i32(self.nnz, perm, coords[(m + 1 + o) % N], t, stream)
                others.append(t)
            v = torch.empty(n, dtype=torch.float32, device=device)
            nsd.nsd_gather_f32(self.nnz, perm, self.val, v, stream)
            plan = build_plan(self.dims[m], self.nnz, segptr, self.item_len, device, stream)
            md = self.desc.mode[m]
            md.mode = m
            md.segptr, md.segidx = segptr.data_ptr(), segidx.data_ptr()
            for o, t in enumerate(others):
                md.idx[o] = t.data_ptr()
            md.val, md.perm = v.data_ptr(), perm.data_ptr()
            md.plan = plan
            md.fiber = 1 if fibers else 0
            self._keep += [segptr, segidx, perm, v, plan] + others
            self.modes.append(dict(segptr=segptr, segidx=segidx, perm=perm, val=v, idx=others,
                                   plan=plan))

    def workspace(self, rank: int):
        n = nsd.nsd_cpn_workspace_size(self.desc, rank)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.val.device)


class DeviceTtv:
    """The projection of an order-N COO tensor (3 <= N <= 6) along one mode
    n (default: the last), built by nsd_ttv_build: the distinct keys of the
    other coordinates in lexicographic order (`ykey`, N - 1 arrays), work
    plans over those keys and over the mode-n coordinate.  It is the layout
    of the mode-n products nsd_ttv / nsd_ttm and their VJPs."""

    def __init__(self, dims, coords, mode=-1, device="cuda", item_len=16, stream=None):
        self.dims = tuple(int(d) for d in dims)
        N = len(self.dims)
        self.order = N
        self.mode = mode % N
        coords = [_dev(c, torch.int32, device) for c in coords]
        if len(coords) != N:
            raise ValueError(f"{len(coords)} coordinate arrays for an order-{N} tensor")
        nnz = int(coords[0].numel())
        n = max(nnz, 1)

        def arr(m):
            return torch.empty(max(m, 1), dtype=torch.int32, device=device)

        self.ykey = [arr(n) for _ in range(N - 1)]
        self.yptr = arr(nnz + 1)
        self.yseg, self.yperm, self.ykidx = arr(n), arr(n), arr(n)
        self.lptr, self.lseg, self.lperm, self.lpair = (arr(self.dims[self.mode] + 1), arr(n),
                                                        arr(n), arr(n))
        ws = torch.empty(max(nsd.nsd_ttv_build_workspace_size(N, self.dims, nnz), 256),
                         dtype=torch.uint8, device=device)
        self.ny = nsd.nsd_ttv_build(N, self.dims, nnz, coords, self.mode, self.ykey, self.yptr,
                                    self.yseg, self.yperm, self.ykidx, self.lptr, self.lseg,
                                    self.lperm, self.lpair, ws, stream)
        self.nnz = nnz
        self.yplan = build_plan(self.ny, nnz, self.yptr, item_len, device, stream)
        self.lplan = build_plan(self.dims[self.mode], nnz, self.lptr, item_len, device, stream)
        T = nsd.nsd_ttv_plan()
        T.order, T.mode = N, self.mode
        T.dims[:N] = self.dims
        T.nnz, T.ny = nnz, self.ny
        for o in range(N - 1):
            T.ykey[o] = self.ykey[o].data_ptr()
        for f in ("yptr", "yseg", "yperm", "ykidx", "lptr", "lseg", "lperm", "lpair"):
            setattr(T, f, getattr(self, f).data_ptr())
        T.yplan, T.lplan = self.yplan, self.lplan
        self.desc = T

    def workspace(self):
        n = nsd.nsd_ttv_workspace_size(self.desc)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.yptr.device)

    def ttm_workspace(self, R: int):
        """Workspace of nsd_ttm / nsd_ttm_vjp at width R."""
        n = nsd.nsd_ttm_workspace_size(self.desc, R)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.yptr.device)
