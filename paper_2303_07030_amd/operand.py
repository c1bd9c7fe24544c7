"""Device-resident sparse operands for the hot path.

A DeviceCsr holds a CSR in HBM together with the arrays the gradient
kernels read: rowidx (the row of every stored entry) and the CSC of the same
matrix (colptr, colidx, rowind, perm).  All of them are produced by the
library's own builders; this module only allocates torch tensors and calls
the binding.
"""
from __future__ import annotations

import numpy as np
import torch

from . import nsd


def _dev(a, dtype, device):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dtype)


class DeviceCsr:
    def __init__(self, nrows: int, ncols: int, rowptr, colind, val, device="cuda",
                 build_csc: bool = True, stream=None):
        self.nrows, self.ncols = int(nrows), int(ncols)
        self.rowptr = _dev(rowptr, torch.int32, device)
        self.colind = _dev(colind, torch.int32, device)
        self.val = _dev(val, torch.float32, device)
        self.nnz = int(self.colind.numel())
        self.rowidx = torch.empty(self.nnz, dtype=torch.int32, device=device)
        nsd.nsd_csr_expand_rows(self.nrows, self.nnz, self.rowptr, self.rowidx, stream)
        self.desc = nsd.csr_desc(self.nrows, self.ncols, self.rowptr, self.rowidx, self.colind,
                                 self.val)
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
        return self.csc

    def workspace(self, k: int):
        n = nsd.nsd_workspace_size(self.nnz, max(self.nrows, self.ncols), k)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.rowptr.device)
