"""Jacobians of the vector kernels of the paper's evaluation, on the GPU.

With the gradient API, the tangent of a tensor-valued program under the
one-hot seed of an input x is the program's Jacobian with respect to x: the
output's keys first, x's keys after (Section 4.3; the batch of tangents of
Section 4.2).  For the two vector kernels of the evaluation (Section 7.1)
that tangent has a closed form on the stored keys, which these functions
build with the library's kernels (the Python side passes arguments only):

  * VVA, f(i) = V1(i) + V2(i):  df/dV1 holds 1 at (k, k) for every stored key
    k of V1 and nothing else: the seed passes through the sum unchanged, and
    the keys only V2 stores have a zero tangent;
  * VSM, f(i) = V(i) * s * s:  df/ds = 2 s V(i) on V's stored keys, and df/dV
    holds s^2 at (k, k) for every stored key k of V.

The trace (Example 3) is a real-valued program; its gradient goes through
the front end (`sdql`), lowered to nsd_diag_keys.
"""
from __future__ import annotations

import torch

from . import nsd
from .operand import DeviceCsr


def vva_jacobian(n: int, keys: torch.Tensor, stream=None) -> DeviceCsr:
    """d(V1 + V2)/dV1 for a sparse vector V1 of length n stored at `keys`
    (int32 device tensor of distinct indices): an n x n CSR with 1 at (k, k)
    for every stored key k (built by nsd_coo_to_csr from the pairs (k, k))."""
    keys = keys.to(dtype=torch.int32).contiguous()
    nnz = int(keys.numel())
    ones = torch.empty(max(nnz, 1), dtype=torch.float32, device=keys.device)
    nsd.nsd_axpby(nnz, 1.0, None, 0.0, ones, stream)
    return DeviceCsr.from_coo(n, n, keys, keys, ones[:nnz], device=keys.device,
                              policy=nsd.NSD_DUP_ERROR, build_csc=False)


def vsm_jacobian_s(val: torch.Tensor, s: float, out: torch.Tensor, stream=None):
    """d(V s s)/ds = 2 s V on V's stored keys: `out` (aligned with V's value
    array `val`) = (2 s) * val."""
    nsd.nsd_axpby(val.numel(), 2.0 * float(s), val, 0.0, out, stream)


def vsm_jacobian_v(nnz: int, s: float, out: torch.Tensor, stream=None):
    """d(V s s)/dV holds s^2 at (k, k) for V's stored keys: its diagonal as a
    value array aligned with V's keys."""
    nsd.nsd_axpby(nnz, float(s) * float(s), None, 0.0, out, stream)
