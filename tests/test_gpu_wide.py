"""Every fused loss at any dense width: k above what one slot of the fused
kernels holds (256 columns with 16-byte aligned rows, 64 otherwise), widths
that are not a multiple of 4, and rows that are not 16-byte aligned, against
the fp64 oracle; and the scalar-lane slots of 16, 32 and 64 lanes that
widths in 9..63 with k % 4 != 0 take on the fused passes.
"""
import numpy as np
import pytest
import torch

from helpers import assert_mag_close
from test_gpu_parity import (check_cp, check_cpn, check_frob, dev, edge_pattern, host,
                             in_input_order, oracle_dok, run_bilinear, run_cp, run_cpn,
                             run_frob)

pytestmark = pytest.mark.gpu

WIDE = [257, 300, 513, 70]     # above a fused slot; 70: scalar lanes above 64
SCALAR = [13, 30, 50]          # scalar lanes, slots of 16, 32 and 64 lanes


@pytest.fixture(scope="module")
def nsd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import nsd as m
    return m


@pytest.fixture(scope="module")
def operand(nsd):
    from paper_2303_07030_amd.operand import DeviceCsr
    return DeviceCsr


def dev_offset(a):
    """a on the device at a 4-byte offset from a 16-byte boundary (rows not
    16-byte aligned whatever the width)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    base = torch.empty(a.size + 1, dtype=torch.float32, device="cuda")
    t = base[1:].view(a.shape)
    t.copy_(torch.from_numpy(a))
    assert t.data_ptr() % 16 == 4
    return t


def empty_offset(shape):
    n = int(np.prod(shape))
    t = torch.full((n + 1,), np.nan, dtype=torch.float32, device="cuda")[1:].view(shape)
    assert t.data_ptr() % 16 == 4
    return t


# ----------------------------------------------------------- factorisation

def mf_case(k, seed=13):
    nrows, ncols, rowptr, colind, val = edge_pattern(seed)
    val = (1 + 4 * np.abs(val)).astype(np.float32)
    rng = np.random.default_rng(k)
    U = (0.1 * rng.standard_normal((nrows, k))).astype(np.float32)
    V = (0.1 * rng.standard_normal((ncols, k))).astype(np.float32)
    return nrows, ncols, rowptr, colind, val, U, V


def check_mf_all(orc, D, U, V, k, Lg, dUg, dVg, seed):
    L, Lm = orc.mf_loss(D, U, V, k)
    dU, dUm = orc.mf_grad(D, U, V, k, 0)
    dV, dVm = orc.mf_grad(D, U, V, k, 1)
    assert_mag_close(Lg, L, Lm, what="loss")
    assert_mag_close(dUg, seed * dU, abs(seed) * dUm, what="dU")
    assert_mag_close(dVg, seed * dV, abs(seed) * dVm, what="dV")


@pytest.mark.parametrize("k", WIDE + SCALAR)
@pytest.mark.parametrize("with_valT", [True, False])
def test_loss_mf_any_width(nsd, operand, orc, k, with_valT):
    nrows, ncols, rowptr, colind, val, U, V = mf_case(k)
    A = operand(nrows, ncols, rowptr, colind, val, k_hint=k)
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dU = torch.full((nrows, k), np.nan, dtype=torch.float32, device="cuda")
    dV = torch.full((ncols, k), np.nan, dtype=torch.float32, device="cuda")
    valT = A.values_in_csc_order() if with_valT else None
    nsd.nsd_loss_mf(A.desc, A.csc, valT, dev(U), dev(V), k, 0.5, loss, dU, dV, A.workspace(k))
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    check_mf_all(orc, D, U, V, k, host(loss)[0], host(dU), host(dV), 0.5)


@pytest.mark.parametrize("k", [128, 256])
def test_loss_mf_unaligned_rows(nsd, operand, orc, k):
    # a multiple of 4 that a fused slot holds only with 16-byte aligned rows
    nrows, ncols, rowptr, colind, val, U, V = mf_case(k, seed=17)
    A = operand(nrows, ncols, rowptr, colind, val, k_hint=k)
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dU, dV = empty_offset((nrows, k)), empty_offset((ncols, k))
    nsd.nsd_loss_mf(A.desc, A.csc, None, dev_offset(U), dev_offset(V), k, -1.5, loss, dU, dV,
                    A.workspace(k))
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    check_mf_all(orc, D, U, V, k, host(loss)[0], host(dU), host(dV), -1.5)


def test_loss_mf_wide_repeats_bitwise(nsd, operand):
    nrows, ncols, rowptr, colind, val, U, V = mf_case(300)
    A = operand(nrows, ncols, rowptr, colind, val, k_hint=300)
    outs = []
    for _ in range(2):
        loss = torch.empty(1, dtype=torch.float64, device="cuda")
        dU = torch.empty((nrows, 300), dtype=torch.float32, device="cuda")
        dV = torch.empty((ncols, 300), dtype=torch.float32, device="cuda")
        nsd.nsd_loss_mf(A.desc, A.csc, None, dev(U), dev(V), 300, 1.0, loss, dU, dV,
                        A.workspace(300))
        outs.append((host(loss), host(dU), host(dV)))
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


# ------------------------------------------------- bilinear, SpMM, SMVM

@pytest.mark.parametrize("k", WIDE + SCALAR)
def test_loss_bilinear_any_width(nsd, operand, orc, k):
    nrows, ncols, rowptr, colind, val = edge_pattern(21)
    A = operand(nrows, ncols, rowptr, colind, val, k_hint=k)
    rng = np.random.default_rng(k)
    H = rng.standard_normal((ncols, k)).astype(np.float32)
    G = rng.standard_normal((nrows, k)).astype(np.float32)
    Lg, dAg, dHg = run_bilinear(nsd, A, H, G, k, seed=0.25)
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    L, Lm = orc.loss_bilinear(D, G, H, k)
    dA, dAm = orc.sddmm(D, G, H, k, rows, colind, alpha=0.25)
    dH, dHm = orc.spmm_t(D, G, k, alpha=0.25)
    assert_mag_close(Lg, L, Lm, what="loss")
    assert_mag_close(dAg, dA, dAm, what="dA")
    assert_mag_close(dHg, dH, dHm, what="dH")


@pytest.mark.parametrize("k", WIDE + SCALAR)
def test_loss_frob_spmm_any_width(nsd, operand, orc, k):
    nrows, ncols, rowptr, colind, val = edge_pattern(22)
    A = operand(nrows, ncols, rowptr, colind, val, k_hint=k)
    B = np.random.default_rng(k).standard_normal((ncols, k)).astype(np.float32)
    got = run_frob(nsd, A, B, k, seed=2.0)
    check_frob(orc, nrows, ncols, rowptr, colind, val, B, k, got, seed=2.0)


@pytest.mark.parametrize("k", [300, 70])
def test_loss_bilinear_unaligned_rows(nsd, operand, orc, k):
    nrows, ncols, rowptr, colind, val = edge_pattern(23)
    A = operand(nrows, ncols, rowptr, colind, val, k_hint=k)
    rng = np.random.default_rng(k + 1)
    H = rng.standard_normal((ncols, k)).astype(np.float32)
    G = rng.standard_normal((nrows, k)).astype(np.float32)
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dA = torch.empty(A.nnz, dtype=torch.float32, device="cuda")
    dH = empty_offset((ncols, k))
    nsd.nsd_loss_bilinear(A.desc, A.csc, dev_offset(H), dev_offset(G), k, 1.0, loss, dA, dH,
                          A.workspace(k))
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    L, Lm = orc.loss_bilinear(D, G, H, k)
    dAr, dAm = orc.sddmm(D, G, H, k, rows, colind)
    dHr, dHm = orc.spmm_t(D, G, k)
    assert_mag_close(host(loss)[0], L, Lm, what="loss")
    assert_mag_close(host(dA), dAr, dAm, what="dA")
    assert_mag_close(host(dH), dHr, dHm, what="dH")


# -------------------------------------------------------------------- CP

def cp_case(rank, dims=(20, 30, 25), nnz=3000):
    rng = np.random.default_rng(rank)
    total = int(np.prod(dims))
    keys = rng.choice(total, size=nnz, replace=False)
    i, j, l = (c.astype(np.int32) for c in np.unravel_index(keys, dims))
    val = rng.standard_normal(nnz).astype(np.float32)
    F = [(0.2 * rng.standard_normal((d, rank))).astype(np.float32) for d in dims]
    return dims, i, j, l, val, F


@pytest.mark.parametrize("rank", WIDE + SCALAR)
def test_loss_cp_any_rank(nsd, orc, rank):
    from paper_2303_07030_amd.operand import DeviceCoo3
    dims, i, j, l, val, F = cp_case(rank)
    X = DeviceCoo3(dims, i, j, l, val, rank_hint=rank)
    got = run_cp(nsd, X, F, rank, seed=0.75)
    check_cp(orc, dims, i, j, l, val, F, rank, got, seed=0.75)


def test_loss_cp_unaligned_rows(nsd, orc):
    from paper_2303_07030_amd.operand import DeviceCoo3
    rank = 128
    dims, i, j, l, val, F = cp_case(rank, dims=(15, 40, 12))
    X = DeviceCoo3(dims, i, j, l, val, rank_hint=rank)
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dX = torch.full((X.nnz,), np.nan, dtype=torch.float32, device="cuda")
    dF = [empty_offset((d, rank)) for d in dims]
    nsd.nsd_loss_cp(X.desc, *[dev_offset(f) for f in F], rank, 1.0, loss, dX, *dF,
                    X.workspace(rank))
    got = (host(loss)[0], in_input_order(X, host(dX)), [host(t) for t in dF])
    check_cp(orc, dims, i, j, l, val, F, rank, got)


@pytest.mark.parametrize("dims,rank", [((8, 9, 7, 6), 257), ((8, 9, 7, 6), 70),
                                       ((5, 4, 3, 6, 4), 300), ((30, 2, 2, 2), 513),
                                       ((6, 5, 4, 3), 30)])
def test_loss_cpn_any_rank(nsd, orc, dims, rank):
    from paper_2303_07030_amd.operand import DeviceCooN
    rng = np.random.default_rng(len(dims) * 1000 + rank)
    size = int(np.prod(dims))
    nnz = min(size // 2, 1500)
    keys = rng.choice(size, size=nnz, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(keys, dims)]
    val = rng.standard_normal(nnz).astype(np.float32)
    F = [(0.3 * rng.standard_normal((d, rank))).astype(np.float32) for d in dims]
    X = DeviceCooN(dims, coords, val, rank_hint=rank, item_len=16)
    got = run_cpn(nsd, X, F, rank, seed=0.5)
    check_cpn(orc, dims, coords, val, F, rank, got, seed=0.5)


def test_wide_losses_on_empty_operands(nsd, operand):
    """No stored entry: the wide forms write zero gradients and a zero loss."""
    from paper_2303_07030_amd.operand import DeviceCoo3
    k = 300
    A = operand(5, 7, np.zeros(6, np.int32), np.empty(0, np.int32), np.empty(0, np.float32),
                k_hint=k)
    loss = torch.full((1,), np.nan, dtype=torch.float64, device="cuda")
    dU = torch.full((5, k), np.nan, dtype=torch.float32, device="cuda")
    dV = torch.full((7, k), np.nan, dtype=torch.float32, device="cuda")
    U = torch.zeros((5, k), device="cuda")
    V = torch.zeros((7, k), device="cuda")
    nsd.nsd_loss_mf(A.desc, A.csc, None, U, V, k, 1.0, loss, dU, dV, A.workspace(k))
    assert host(loss)[0] == 0 and np.all(host(dU) == 0) and np.all(host(dV) == 0)
    e = np.empty(0, np.int32)
    X = DeviceCoo3((4, 5, 6), e, e, e, np.empty(0, np.float32), rank_hint=k)
    F = [torch.zeros((d, k), device="cuda") for d in (4, 5, 6)]
    dF = [torch.full((d, k), np.nan, dtype=torch.float32, device="cuda") for d in (4, 5, 6)]
    dX = torch.empty(1, dtype=torch.float32, device="cuda")
    nsd.nsd_loss_cp(X.desc, *F, k, 1.0, loss, dX, *dF, X.workspace(k))
    assert host(loss)[0] == 0 and all(np.all(host(t) == 0) for t in dF)
