"""Seeded random cases through the C ABI against the oracle.

Each case draws a shape, a row-length profile (power law with a random cap,
empty rows, sometimes one row spanning most columns), a dense width k and a
plan item length (the library's choice or a short one that cuts most rows
into chunks), so that the chunk partials, their in-wave sums at every group
offset and the combine (by waves or by workgroups) are all exercised at
widths taking every lane layout.  Same tolerance as the other parity tests.
"""
import numpy as np
import pytest
import torch

from helpers import assert_mag_close
from test_gpu_parity import (check_cp, check_cpn, check_frob, check_mf, dev, host, make_csr,
                             oracle_dok, run_bilinear, run_cp, run_cpn, run_frob, run_mf)

pytestmark = pytest.mark.gpu

# 13, 30 and 50 take scalar-lane slots of 16, 32 and 64 lanes on the fused
# passes; 70, 264 and 300 are wider than a fused slot
KS = [1, 2, 3, 5, 8, 12, 13, 16, 24, 30, 32, 48, 50, 64, 70, 100, 128, 200, 256, 264, 300]
ITEM_LENS = [None, 2, 3, 4, 7, 8, 16, 33, 64]


@pytest.fixture(scope="module")
def nsd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import nsd as m
    return m


def random_csr(rng):
    nrows, ncols = int(rng.integers(1, 2000)), int(rng.integers(1, 2000))
    cap = int(rng.integers(1, ncols + 1))
    lengths = np.minimum((rng.pareto(rng.uniform(0.8, 2.0), nrows) * rng.uniform(1, 30))
                         .astype(np.int64), cap)
    lengths[rng.random(nrows) < 0.1] = 0
    if rng.random() < 0.5:
        lengths[rng.integers(nrows)] = int(ncols * rng.uniform(0.5, 1.0))
    if lengths.sum() == 0:  # empty operands have tests of their own
        lengths[0] = 1
    return nrows, ncols, *make_csr(rng, nrows, ncols, lengths)


@pytest.mark.parametrize("case", range(64))
def test_random_csr_paths(nsd, orc, case):
    from paper_2303_07030_amd.operand import DeviceCsr
    rng = np.random.default_rng(1000 + case)
    nrows, ncols, rowptr, colind, val = random_csr(rng)
    k = KS[case % len(KS)]  # every width, with changing item lengths
    L = ITEM_LENS[(7 * case) % len(ITEM_LENS)]
    what = f"case {case}: {nrows}x{ncols}, nnz {len(colind)}, k {k}, item_len {L}"
    A = DeviceCsr(nrows, ncols, rowptr, colind, val, item_len=L, k_hint=k)
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    B = rng.standard_normal((ncols, k)).astype(np.float32)
    G = rng.standard_normal((nrows, k)).astype(np.float32)

    C = torch.full((nrows, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm(A.desc, dev(B), k, C, A.workspace(k))
    ref, mag = orc.spmm(D, B, k)
    assert_mag_close(host(C), ref, mag, what=f"spmm, {what}")

    T = torch.full((ncols, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm_t(A.desc, A.csc, dev(G), k, -0.5, T, A.workspace(k))
    ref, mag = orc.spmm_t(D, G, k, alpha=-0.5)
    assert_mag_close(host(T), ref, mag, what=f"spmm_t, {what}")

    S = torch.full((max(len(colind), 1),), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_sddmm(A.desc, dev(G), dev(B), k, 2.0, S)
    ref, mag = orc.sddmm(D, G, B, k, rows, colind, alpha=2.0)
    assert_mag_close(host(S)[: len(colind)], ref, mag, what=f"sddmm, {what}")

    check_frob(orc, nrows, ncols, rowptr, colind, val, B, k, run_frob(nsd, A, B, k, 1.5),
               seed=1.5)

    # every fused loss takes every width (wider ones in their unfused form)
    Lg, dAg, dHg = run_bilinear(nsd, A, B, G, k)
    L, Lm = orc.loss_bilinear(D, G, B, k)
    assert_mag_close(Lg, L, Lm, what=f"bilinear loss, {what}")
    ref, mag = orc.sddmm(D, G, B, k, rows, colind)
    assert_mag_close(dAg[: len(colind)], ref, mag, what=f"bilinear dA, {what}")
    ref, mag = orc.spmm_t(D, G, k)
    assert_mag_close(dHg, ref, mag, what=f"bilinear dH, {what}")

    U = (0.3 * rng.standard_normal((nrows, k))).astype(np.float32)
    V = (0.3 * rng.standard_normal((ncols, k))).astype(np.float32)
    check_mf(orc, D, U, V, k, run_mf(nsd, A, U, V, k))


@pytest.mark.parametrize("case", range(32))
def test_random_cp_paths(nsd, orc, case):
    from paper_2303_07030_amd.operand import DeviceCoo3, DeviceCooN
    rng = np.random.default_rng(2000 + case)
    order = 3 if case % 2 == 0 else 4
    dims = tuple(int(d) for d in rng.integers(1, 60, order))
    size = int(np.prod(dims))
    nnz = int(rng.integers(1, min(size, 30_000) + 1))
    flat = rng.choice(size, size=nnz, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(flat, dims)]
    val = rng.standard_normal(nnz).astype(np.float32)
    rank = int(rng.choice([1, 2, 3, 4, 8, 13, 16, 30, 32, 33, 50, 64, 70, 257]))
    L = [None, 2, 5, 8, 24][int(rng.integers(5))]
    F = [(0.5 * rng.standard_normal((d, rank))).astype(np.float32) for d in dims]
    if order == 3:
        X = DeviceCoo3(dims, *coords, val, rank_hint=rank, item_len=L)
        check_cp(orc, dims, *coords, val, F, rank, run_cp(nsd, X, F, rank))
    else:
        X = DeviceCooN(dims, coords, val, rank_hint=rank, item_len=L)
        check_cpn(orc, dims, coords, val, F, rank, run_cpn(nsd, X, F, rank))
