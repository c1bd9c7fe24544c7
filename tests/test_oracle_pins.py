"""Pins for the fp64 oracle, against things other than the oracle itself.

Each check ties an oracle function to a library routine (scipy.sparse, numpy
sorts), to dense brute force with PyTorch CPU autograd in fp64 read at the
stored keys, to central finite differences, to closed forms the paper states,
or to special cases that reduce to a textbook routine.  A plausible slip in
the oracle (a dropped term, a transposed operand, a wrong sign or factor, an
index mix-up, a lost duplicate) fails at least one of them.
"""
import json
import os

import numpy as np
import pytest
import scipy.sparse as sp
import torch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_coo(rng, nr, nc, nnz, dups=0):
    keys = rng.choice(nr * nc, size=nnz, replace=False)
    if dups:
        keys = np.concatenate([keys, rng.choice(keys, size=dups)])
        rng.shuffle(keys)
    row = (keys // nc).astype(np.int32)
    col = (keys % nc).astype(np.int32)
    val = rng.standard_normal(len(keys)).astype(np.float32)
    return row, col, val


def dense_of(nr, nc, row, col, val):
    D = np.zeros((nr, nc))
    np.add.at(D, (row, col), val.astype(np.float64))
    return D


# ------------------------------------------------------------ DOK semantics

def test_dok_lookup_absent_is_zero_and_insert_adds(orc):
    # lookup of an absent key returns the additive identity; inserting an
    # existing key adds (semi-ring dictionary, Section 2.2)
    A = orc.Dok((4, 5), ([1, 1, 3], [2, 2, 0]), np.array([1.5, 2.0, -1.0], np.float32))
    v, pres = A.lookup([1, 3, 0, 2], [2, 0, 0, 4])
    assert np.array_equal(v, [3.5, -1.0, 0.0, 0.0])
    assert np.array_equal(pres, [True, True, False, False])
    assert A.nkeys == 2


# ----------------------------------------------------------------- formats

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_coo_to_csr_matches_lexsort_and_scipy(orc, seed):
    rng = np.random.default_rng(seed)
    nr, nc = 37, 53
    row, col, val = rand_coo(rng, nr, nc, 400, dups=60)
    rowptr, colind, v, first = orc.coo_to_csr(orc.Dok((nr, nc), (row, col), val))
    keys = row.astype(np.int64) * nc + col
    uk, idx = np.unique(keys, return_index=True)  # sorted keys, first occurrence
    assert np.array_equal(colind, (uk % nc).astype(np.int32))
    assert np.array_equal(first, idx)
    ref = sp.coo_matrix((val.astype(np.float64), (row, col)), shape=(nr, nc)).tocsr()
    ref.sort_indices()
    assert np.array_equal(rowptr, ref.indptr)
    assert np.array_equal(colind, ref.indices)
    np.testing.assert_allclose(v, ref.data, rtol=0, atol=1e-12)
    # lexicographic order with np.lexsort, stable: first occurrences first
    order = np.lexsort((np.arange(len(keys)), col, row))
    srt = keys[order]
    keep = np.ones(len(srt), bool)
    keep[1:] = srt[1:] != srt[:-1]
    assert np.array_equal(order[keep], first)


@pytest.mark.parametrize("seed", [0, 5])
def test_stable_sort_is_csc(orc, seed):
    rng = np.random.default_rng(seed)
    nr, nc = 41, 29
    row, col, val = rand_coo(rng, nr, nc, 300)
    csr = sp.coo_matrix((val, (row, col)), shape=(nr, nc)).tocsr()
    csr.sort_indices()
    colptr, skey, perm = orc.stable_sort_by_key(csr.indices, nc)
    assert np.array_equal(perm, np.argsort(csr.indices, kind="stable"))
    csc = csr.tocsc()
    csc.sort_indices()
    rows_of_csr = np.repeat(np.arange(nr), np.diff(csr.indptr))
    assert np.array_equal(colptr, csc.indptr)
    assert np.array_equal(rows_of_csr[perm], csc.indices)
    assert np.array_equal(csr.data[perm], csc.data)
    assert np.array_equal(skey, np.sort(csr.indices))


def test_stable_sort_ties_keep_position_order(orc):
    key = np.array([2, 0, 2, 1, 0, 2, 2], np.int32)
    segptr, skey, perm = orc.stable_sort_by_key(key, 4)
    assert perm.tolist() == [1, 4, 3, 0, 2, 5, 6]
    assert segptr.tolist() == [0, 2, 3, 7, 7]


# ---------------------------------------------------------------- products

@pytest.mark.parametrize("k", [1, 3, 8])
def test_spmm_and_transpose_match_dense(orc, k):
    rng = np.random.default_rng(10 + k)
    nr, nc = 23, 31
    row, col, val = rand_coo(rng, nr, nc, 150, dups=20)
    A = orc.Dok((nr, nc), (row, col), val)
    D = dense_of(nr, nc, row, col, val)
    B = rng.standard_normal((nc, k))
    G = rng.standard_normal((nr, k))
    Cm, Cmag = orc.spmm(A, B, k)
    np.testing.assert_allclose(Cm, D @ B, rtol=1e-12, atol=1e-12)
    absA = np.abs(D)
    np.testing.assert_allclose(Cmag, absA @ np.abs(B), rtol=1e-12, atol=1e-12)
    T, Tmag = orc.spmm_t(A, G, k, alpha=-0.5)
    np.testing.assert_allclose(T, -0.5 * D.T @ G, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Tmag, 0.5 * absA.T @ np.abs(G), rtol=1e-12, atol=1e-12)
    # selected rows / columns equal the full result's rows / columns
    rs = np.array([5, 0, 22], np.int32)
    Cs, _ = orc.spmm(A, B, k, rows=rs)
    np.testing.assert_array_equal(Cs, Cm[rs])
    cs = np.array([30, 2], np.int32)
    Ts, _ = orc.spmm_t(A, G, k, alpha=-0.5, cols=cs)
    np.testing.assert_array_equal(Ts, T[cs])


def test_spmm_t_ones_is_column_sums(orc):
    rng = np.random.default_rng(3)
    row, col, val = rand_coo(rng, 20, 30, 90)
    A = orc.Dok((20, 30), (row, col), val)
    ref = sp.coo_matrix((val.astype(np.float64), (row, col)), shape=(20, 30)).sum(axis=0).A1
    out, _ = orc.spmm_t(A, None, 1)
    np.testing.assert_allclose(out[:, 0], ref, rtol=1e-12, atol=1e-12)


def test_sddmm_is_masked_dense_product(orc):
    rng = np.random.default_rng(4)
    nr, nc, k = 17, 19, 6
    row, col, val = rand_coo(rng, nr, nc, 80)
    A = orc.Dok((nr, nc), (row, col), val)
    X, Y = rng.standard_normal((nr, k)), rng.standard_normal((nc, k))
    out, mag = orc.sddmm(A, X, Y, k, row, col, alpha=2.0)
    np.testing.assert_allclose(out, 2.0 * (X @ Y.T)[row, col], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(mag, 2.0 * (np.abs(X) @ np.abs(Y).T)[row, col], rtol=1e-12)
    # a key that is not stored is outside the one-hot seed: gradient 0
    absent = np.setdiff1d(np.arange(nr * nc), row.astype(np.int64) * nc + col)[:5]
    o2, m2 = orc.sddmm(A, X, Y, k, absent // nc, absent % nc)
    assert np.all(o2 == 0) and np.all(m2 == 0)


# ----------------------------------------------- losses: dense brute force

def _torch_masked(nr, nc, row, col, val):
    idx = torch.from_numpy(np.stack([row, col]).astype(np.int64))
    a = torch.tensor(val.astype(np.float64), requires_grad=True)
    A = torch.zeros(nr, nc, dtype=torch.float64).index_put((idx[0], idx[1]), a, accumulate=True)
    return a, A


def test_spmv_sum_loss_closed_forms(orc):
    # SMVM: f = sum_ij A(i,j) X(j); df/dX = A^T 1 (experiments section);
    # df/dA on the stored keys = X(j) (dot-product example, Section 5.2)
    rng = np.random.default_rng(7)
    nr, nc = 30, 40
    row, col, val = rand_coo(rng, nr, nc, 200)
    x = rng.standard_normal(nc).astype(np.float32)
    A = orc.Dok((nr, nc), (row, col), val)
    L, Lm = orc.loss_sum_spmv(A, x)
    S = sp.coo_matrix((val.astype(np.float64), (row, col)), shape=(nr, nc)).tocsr()
    assert L == pytest.approx(float((S @ x.astype(np.float64)).sum()), rel=1e-12)
    assert Lm == pytest.approx(float((abs(S) @ np.abs(x.astype(np.float64))).sum()), rel=1e-12)
    dA, _ = orc.sddmm(A, np.ones((nr, 1)), x.reshape(-1, 1), 1, row, col)
    assert np.array_equal(dA, x[col].astype(np.float64))
    dx, _ = orc.spmm_t(A, None, 1)
    np.testing.assert_allclose(dx[:, 0], np.asarray(S.sum(axis=0)).ravel(), rtol=1e-12, atol=1e-12)
    # autograd of the dense masked form
    a, Ad = _torch_masked(nr, nc, row, col, val)
    xt = torch.tensor(x.astype(np.float64), requires_grad=True)
    (Ad @ xt).sum().backward()
    np.testing.assert_allclose(dA, a.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dx[:, 0], xt.grad.numpy(), rtol=1e-12, atol=1e-12)


def frob_spmm_oracle(orc, A, row, col, B, k, seed=1.0):
    Cm, Cmag = orc.spmm(A, B, k)
    L, Lm = orc.loss_half_sq(Cm, Cmag)
    dA, _ = orc.sddmm(A, Cm, B, k, row, col, alpha=seed, Xmag=Cmag)
    dB, _ = orc.spmm_t(A, Cm, k, alpha=seed, Gmag=Cmag)
    return L, dA, dB


def test_frob_spmm_matches_autograd_and_fd(orc):
    rng = np.random.default_rng(11)
    nr, nc, k = 12, 9, 5
    row, col, val = rand_coo(rng, nr, nc, 40)
    B = rng.standard_normal((nc, k))
    A = orc.Dok((nr, nc), (row, col), val)
    L, dA, dB = frob_spmm_oracle(orc, A, row, col, B, k)
    a, Ad = _torch_masked(nr, nc, row, col, val)
    Bt = torch.tensor(B, requires_grad=True)
    Lt = 0.5 * ((Ad @ Bt) ** 2).sum()
    Lt.backward()
    assert L == pytest.approx(Lt.item(), rel=1e-12)
    np.testing.assert_allclose(dA, a.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dB, Bt.grad.numpy(), rtol=1e-10, atol=1e-12)
    # central differences are exact for a quadratic along each coordinate
    h = 1e-3
    for p in [0, 7, 39]:
        vp, vm = val.astype(np.float64).copy(), val.astype(np.float64).copy()
        vp[p] += h
        vm[p] -= h
        Dp, Dm = dense_of(nr, nc, row, col, vp), dense_of(nr, nc, row, col, vm)
        fd = (0.5 * ((Dp @ B) ** 2).sum() - 0.5 * ((Dm @ B) ** 2).sum()) / (2 * h)
        assert dA[p] == pytest.approx(fd, rel=1e-7, abs=1e-9)


def test_bilinear_matches_autograd(orc):
    rng = np.random.default_rng(12)
    n, k = 14, 7
    row, col, val = rand_coo(rng, n, n, 60)
    val = np.abs(val)
    H, G = rng.standard_normal((n, k)), rng.standard_normal((n, k))
    A = orc.Dok((n, n), (row, col), val)
    L, Lm = orc.loss_bilinear(A, G, H, k)
    dA, _ = orc.sddmm(A, G, H, k, row, col)
    dH, _ = orc.spmm_t(A, G, k)
    a, Ad = _torch_masked(n, n, row, col, val)
    Ht = torch.tensor(H, requires_grad=True)
    Lt = ((Ad @ Ht) * torch.tensor(G)).sum()
    Lt.backward()
    assert L == pytest.approx(Lt.item(), rel=1e-12)
    np.testing.assert_allclose(dA, a.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dH, Ht.grad.numpy(), rtol=1e-10, atol=1e-12)
    # the loss is the pattern-weighted sum of the sparse gradient
    assert L == pytest.approx(float(np.dot(val.astype(np.float64), dA)), rel=1e-12)


def test_mf_matches_autograd_and_special_cases(orc):
    rng = np.random.default_rng(13)
    nr, nc, k = 15, 11, 4
    row, col, _ = rand_coo(rng, nr, nc, 70)
    val = (1 + 4 * rng.random(70)).astype(np.float32)
    U, V = 0.3 * rng.standard_normal((nr, k)), 0.3 * rng.standard_normal((nc, k))
    A = orc.Dok((nr, nc), (row, col), val)
    L, _ = orc.mf_loss(A, U, V, k)
    r, _ = orc.mf_resid(A, U, V, k, row, col)
    dU, _ = orc.mf_grad(A, U, V, k, 0)
    dV, _ = orc.mf_grad(A, U, V, k, 1)
    Ut = torch.tensor(U, requires_grad=True)
    Vt = torch.tensor(V, requires_grad=True)
    rt = torch.tensor(val.astype(np.float64)) - (Ut[row] * Vt[col]).sum(1)
    Lt = (rt ** 2).sum()
    Lt.backward()
    assert L == pytest.approx(Lt.item(), rel=1e-12)
    np.testing.assert_allclose(r, rt.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dU, Ut.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dV, Vt.grad.numpy(), rtol=1e-10, atol=1e-12)
    # V = 0: r = A, dU = 0 exactly, dV = -2 A^T U (scipy)
    V0 = np.zeros_like(V)
    dU0, _ = orc.mf_grad(A, U, V0, k, 0)
    dV0, _ = orc.mf_grad(A, U, V0, k, 1)
    S = sp.coo_matrix((val.astype(np.float64), (row, col)), shape=(nr, nc)).tocsr()
    assert np.all(dU0 == 0)
    np.testing.assert_allclose(dV0, -2 * (S.T @ U), rtol=1e-12, atol=1e-12)
    L0, _ = orc.mf_loss(A, np.zeros_like(U), V0, k)
    assert L0 == pytest.approx(float((val.astype(np.float64) ** 2).sum()), rel=1e-12)


def test_cp_matches_dense_einsum_and_special_cases(orc):
    rng = np.random.default_rng(14)
    d, R, nnz = 9, 5, 150
    keys = rng.choice(d ** 3, size=nnz, replace=False)
    i, j, l = keys // (d * d), (keys // d) % d, keys % d
    x = rng.standard_normal(nnz).astype(np.float32)
    F = [0.5 * rng.standard_normal((d, R)) for _ in range(3)]
    X = orc.Dok((d, d, d), (i, j, l), x)
    M = np.zeros((d, d, d))
    M[i, j, l] = 1
    Xd = np.zeros((d, d, d))
    Xd[i, j, l] = x
    m = np.einsum("ir,jr,kr->ijk", *F)
    Rd = (Xd - m) * M
    L, _ = orc.cp_loss(X, *F, R)
    assert L == pytest.approx(0.5 * (Rd ** 2).sum(), rel=1e-12)
    res, _ = orc.cp_resid(X, *F, R, i, j, l)
    np.testing.assert_allclose(res, Rd[i, j, l], rtol=1e-12, atol=1e-12)
    refs = [-np.einsum("ijk,jr,kr->ir", Rd, F[1], F[2]),
            -np.einsum("ijk,ir,kr->jr", Rd, F[0], F[2]),
            -np.einsum("ijk,ir,jr->kr", Rd, F[0], F[1])]
    for mode in range(3):
        g, _ = orc.cp_grad(X, *F, R, mode)
        np.testing.assert_allclose(g, refs[mode], rtol=1e-10, atol=1e-12)
    # all factors 1: m = R everywhere, dF1(i,:) = -(sum of the slice's residual)
    ones = [np.ones((d, R))] * 3
    g1, _ = orc.cp_grad(X, *ones, R, 0)
    slice_sum = np.bincount(i, weights=x.astype(np.float64) - R, minlength=d)
    np.testing.assert_allclose(g1, -np.repeat(slice_sum[:, None], R, 1), rtol=1e-12, atol=1e-12)


def test_cp_finite_differences(orc):
    rng = np.random.default_rng(15)
    d, R, nnz = 6, 3, 60
    keys = rng.choice(d ** 3, size=nnz, replace=False)
    i, j, l = keys // (d * d), (keys // d) % d, keys % d
    x = rng.standard_normal(nnz).astype(np.float32)
    F = [0.5 * rng.standard_normal((d, R)) for _ in range(3)]
    X = orc.Dok((d, d, d), (i, j, l), x)
    g, _ = orc.cp_grad(X, *F, R, 1)
    h = 1e-4
    for (a, b) in [(0, 0), (3, 2), (5, 1)]:
        Fp = [f.copy() for f in F]
        Fm = [f.copy() for f in F]
        Fp[1][a, b] += h
        Fm[1][a, b] -= h
        fd = (orc.cp_loss(X, *Fp, R)[0] - orc.cp_loss(X, *Fm, R)[0]) / (2 * h)
        assert g[a, b] == pytest.approx(fd, rel=1e-6, abs=1e-9)


def test_ttv_and_vjp_match_autograd(orc):
    rng = np.random.default_rng(16)
    d, nnz = 7, 80
    keys = rng.choice(d ** 3, size=nnz, replace=False)
    i, j, l = keys // (d * d), (keys // d) % d, keys % d
    x = rng.standard_normal(nnz).astype(np.float32)
    v = rng.standard_normal(d)
    X = orc.Dok((d, d, d), (i, j, l), x)
    yi, yj, y, _ = orc.ttv(X, v)
    proj = np.unique(i.astype(np.int64) * d + j)
    assert np.array_equal(yi.astype(np.int64) * d + yj, proj)
    xt = torch.tensor(x.astype(np.float64), requires_grad=True)
    vt = torch.tensor(v, requires_grad=True)
    Yd = torch.zeros(d, d, dtype=torch.float64).index_put(
        (torch.from_numpy(i), torch.from_numpy(j)), xt * vt[torch.from_numpy(l)], accumulate=True)
    np.testing.assert_allclose(y, Yd.detach().numpy()[yi, yj], rtol=1e-12, atol=1e-12)
    gy = rng.standard_normal(len(yi)).astype(np.float32)
    gY = orc.Dok((d, d), (yi, yj), gy)
    Gd = torch.zeros(d, d, dtype=torch.float64)
    Gd[yi, yj] = torch.tensor(gy.astype(np.float64))
    (Yd * Gd).sum().backward()
    dX, _, dv, _ = orc.ttv_vjp(X, v, gY, i, j, l)
    np.testing.assert_allclose(dX, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dv, vt.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("R", [1, 5])
def test_ttm_and_vjp_match_autograd(orc, R):
    # Y(i, j, :) = sum_l X(i, j, l) U(l, :) on the projected keys: autograd of
    # the dense einsum, with the upstream placed on those keys
    rng = np.random.default_rng(17 + R)
    d0, d1, d2, nnz = 6, 5, 7, 90
    keys = rng.choice(d0 * d1 * d2, size=nnz, replace=False)
    i, j, l = keys // (d1 * d2), (keys // d2) % d1, keys % d2
    x = rng.standard_normal(nnz).astype(np.float32)
    U = rng.standard_normal((d2, R))
    X = orc.Dok((d0, d1, d2), (i, j, l), x)
    yi, yj, y, ym = orc.ttm(X, U, R)
    proj = np.unique(i.astype(np.int64) * d1 + j)
    assert np.array_equal(yi.astype(np.int64) * d1 + yj, proj)
    Xd = torch.zeros(d0, d1, d2, dtype=torch.float64)
    Xd[i, j, l] = torch.tensor(x.astype(np.float64))
    Xd.requires_grad_(True)
    Ut = torch.tensor(U, requires_grad=True)
    Yd = torch.einsum("ijl,lr->ijr", Xd, Ut)
    np.testing.assert_allclose(y, Yd.detach().numpy()[yi, yj], rtol=1e-12, atol=1e-12)
    assert np.all(ym >= np.abs(y) - 1e-12)
    gy = rng.standard_normal((len(yi), R))
    Gd = torch.zeros(d0, d1, R, dtype=torch.float64)
    Gd[yi, yj] = torch.tensor(gy)
    (Yd * Gd).sum().backward()
    dX, _, dU, _ = orc.ttm_vjp(X, U, R, gy, i, j, l)
    np.testing.assert_allclose(dX, Xd.grad.numpy()[i, j, l], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dU, Ut.grad.numpy(), rtol=1e-12, atol=1e-12)
    # R = 1 is TTV
    if R == 1:
        _, _, yv, _ = orc.ttv(X, U[:, 0])
        np.testing.assert_allclose(y[:, 0], yv, rtol=1e-12, atol=1e-14)


def test_mag_bounds_value_and_equals_it_for_nonnegative_terms(orc):
    rng = np.random.default_rng(17)
    row, col, val = rand_coo(rng, 25, 25, 100)
    A = orc.Dok((25, 25), (row, col), val)
    B = rng.standard_normal((25, 4))
    Cm, Cmag = orc.spmm(A, B, 4)
    assert np.all(Cmag >= np.abs(Cm) - 1e-12)
    Ap = orc.Dok((25, 25), (row, col), np.abs(val))
    Cp, Cpmag = orc.spmm(Ap, np.abs(B), 4)
    np.testing.assert_allclose(Cp, Cpmag, rtol=1e-14)


# -------------------------------------------------- the paper's examples

def _load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_golden_dot_product_gradient(orc):
    # Example 1: the gradient of V1 . V2 w.r.t. V1 is V2 on V2's stored keys
    g = _load_golden("example1_dot_gradient.json")
    V2 = {int(k): v for k, v in g["V2"].items()}
    n = g["length"]
    keys = np.array(sorted(V2), np.int32)
    vals = np.array([V2[k] for k in keys], np.float32)
    # V1 . V2 as a one-row SMVM: A = V2 as a 1 x n row, X = V1 dense
    A = orc.Dok((1, n), (np.zeros_like(keys), keys), vals)
    grad, _ = orc.spmm_t(A, None, 1)  # d/dV1 of sum_i V2(i) V1(i)
    expect = np.zeros(n)
    for k, v in g["expected_gradient_wrt_V1"].items():
        expect[int(k)] = v
    assert np.array_equal(grad[:, 0], expect)


def test_golden_trace_gradient(orc):
    # Example 3: d trace(M)/dM is 1 on the stored diagonal keys, 0 elsewhere
    g = _load_golden("example3_trace_gradient.json")
    n = g["n"]
    row = np.array([e[0] for e in g["M_keys"]], np.int32)
    col = np.array([e[1] for e in g["M_keys"]], np.int32)
    val = np.array(g["M_values"], np.float32)
    M = orc.Dok((n, n), (row, col), val)
    # trace(M) = sum over stored (i, j) of [i == j] * M(i, j): SDDMM with X = Y = I
    eye = np.eye(n)
    grad, _ = orc.sddmm(M, eye, eye, n, row, col)
    assert grad.tolist() == g["expected_gradient_on_keys"]


# ------------------------------------------------------- BATAX Jacobian

def _batax_case(rng, nr=9, nc=7, nnz=24):
    row, col, val = rand_coo(rng, nr, nc, nnz)
    val[3] = 0.0  # a stored zero keeps its keys
    return row, col, val


def test_batax_jacobian_matches_autograd_and_dense(orc):
    """J of f(x) = beta A^T (A x) by PyTorch fp64 autograd on the dense A;
    keys = pairs of stored keys that share a row (structural, stored zeros
    included); values = beta A^T A, 0 off the keys."""
    rng = np.random.default_rng(21)
    nr, nc, beta = 9, 7, 1.75
    row, col, val = _batax_case(rng, nr, nc)
    D = orc.Dok((nr, nc), (row, col), val)
    rowptr, colind, jv, jm = orc.batax_jacobian(D, beta)
    A = torch.tensor(dense_of(nr, nc, row, col, val))
    x0 = torch.tensor(rng.standard_normal(nc))
    Jt = torch.autograd.functional.jacobian(lambda x: beta * (A.T @ (A @ x)), x0).numpy()
    J = np.zeros((nc, nc))
    rows = np.repeat(np.arange(nc), np.diff(rowptr))
    J[rows, colind] = jv
    assert np.allclose(J, Jt, rtol=0, atol=1e-12)
    S = dense_of(nr, nc, row, col, np.ones_like(val)) > 0
    keys = (S.T.astype(int) @ S.astype(int)) > 0
    got = np.zeros((nc, nc), bool)
    got[rows, colind] = True
    assert np.array_equal(got, keys)
    assert np.all(jm >= np.abs(jv) - 1e-15)
    # sorted CSR emission, symmetric result
    for r in range(nc):
        assert np.all(np.diff(colind[rowptr[r]:rowptr[r + 1]]) > 0)
    assert np.allclose(J, J.T, atol=0)


def test_batax_jacobian_matrix_free_identity(orc):
    """J x = beta A^T (A x) with scipy products on a larger random matrix."""
    rng = np.random.default_rng(22)
    nr, nc, beta = 300, 200, -0.5
    row, col, val = rand_coo(rng, nr, nc, 2500)
    D = orc.Dok((nr, nc), (row, col), val)
    rowptr, colind, jv, _ = orc.batax_jacobian(D, beta)
    J = sp.csr_matrix((jv, colind, rowptr), shape=(nc, nc))
    A = sp.csr_matrix((val.astype(np.float64), (row, col)), shape=(nr, nc))
    x = rng.standard_normal(nc)
    assert np.allclose(J @ x, beta * (A.T @ (A @ x)), rtol=1e-12, atol=1e-12)


def test_batax_jacobian_row_outer_products(orc):
    """A single stored row r gives exactly beta r r^T on r's keys."""
    D = orc.Dok((1, 5), (np.array([0, 0, 0], np.int32), np.array([0, 2, 4], np.int32)),
                np.array([1.0, -2.0, 3.0], np.float32))
    rowptr, colind, jv, jm = orc.batax_jacobian(D, 2.0)
    r = np.array([1.0, 0.0, -2.0, 0.0, 3.0])
    J = np.zeros((5, 5))
    J[np.repeat(np.arange(5), np.diff(rowptr)), colind] = jv
    assert np.array_equal(J, 2.0 * np.outer(r, r))
    assert len(colind) == 9 and np.array_equal(jm, np.abs(jv))


# ------------------------------------------------- forward-mode tangent

def test_spmm_jvp_matches_torch_forward_mode(orc):
    """dC of C = A B by PyTorch's forward-mode jvp on the dense operands, the
    tangent of A masked to A's keys; C equals the dense product."""
    from torch.func import jvp
    rng = np.random.default_rng(31)
    nr, nc, k = 8, 6, 5
    row, col, val = rand_coo(rng, nr, nc, 20)
    dval = rng.standard_normal(len(val)).astype(np.float32)
    A = orc.Dok((nr, nc), (row, col), val)
    dA = orc.Dok((nr, nc), (row, col), dval)
    B = rng.standard_normal((nc, k)).astype(np.float32)
    dB = rng.standard_normal((nc, k)).astype(np.float32)
    C, Cm, dC, dCm = orc.spmm_jvp(A, dA, B, dB, k)
    Ad = torch.tensor(dense_of(nr, nc, row, col, val))
    dAd = torch.tensor(dense_of(nr, nc, row, col, dval))
    Ct, dCt = jvp(lambda a, b: a @ b, (Ad, torch.tensor(B, dtype=torch.float64)),
                  (dAd, torch.tensor(dB, dtype=torch.float64)))
    assert np.allclose(C, Ct.numpy(), rtol=0, atol=1e-12)
    assert np.allclose(dC, dCt.numpy(), rtol=0, atol=1e-12)
    assert np.all(Cm >= np.abs(C) - 1e-15) and np.all(dCm >= np.abs(dC) - 1e-15)


def test_spmm_jvp_linear_in_the_tangent(orc):
    """Zero tangents give dC = 0; dB alone gives A dB; dA alone gives dA B."""
    rng = np.random.default_rng(32)
    nr, nc, k = 30, 20, 3
    row, col, val = rand_coo(rng, nr, nc, 90)
    A = orc.Dok((nr, nc), (row, col), val)
    zero = orc.Dok((nr, nc), (row, col), np.zeros_like(val))
    B = rng.standard_normal((nc, k)).astype(np.float32)
    dB = rng.standard_normal((nc, k)).astype(np.float32)
    _, _, d0, m0 = orc.spmm_jvp(A, zero, B, np.zeros_like(B), k)
    assert np.array_equal(d0, np.zeros_like(d0)) and np.array_equal(m0, np.zeros_like(m0))
    _, _, d1, _ = orc.spmm_jvp(A, zero, B, dB, k)
    As = sp.csr_matrix((val.astype(np.float64), (row, col)), shape=(nr, nc))
    assert np.allclose(d1, As @ dB.astype(np.float64), rtol=1e-12, atol=1e-12)
    dval = rng.standard_normal(len(val)).astype(np.float32)
    _, _, d2, _ = orc.spmm_jvp(A, orc.Dok((nr, nc), (row, col), dval), B, np.zeros_like(B), k)
    dAs = sp.csr_matrix((dval.astype(np.float64), (row, col)), shape=(nr, nc))
    assert np.allclose(d2, dAs @ B.astype(np.float64), rtol=1e-12, atol=1e-12)


# ----------------------------------------------------- order-N CP gradient

@pytest.mark.parametrize("dims", [(4, 5, 3, 6), (3, 4, 3, 2, 5)])
def test_cpn_matches_autograd(orc, dims):
    """Order-4 and order-5 CP: loss, residual and every factor gradient by
    PyTorch fp64 autograd of 1/2 sum over the stored keys of (x - m)^2 with
    m from a dense einsum."""
    rng = np.random.default_rng(sum(dims))
    N, R = len(dims), 3
    size = int(np.prod(dims))
    keys = rng.choice(size, size=size // 3, replace=False)
    coords = np.unravel_index(keys, dims)
    coords = [c.astype(np.int32) for c in coords]
    val = rng.standard_normal(len(keys)).astype(np.float32)
    F = [rng.standard_normal((d, R)).astype(np.float32) for d in dims]
    X = orc.Dok(dims, coords, val)
    L, Lm = orc.cpn_loss(X, F, R)
    Ft = [torch.tensor(f, dtype=torch.float64, requires_grad=True) for f in F]
    letters = "abcdef"[:N]
    m = torch.einsum(",".join(f"{l}r" for l in letters) + "->" + letters, *Ft)
    x = torch.tensor(val, dtype=torch.float64)
    res = x - m[tuple(torch.tensor(c, dtype=torch.long) for c in coords)]
    Lt = 0.5 * (res ** 2).sum()
    Lt.backward()
    assert abs(L - Lt.item()) <= 1e-12 * max(1.0, Lm)
    r, rm = orc.cpn_resid(X, F, R, coords)
    assert np.allclose(r, res.detach().numpy(), rtol=0, atol=1e-12)
    for n in range(N):
        g, gm = orc.cpn_grad(X, F, R, n)
        assert np.allclose(g, Ft[n].grad.numpy(), rtol=0, atol=1e-12)
        assert np.all(gm >= np.abs(g) - 1e-12)
    # a selection gives the same rows
    sel = np.array([dims[0] - 1, 0], np.int32)
    g0, _ = orc.cpn_grad(X, F, R, 0, sel=sel)
    assert np.array_equal(g0, orc.cpn_grad(X, F, R, 0)[0][sel])


def test_cpn_order3_equals_the_order3_oracle(orc):
    rng = np.random.default_rng(41)
    dims, R = (7, 6, 5), 4
    keys = rng.choice(210, size=60, replace=False)
    i, j, l = (c.astype(np.int32) for c in np.unravel_index(keys, dims))
    val = rng.standard_normal(60).astype(np.float32)
    F = [rng.standard_normal((d, R)).astype(np.float32) for d in dims]
    X3 = orc.Dok(dims, (i, j, l), val)
    assert np.isclose(orc.cpn_loss(X3, F, R)[0], orc.cp_loss(X3, *F, R)[0], rtol=1e-14)
    for n in range(3):
        assert np.allclose(orc.cpn_grad(X3, F, R, n)[0], orc.cp_grad(X3, *F, R, n)[0],
                           rtol=1e-13, atol=1e-13)


# ----------------------------------------------------- threads by owner

def test_owner_parallel_loops_are_bitwise_single_threaded(orc):
    """The gradient loops split their outputs by owner across threads; each
    output keeps its single-threaded order of terms, so any thread count
    gives bitwise the single-threaded result."""
    rng = np.random.default_rng(51)
    nr, nc, k = 60, 45, 6
    row, col, val = rand_coo(rng, nr, nc, 900)
    A = orc.Dok((nr, nc), (row, col), val)
    B, G = rng.standard_normal((nc, k)), rng.standard_normal((nr, k))
    U, V = rng.standard_normal((nr, k)), rng.standard_normal((nc, k))
    d, R = 12, 4
    keys = rng.choice(d ** 3, size=500, replace=False)
    i, j, l = (c.astype(np.int32) for c in np.unravel_index(keys, (d, d, d)))
    x = rng.standard_normal(500).astype(np.float32)
    X = orc.Dok((d, d, d), (i, j, l), x)
    F = [rng.standard_normal((d, R)) for _ in range(3)]

    def run():
        out = [orc.spmm(A, B, k), orc.spmm_t(A, G, k, alpha=0.5),
               orc.sddmm(A, G, B, k, row, col), orc.mf_grad(A, U, V, k, 0),
               orc.mf_grad(A, U, V, k, 1), orc.loss_bilinear(A, G, B, k)]
        out += [orc.cp_grad(X, *F, R, m) for m in range(3)]
        out += [orc.cpn_grad(X, F, R, m) for m in range(3)]
        return out

    try:
        orc.set_threads(1)
        one = run()
        orc.set_threads(5)
        many = run()
    finally:
        orc.set_threads(1)
    for a, b in zip(one, many):
        for x1, x2 in zip(a, b):
            assert np.array_equal(np.asarray(x1), np.asarray(x2))


# ------------------------------------------- mode products of any order

@pytest.mark.parametrize("dims", [(5, 4, 6), (3, 4, 2, 5), (3, 2, 4, 2, 3)])
def test_ttmn_matches_autograd_in_every_mode(orc, dims):
    """Y = X x_n U on the projected keys and its VJP, every mode of orders
    3 to 5: PyTorch fp64 autograd of the dense einsum, the upstream placed on
    the projected keys; the keys are the distinct projections in
    lexicographic order."""
    N, R = len(dims), 3
    rng = np.random.default_rng(sum(dims) + N)
    size = int(np.prod(dims))
    keys = rng.choice(size, size=size // 3, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(keys, dims)]
    x = rng.standard_normal(len(keys)).astype(np.float32)
    X = orc.Dok(dims, coords, x)
    letters = "abcdef"[:N]
    for n in range(N):
        U = rng.standard_normal((dims[n], R))
        yk, y, ym = orc.ttmn(X, n, U, R)
        others = [m for m in range(N) if m != n]
        proj = np.unique(np.ravel_multi_index([coords[m] for m in others],
                                              [dims[m] for m in others]))
        want = np.unravel_index(proj, [dims[m] for m in others])
        for o in range(N - 1):
            assert np.array_equal(yk[o], want[o])
        Xd = torch.zeros(dims, dtype=torch.float64)
        Xd[tuple(torch.from_numpy(c.astype(np.int64)) for c in coords)] = \
            torch.tensor(x.astype(np.float64))
        Xd.requires_grad_(True)
        Ut = torch.tensor(U, requires_grad=True)
        out = "".join(letters[m] for m in others) + "r"
        Yd = torch.einsum(f"{letters},{letters[n]}r->{out}", Xd, Ut)
        idx = tuple(torch.from_numpy(k.astype(np.int64)) for k in yk)
        np.testing.assert_allclose(y, Yd.detach().numpy()[idx], rtol=1e-12, atol=1e-12)
        assert np.all(ym >= np.abs(y) - 1e-12)
        gy = rng.standard_normal((len(yk[0]), R))
        Gd = torch.zeros(Yd.shape, dtype=torch.float64)
        Gd[idx] = torch.tensor(gy)
        (Yd * Gd).sum().backward()
        dX, _, dU, _ = orc.ttmn_vjp(X, n, U, R, gy, coords)
        cidx = tuple(torch.from_numpy(c.astype(np.int64)) for c in coords)
        np.testing.assert_allclose(dX, Xd.grad.numpy()[tuple(c.numpy() for c in cidx)],
                                   rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(dU, Ut.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_ttmn_last_mode_of_order3_is_ttm_and_ttv(orc):
    rng = np.random.default_rng(77)
    dims, R = (6, 5, 7), 4
    keys = rng.choice(210, size=90, replace=False)
    i, j, l = (c.astype(np.int32) for c in np.unravel_index(keys, dims))
    x = rng.standard_normal(90).astype(np.float32)
    X = orc.Dok(dims, (i, j, l), x)
    U = rng.standard_normal((dims[2], R))
    yk, y, ym = orc.ttmn(X, 2, U, R)
    yi, yj, y3, ym3 = orc.ttm(X, U, R)
    assert np.array_equal(yk[0], yi) and np.array_equal(yk[1], yj)
    assert np.array_equal(y, y3) and np.array_equal(ym, ym3)
    _, _, yv, _ = orc.ttv(X, U[:, 0])
    np.testing.assert_allclose(orc.ttmn(X, 2, U[:, :1], 1)[1][:, 0], yv, rtol=1e-14, atol=1e-15)
