"""Pins for the oracle's magnitude companions ("mag").

Every floating-point output of the oracle comes with mag, the same
expression evaluated on the absolute values of its terms (a subtraction
counted as an addition).  The parity bar of every GPU comparison is
|got - ref| <= 1e-4 * mag, so a mag that is too large (a stray factor, a
product where a sum belongs) would loosen parity silently.  Each test below
recomputes a mag from its definition in a different form than the oracle's
dictionary loops -- dense numpy arrays with a 0/1 mask of the stored keys,
matrix products and einsums over |terms| -- on inputs of at most a few
hundred entries, and checks two further properties that do not depend on
that recomputation:
  * mag >= |value| for every output (the triangle inequality), and
  * mag == |value| exactly (up to rounding) when every term is
    non-negative and the expression has no subtraction.
"""
import numpy as np
import pytest


def _keys(rng, shape, n):
    size = int(np.prod(shape))
    k = rng.choice(size, size=n, replace=False)
    return [c.astype(np.int32) for c in np.unravel_index(k, shape)]


def _mask(shape, coords):
    M = np.zeros(shape)
    M[tuple(coords)] = 1.0
    return M


def _dense(shape, coords, val):
    D = np.zeros(shape)
    D[tuple(coords)] = val.astype(np.float64)
    return D


def _close(a, b):
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-300)


def _bounds(value, mag):
    assert np.all(np.asarray(mag) >= np.abs(value) * (1 - 1e-12))


# ---------------------------------------------------------- loss_half_sq

def test_loss_half_sq_mag(orc):
    rng = np.random.default_rng(101)
    C = rng.standard_normal((6, 5))
    Cm = np.abs(C) + rng.random((6, 5))  # a companion mag larger than |C|
    L, M = orc.loss_half_sq(C, Cm)
    assert M == pytest.approx(0.5 * np.sum(Cm * Cm), rel=1e-14)
    assert L == pytest.approx(0.5 * np.sum(C * C), rel=1e-14)
    _bounds(L, M)
    # non-negative terms: mag == value
    L2, M2 = orc.loss_half_sq(np.abs(C), np.abs(C))
    assert M2 == pytest.approx(L2, rel=1e-15)


# ------------------------------------------------------- loss_sum_spmv

def test_loss_sum_spmv_mag(orc):
    rng = np.random.default_rng(102)
    nr, nc = 8, 7
    row, col = _keys(rng, (nr, nc), 25)
    val = rng.standard_normal(25).astype(np.float32)
    x = rng.standard_normal(nc).astype(np.float32)
    A = orc.Dok((nr, nc), (row, col), val)
    L, M = orc.loss_sum_spmv(A, x)
    Ad = _dense((nr, nc), (row, col), val)
    assert M == pytest.approx(float(np.sum(np.abs(Ad) @ np.abs(x.astype(np.float64)))), rel=1e-13)
    _bounds(L, M)
    Ap = orc.Dok((nr, nc), (row, col), np.abs(val))
    L2, M2 = orc.loss_sum_spmv(Ap, np.abs(x))
    assert M2 == pytest.approx(L2, rel=1e-14)


# -------------------------------------------------------- loss_bilinear

def test_loss_bilinear_mag(orc):
    rng = np.random.default_rng(103)
    n, k = 8, 5
    row, col = _keys(rng, (n, n), 30)
    val = rng.standard_normal(30).astype(np.float32)
    G, H = rng.standard_normal((n, k)), rng.standard_normal((n, k))
    A = orc.Dok((n, n), (row, col), val)
    L, M = orc.loss_bilinear(A, G, H, k)
    Ad = _dense((n, n), (row, col), val)
    # sum over the keys of |a| * sum_f |G_if H_jf|
    assert M == pytest.approx(float(np.sum(np.abs(Ad) * (np.abs(G) @ np.abs(H).T))), rel=1e-13)
    _bounds(L, M)
    Ap = orc.Dok((n, n), (row, col), np.abs(val))
    L2, M2 = orc.loss_bilinear(Ap, np.abs(G), np.abs(H), k)
    assert M2 == pytest.approx(L2, rel=1e-14)


# ------------------------------------------------------- factorisation

def _mf_case(rng, nr=8, nc=7, k=4, n=28):
    row, col = _keys(rng, (nr, nc), n)
    val = (1 + 4 * rng.random(n)).astype(np.float32)
    U, V = rng.standard_normal((nr, k)), rng.standard_normal((nc, k))
    return row, col, val, U, V


def test_mf_mags(orc):
    rng = np.random.default_rng(104)
    nr, nc, k = 8, 7, 4
    row, col, val, U, V = _mf_case(rng, nr, nc, k)
    A = orc.Dok((nr, nc), (row, col), val)
    Msk = _mask((nr, nc), (row, col))
    Ad = _dense((nr, nc), (row, col), val)
    # residual r = a - <U_i, V_j>: mag = |a| + sum_c |U_ic V_jc|
    Rmag = (np.abs(Ad) + np.abs(U) @ np.abs(V).T) * Msk
    r, rm = orc.mf_resid(A, U, V, k, row, col)
    _close(rm, Rmag[row, col])
    _bounds(r, rm)
    # loss sum r^2: mag = sum rmag^2
    L, M = orc.mf_loss(A, U, V, k)
    assert M == pytest.approx(float(np.sum(Rmag ** 2)), rel=1e-13)
    _bounds(L, M)
    # dU = -2 sum_j r V_j: mag = 2 sum_j rmag |V_j|;  dV likewise with U
    dU, dUm = orc.mf_grad(A, U, V, k, 0)
    dV, dVm = orc.mf_grad(A, U, V, k, 1)
    _close(dUm, 2.0 * Rmag @ np.abs(V))
    _close(dVm, 2.0 * Rmag.T @ np.abs(U))
    _bounds(dU, dUm)
    _bounds(dV, dVm)
    # no subtraction left when U = 0 (r = a > 0): mag == value for the loss
    # and the residual; with V >= 0 as well, dU's terms all have one sign
    U0 = np.zeros_like(U)
    L0, M0 = orc.mf_loss(A, U0, V, k)
    assert M0 == pytest.approx(L0, rel=1e-14)
    r0, rm0 = orc.mf_resid(A, U0, V, k, row, col)
    _close(rm0, np.abs(r0))
    g0, gm0 = orc.mf_grad(A, U0, np.abs(V), k, 0)
    _close(gm0, np.abs(g0))


# ----------------------------------------------------------------- CP

def _cp_case(rng, dims=(6, 5, 7), R=3, n=50):
    c = _keys(rng, dims, n)
    x = rng.standard_normal(n).astype(np.float32)
    F = [rng.standard_normal((d, R)) for d in dims]
    return c, x, F


def test_cp_mags(orc):
    rng = np.random.default_rng(105)
    dims, R = (6, 5, 7), 3
    (i, j, l), x, F = _cp_case(rng, dims, R)
    X = orc.Dok(dims, (i, j, l), x)
    Msk = _mask(dims, (i, j, l))
    Xd = _dense(dims, (i, j, l), x)
    aF = [np.abs(f) for f in F]
    Rmag = (np.abs(Xd) + np.einsum("ir,jr,kr->ijk", *aF)) * Msk
    res, rm = orc.cp_resid(X, *F, R, i, j, l)
    _close(rm, Rmag[i, j, l])
    _bounds(res, rm)
    L, M = orc.cp_loss(X, *F, R)
    assert M == pytest.approx(0.5 * float(np.sum(Rmag ** 2)), rel=1e-13)
    _bounds(L, M)
    refs = [np.einsum("ijk,jr,kr->ir", Rmag, aF[1], aF[2]),
            np.einsum("ijk,ir,kr->jr", Rmag, aF[0], aF[2]),
            np.einsum("ijk,ir,jr->kr", Rmag, aF[0], aF[1])]
    for mode in range(3):
        g, gm = orc.cp_grad(X, *F, R, mode)
        _close(gm, refs[mode])
        _bounds(g, gm)
    # zero factors: R = x, no subtraction; with x >= 0 and F >= 0 elsewhere
    # the gradient's terms have one sign
    Z = [np.zeros_like(f) for f in F]
    L0, M0 = orc.cp_loss(X, *Z, R)
    assert M0 == pytest.approx(L0, rel=1e-14)
    Xp = orc.Dok(dims, (i, j, l), np.abs(x))
    g0, gm0 = orc.cp_grad(Xp, Z[0], aF[1], aF[2], R, 0)
    _close(gm0, np.abs(g0))


@pytest.mark.parametrize("dims", [(4, 3, 5, 3), (3, 4, 2, 3, 4)])
def test_cpn_mags(orc, dims):
    rng = np.random.default_rng(106 + len(dims))
    N, R = len(dims), 3
    c = _keys(rng, dims, int(np.prod(dims)) // 3)
    x = rng.standard_normal(len(c[0])).astype(np.float32)
    F = [rng.standard_normal((d, R)) for d in dims]
    X = orc.Dok(dims, c, x)
    Msk = _mask(dims, c)
    Xd = _dense(dims, c, x)
    aF = [np.abs(f) for f in F]
    letters = "abcdef"[:N]
    model_abs = np.einsum(",".join(f"{a}r" for a in letters) + "->" + letters, *aF)
    Rmag = (np.abs(Xd) + model_abs) * Msk
    r, rm = orc.cpn_resid(X, F, R, c)
    _close(rm, Rmag[tuple(c)])
    _bounds(r, rm)
    L, M = orc.cpn_loss(X, F, R)
    assert M == pytest.approx(0.5 * float(np.sum(Rmag ** 2)), rel=1e-13)
    _bounds(L, M)
    for n in range(N):
        others = [m for m in range(N) if m != n]
        spec = letters + "," + ",".join(f"{letters[m]}r" for m in others) + f"->{letters[n]}r"
        g, gm = orc.cpn_grad(X, F, R, n)
        _close(gm, np.einsum(spec, Rmag, *[aF[m] for m in others]))
        _bounds(g, gm)
    Z = [np.zeros_like(f) for f in F]
    L0, M0 = orc.cpn_loss(X, Z, R)
    assert M0 == pytest.approx(L0, rel=1e-14)


# ------------------------------------------------------------ TTV / TTM

def test_ttv_mags(orc):
    rng = np.random.default_rng(108)
    dims = (5, 6, 7)
    (i, j, l) = _keys(rng, dims, 60)
    x = rng.standard_normal(60).astype(np.float32)
    v = rng.standard_normal(dims[2])
    X = orc.Dok(dims, (i, j, l), x)
    Xd = _dense(dims, (i, j, l), x)
    yi, yj, y, ym = orc.ttv(X, v)
    _close(ym, (np.abs(Xd) @ np.abs(v))[yi, yj])
    _bounds(y, ym)
    gy = rng.standard_normal(len(yi)).astype(np.float32)
    gY = orc.Dok(dims[:2], (yi, yj), gy)
    Gd = _dense(dims[:2], (yi, yj), gy)
    dX, dXm, dv, dvm = orc.ttv_vjp(X, v, gY, i, j, l)
    # dX_p = gY(i, j) v(l) is one term: mag == |value|
    _close(dXm, np.abs(dX))
    _close(dvm, np.einsum("ijl,ij->l", np.abs(Xd), np.abs(Gd)))
    _bounds(dv, dvm)
    Xp = orc.Dok(dims, (i, j, l), np.abs(x))
    _, _, y2, ym2 = orc.ttv(Xp, np.abs(v))
    _close(ym2, y2)


@pytest.mark.parametrize("R", [1, 4])
def test_ttm_mags(orc, R):
    rng = np.random.default_rng(109 + R)
    dims = (5, 4, 6)
    (i, j, l) = _keys(rng, dims, 50)
    x = rng.standard_normal(50).astype(np.float32)
    U = rng.standard_normal((dims[2], R))
    X = orc.Dok(dims, (i, j, l), x)
    Xd = _dense(dims, (i, j, l), x)
    yi, yj, y, ym = orc.ttm(X, U, R)
    _close(ym, np.einsum("ijl,lr->ijr", np.abs(Xd), np.abs(U))[yi, yj])
    _bounds(y, ym)
    gY = rng.standard_normal((len(yi), R))
    Gd = np.zeros(dims[:2] + (R,))
    Gd[yi, yj] = gY
    dX, dXm, dU, dUm = orc.ttm_vjp(X, U, R, gY, i, j, l)
    _close(dXm, np.einsum("pr,pr->p", np.abs(Gd[i, j]), np.abs(U[l])))
    _close(dUm, np.einsum("ijl,ijr->lr", np.abs(Xd), np.abs(Gd)))
    _bounds(dX, dXm)
    _bounds(dU, dUm)
    Xp = orc.Dok(dims, (i, j, l), np.abs(x))
    _, _, y2, ym2 = orc.ttm(Xp, np.abs(U), R)
    _close(ym2, y2)


# --------------------------------------------------------------- BATAX

def test_batax_mag(orc):
    rng = np.random.default_rng(111)
    nr, nc, beta = 9, 6, -1.25
    row, col = _keys(rng, (nr, nc), 22)
    val = rng.standard_normal(22).astype(np.float32)
    A = orc.Dok((nr, nc), (row, col), val)
    rowptr, colind, jv, jm = orc.batax_jacobian(A, beta)
    aA = np.abs(_dense((nr, nc), (row, col), val))
    rows = np.repeat(np.arange(nc), np.diff(rowptr))
    _close(jm, (abs(beta) * aA.T @ aA)[rows, colind])
    _bounds(jv, jm)
    Ap = orc.Dok((nr, nc), (row, col), np.abs(val))
    _, _, jv2, jm2 = orc.batax_jacobian(Ap, 2.0)
    _close(jm2, jv2)


# ------------------------------------------------------ tangent of A B

def test_spmm_jvp_mags(orc):
    rng = np.random.default_rng(112)
    nr, nc, k = 7, 6, 3
    row, col = _keys(rng, (nr, nc), 20)
    val = rng.standard_normal(20).astype(np.float32)
    dval = rng.standard_normal(20).astype(np.float32)
    B = rng.standard_normal((nc, k)).astype(np.float32)
    dB = rng.standard_normal((nc, k)).astype(np.float32)
    A = orc.Dok((nr, nc), (row, col), val)
    dA = orc.Dok((nr, nc), (row, col), dval)
    C, Cm, dC, dCm = orc.spmm_jvp(A, dA, B, dB, k)
    aA = np.abs(_dense((nr, nc), (row, col), val))
    adA = np.abs(_dense((nr, nc), (row, col), dval))
    aB, adB = np.abs(B.astype(np.float64)), np.abs(dB.astype(np.float64))
    _close(Cm, aA @ aB)
    _close(dCm, adA @ aB + aA @ adB)
    _bounds(C, Cm)
    _bounds(dC, dCm)
    Ap = orc.Dok((nr, nc), (row, col), np.abs(val))
    dAp = orc.Dok((nr, nc), (row, col), np.abs(dval))
    C2, Cm2, dC2, dCm2 = orc.spmm_jvp(Ap, dAp, np.abs(B), np.abs(dB), k)
    _close(Cm2, C2)
    _close(dCm2, dC2)


@pytest.mark.parametrize("mode", [0, 1, 3])
def test_ttmn_mags(orc, mode):
    rng = np.random.default_rng(120 + mode)
    dims, R = (4, 3, 5, 4), 3
    c = _keys(rng, dims, 80)
    x = rng.standard_normal(80).astype(np.float32)
    X = orc.Dok(dims, c, x)
    Xd = _dense(dims, c, x)
    U = rng.standard_normal((dims[mode], R))
    others = [m for m in range(4) if m != mode]
    letters = "abcd"
    out = "".join(letters[m] for m in others) + "r"
    yk, y, ym = orc.ttmn(X, mode, U, R)
    Ymag = np.einsum(f"{letters},{letters[mode]}r->{out}", np.abs(Xd), np.abs(U))
    _close(ym, Ymag[tuple(yk)])
    _bounds(y, ym)
    gY = rng.standard_normal((len(yk[0]), R))
    Gd = np.zeros([dims[m] for m in others] + [R])
    Gd[tuple(yk)] = gY
    dX, dXm, dU, dUm = orc.ttmn_vjp(X, mode, U, R, gY, c)
    Gat = Gd[tuple(c[m] for m in others)]  # upstream row of every stored key
    _close(dXm, np.einsum("pr,pr->p", np.abs(Gat), np.abs(U[c[mode]])))
    _close(dUm, np.einsum(f"{letters},{out}->{letters[mode]}r", np.abs(Xd), np.abs(Gd)))
    _bounds(dX, dXm)
    _bounds(dU, dUm)
