"""Front end on the GPU: programs in Logical SDQLite, differentiated and lowered
to the library's kernels, against the fp64 oracle.

At moderate size (several tiles, empty rows, a row spread over many slots)
each result is checked against the C oracle's routines for the same
quantity, with their magnitudes; on tiny inputs the gradients of the
programs with positive coefficients are checked against the reference
interpreter's forward-mode gradient, the magnitude being that gradient
evaluated on absolute values.
"""
import numpy as np
import pytest
import torch

from helpers import assert_mag_close
from oracle import sdql as ref
from test_gpu_parity import edge_pattern
from test_sdql import FROB, GNN, MF, MF_INNER, QUAD, SMVM, DOT1, rand_csr

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import sdql
    return sdql


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def operand(nrows, ncols, rowptr, colind, val):
    from paper_2303_07030_amd.operand import DeviceCsr
    return DeviceCsr(nrows, ncols, rowptr, colind, val)


@pytest.fixture(scope="module")
def mat(orc, S):
    nrows, ncols, rowptr, colind, val = edge_pattern(21)
    A = operand(nrows, ncols, rowptr, colind, val)
    D = orc.Dok.from_csr(nrows, ncols, rowptr, colind, val)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    return A, D, rows, colind


@pytest.mark.parametrize("fuse", [True, False])
def test_smvm(S, orc, mat, fuse):
    A, D, rows, cols = mat
    x = np.random.default_rng(1).standard_normal(A.ncols).astype(np.float32)
    prog = S.compile(SMVM, A=S.Sparse(A.nrows, A.ncols), x=S.Dense(A.ncols))
    out = prog.run({"A": A, "x": dev(x)}, grads=("A", "x"), fuse=fuse)
    L, Lm = orc.loss_sum_spmv(D, x)
    assert_mag_close(host(out["value"])[0], L, Lm, what="value")
    dA, dAm = orc.sddmm(D, None, x.reshape(-1, 1), 1, rows, cols)
    assert_mag_close(host(out["dA"]), dA, dAm, what="dA")
    dx, dxm = orc.spmm_t(D, None, 1)
    assert_mag_close(host(out["dx"]), dx[:, 0], dxm[:, 0], what="dx")


@pytest.mark.parametrize("fuse", [True, False])
@pytest.mark.parametrize("k", [1, 12, 64])
def test_frob(S, orc, mat, k, fuse):
    A, D, rows, cols = mat
    B = np.random.default_rng(k).standard_normal((A.ncols, k)).astype(np.float32)
    prog = S.compile(FROB, A=S.Sparse(A.nrows, A.ncols), B=S.Dense(A.ncols, k))
    out = prog.run({"A": A, "B": dev(B)}, grads=("A", "B"), fuse=fuse)
    C, Cm = orc.spmm(D, B, k)
    L, Lm = orc.loss_half_sq(C, Cm)
    assert_mag_close(host(out["value"])[0], L, Lm, what="value")
    dA, dAm = orc.sddmm(D, C, B, k, rows, cols, Xmag=Cm)
    assert_mag_close(host(out["dA"]), dA, dAm, what="dA")
    dB, dBm = orc.spmm_t(D, C, k, Gmag=Cm)
    assert_mag_close(host(out["dB"]), dB, dBm, what="dB")


@pytest.mark.parametrize("fuse", [True, False])
def test_gnn(S, orc, mat, fuse):
    A, D, rows, cols = mat
    k = 16
    rng = np.random.default_rng(2)
    H = rng.standard_normal((A.ncols, k)).astype(np.float32)
    G = rng.standard_normal((A.nrows, k)).astype(np.float32)
    prog = S.compile(GNN, A=S.Sparse(A.nrows, A.ncols), H=S.Dense(A.ncols, k),
                     G=S.Dense(A.nrows, k))
    out = prog.run({"A": A, "H": dev(H), "G": dev(G)}, grads=("A", "H", "G"), fuse=fuse)
    L, Lm = orc.loss_bilinear(D, G, H, k)
    assert_mag_close(host(out["value"])[0], L, Lm, what="value")
    dA, dAm = orc.sddmm(D, G, H, k, rows, cols)
    assert_mag_close(host(out["dA"]), dA, dAm, what="dA")
    dH, dHm = orc.spmm_t(D, G, k)
    assert_mag_close(host(out["dH"]), dH, dHm, what="dH")
    dG, dGm = orc.spmm(D, H, k)
    assert_mag_close(host(out["dG"]), dG, dGm, what="dG")


@pytest.mark.parametrize("grads", [("A", "U", "V"), ("U", "V")], ids=["with_dA", "fused"])
@pytest.mark.parametrize("text", [MF, MF_INNER], ids=["let_outside", "let_inside"])
def test_mf(S, orc, mat, text, grads):
    A, D, rows, cols = mat
    k = 12
    rng = np.random.default_rng(3)
    U = (0.3 * rng.standard_normal((A.nrows, k))).astype(np.float32)
    V = (0.3 * rng.standard_normal((A.ncols, k))).astype(np.float32)
    prog = S.compile(text, A=S.Sparse(A.nrows, A.ncols), U=S.Dense(A.nrows, k),
                     V=S.Dense(A.ncols, k))
    plan = prog.plan(grads)
    assert (plan.kernels() == ["loss_mf"]) == ("A" not in grads)
    out = prog.run({"A": A, "U": dev(U), "V": dev(V)}, grads=grads)
    L, Lm = orc.mf_loss(D, U, V, k)
    assert_mag_close(host(out["value"])[0], L, Lm, what="value")
    dU, dUm = orc.mf_grad(D, U, V, k, 0)
    assert_mag_close(host(out["dU"]), dU, dUm, what="dU")
    dV, dVm = orc.mf_grad(D, U, V, k, 1)
    assert_mag_close(host(out["dV"]), dV, dVm, what="dV")
    if "A" in grads:
        r, rm = orc.mf_resid(D, U, V, k, rows, cols)
        assert_mag_close(host(out["dA"]), 2 * r, 2 * rm, what="dA")


def test_two_terms_accumulate(S, orc):
    # d/dx of sum A_ij x_j x_i = A^T x + A x: two kernels into one result
    n, _, rowptr, colind, val = edge_pattern(23, nrows=900, ncols=900)
    A = operand(n, n, rowptr, colind, val)
    D = orc.Dok.from_csr(n, n, rowptr, colind, val)
    x = np.random.default_rng(4).standard_normal(n).astype(np.float32)
    prog = S.compile(QUAD, A=S.Sparse(n, n), x=S.Dense(n))
    out = prog.run({"A": A, "x": dev(x)}, grads=("x",), value=False)
    t1, m1 = orc.spmm_t(D, x.reshape(-1, 1), 1)
    t2, m2 = orc.spmm(D, x.reshape(-1, 1), 1)
    assert_mag_close(host(out["dx"]), (t1 + t2)[:, 0], (m1 + m2)[:, 0], what="dx")


@pytest.mark.parametrize("n", [0, 1, 1000, 300001])
def test_dense_dot_product(S, n):
    rng = np.random.default_rng(n)
    v1 = rng.standard_normal(n).astype(np.float32)
    v2 = rng.standard_normal(n).astype(np.float32)
    prog = S.compile(DOT1, V1=S.Dense(n), V2=S.Dense(n))
    out = prog.run({"V1": dev(v1), "V2": dev(v2)}, grads=("V1", "V2"))
    a, b = v1.astype(np.float64), v2.astype(np.float64)
    assert_mag_close(host(out["value"])[0], a @ b, np.abs(a) @ np.abs(b), what="value")
    assert np.array_equal(host(out["dV1"]), v2)
    assert np.array_equal(host(out["dV2"]), v1)


def test_repeat_runs_are_bitwise_equal(S, mat):
    A = mat[0]
    k = 8
    B = np.random.default_rng(5).standard_normal((A.ncols, k)).astype(np.float32)
    prog = S.compile(FROB, A=S.Sparse(A.nrows, A.ncols), B=S.Dense(A.ncols, k))
    r1 = prog.run({"A": A, "B": dev(B)}, grads=("A", "B"))
    r2 = prog.run({"A": A, "B": dev(B)}, grads=("A", "B"))
    for name in r1:
        assert np.array_equal(host(r1[name]), host(r2[name])), name


TINY = [
    ("smvm", SMVM, lambda nr, nc, k: dict(x=(nc,)), ("A", "x")),
    ("frob", FROB, lambda nr, nc, k: dict(B=(nc, k)), ("A", "B")),
    ("gnn", GNN, lambda nr, nc, k: dict(H=(nc, k), G=(nr, k)), ("A", "H", "G")),
    ("quad", QUAD, lambda nr, nc, k: dict(x=(nc,)), ("A", "x")),
]


@pytest.mark.parametrize("name,text,dense,grads", TINY, ids=[c[0] for c in TINY])
def test_tiny_against_the_interpreter(S, name, text, dense, grads):
    rng = np.random.default_rng(6)
    nr = nc = 8
    k = 3
    rowptr, colind, val = rand_csr(rng, nr, nc, 22)
    val = val.astype(np.float32)
    decls = {"A": S.Sparse(nr, nc)}
    env = {"A": ref.csr_dict(rowptr, colind, val.astype(np.float64))}
    env_abs = {"A": ref.csr_dict(rowptr, colind, np.abs(val).astype(np.float64))}
    inputs = {"A": operand(nr, nc, rowptr.astype(np.int32), colind.astype(np.int32), val)}
    for n, shape in dense(nr, nc, k).items():
        a = rng.standard_normal(shape).astype(np.float32)
        decls[n] = S.Dense(*shape)
        env[n] = ref.dense_dict(a.astype(np.float64))
        env_abs[n] = ref.dense_dict(np.abs(a).astype(np.float64))
        inputs[n] = dev(a)
    out = S.compile(text, **decls).run(inputs, grads=grads)
    assert_mag_close(host(out["value"])[0], ref.value(text, env), ref.value(text, env_abs),
                     what="value")
    for x in grads:
        want, mag = ref.gradient(text, env, x), ref.gradient(text, env_abs, x)
        got = host(out["d" + x])
        keys = sorted(want)   # row-major: CSR order for A
        g = got if x == "A" else np.array([got[key] for key in keys])
        assert_mag_close(g, np.array([want[q] for q in keys]), np.array([mag[q] for q in keys]),
                         what=f"d{x}")
