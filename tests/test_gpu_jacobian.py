"""Jacobians and batches of tangents through the front end and the library,
against the oracle.

Jacobians of tensor-valued programs (the gradient API's one-hot seed,
Section 4.3) are compared with the reference interpreter's literal
tensorized evaluation of the same program; J V for a batch of tangents
(Section 4.2) with the interpreter's tensorized forward mode seeded with the
whole batch, and for the matrix product with the C oracle's forward-mode
tangent, one tangent at a time.  Results on stored keys are compared key by
key; the magnitudes are the same quantities evaluated on absolute values.
Indices and exact copies are bit-exact.
"""
import numpy as np
import pytest
import torch

from helpers import assert_mag_close
from oracle import sdql as ref
from test_gpu_parity import dev, edge_pattern, host, make_csr

pytestmark = pytest.mark.gpu

# the vector kernels of Section 7.1 (VVA parenthesised: a sum's body runs to
# the end of the expression), a sparse matrix-vector product, a
# matrix-valued program on a matrix's keys, the trace (Example 3) and the
# matrix product
VVA = "(sum(<i,v> in V1) {i -> v}) + (sum(<i,v> in V2) {i -> v})"
VSM = "sum(<i,v> in V) {i -> v * s * s}"
MATVEC = "sum(<i,r> in M) {i -> sum(<j,a> in r) a * x(j)}"
MATSQ = "sum(<i,r> in M) {i -> sum(<j,a> in r) {j -> a * a * x(j) * s}}"
TRACE = "sum(<i,r> in M) r(i)"
SPMM = "sum(<i,r> in A) {i -> sum(<j,a> in r) sum(<c,b> in B(j)) {c -> a * b}}"
SAMPLED = ("sum(<i,r> in A) {i -> sum(<j,a> in r) {j -> a * sum(<c,x> in X(i)) x * Y(j)(c)}}")


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import sdql
    return sdql


@pytest.fixture(scope="module")
def nsd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import nsd as m
    return m


def sparse_vector(rng, n, nnz):
    keys = np.sort(rng.choice(n, size=nnz, replace=False)).astype(np.int32)
    return keys, rng.standard_normal(nnz).astype(np.float32)


def svec(n, keys, val):
    from paper_2303_07030_amd.operand import DeviceSparseVec
    return DeviceSparseVec(n, keys, val)


def real(s):
    return torch.tensor([s], dtype=torch.float64, device="cuda")


def matrix(seed, nrows=160, ncols=200):
    """Power-law rows with empty ones (first, middle, last) and a long row;
    the default shape of edge_pattern when asked for it."""
    from paper_2303_07030_amd.operand import DeviceCsr
    if nrows >= 700:
        nr, nc, rowptr, colind, val = edge_pattern(seed, nrows, ncols)
    else:
        rng = np.random.default_rng(seed)
        lengths = np.minimum((8 * rng.pareto(1.2, nrows)).astype(np.int64), ncols // 2)
        lengths[[0, nrows // 2, nrows - 1]] = 0
        lengths[nrows // 3] = ncols - 10
        nr, nc = nrows, ncols
        rowptr, colind, val = make_csr(rng, nrows, ncols, lengths, hot_col=3)
    rows = np.repeat(np.arange(nr, dtype=np.int32), np.diff(rowptr))
    return DeviceCsr(nr, nc, rowptr, colind, val), rowptr, colind, val, rows


def as_dict(layout, arr, coords):
    """A result as {key: value}: coords maps a sparse input to its stored
    keys' coordinate arrays."""
    kind, P, keymap, shape = layout
    arr = np.asarray(arr)
    if kind == "pattern":
        cs = coords[P]
        return {tuple(int(cs[i][e]) for i in keymap): float(arr[e]) for e in range(arr.shape[0])}
    if kind == "scalar":
        return {(): float(arr.reshape(-1)[0])}
    return {idx: float(arr[idx]) for idx in np.ndindex(*shape)}


def compare(got, want, mag, what, exact=False):
    """Key-by-key parity: every key the oracle stores is a key of the result
    (pattern results hold all stored keys, absent ones being 0)."""
    missing = set(want) - set(got)
    assert not missing, f"{what}: keys {sorted(missing)[:5]} missing"
    keys = sorted(got)
    g = np.array([got[k] for k in keys])
    w = np.array([want.get(k, 0.0) for k in keys])
    if exact:
        assert np.array_equal(g.astype(np.float32), w.astype(np.float32)), what
        return
    m = np.array([mag.get(k, 0.0) for k in keys])
    assert_mag_close(g, w, m, what=what)


def abs_env(env):
    return {n: ref._replace_leaves(v, lambda _, x: abs(x)) if isinstance(v, dict) else abs(v)
            for n, v in env.items()}


def vec_env(keys, val):
    return {int(k): float(v) for k, v in zip(keys, val.astype(np.float64))}


# ------------------------------------------- Jacobians (the gradient API)


@pytest.mark.parametrize("n,nnz", [(1, 1), (300, 37), (5000, 700)])
def test_vva_value_and_jacobians(S, n, nnz):
    rng = np.random.default_rng(n)
    k1, v1 = sparse_vector(rng, n, nnz)
    k2, v2 = sparse_vector(rng, n, max(1, nnz // 2))
    prog = S.compile(VVA, V1=S.SparseVec(n), V2=S.SparseVec(n))
    V1, V2 = svec(n, k1, v1), svec(n, k2, v2)
    plan = prog.plan(("V1", "V2"))
    out = plan.execute({"V1": V1, "V2": V2})
    env = {"V1": vec_env(k1, v1), "V2": vec_env(k2, v2)}
    coords = {"V1": (k1,), "V2": (k2,)}
    compare(as_dict(plan.layout("value"), host(out["value"]), coords),
            dict(ref.leaves(ref.value(VVA, env))),
            dict(ref.leaves(ref.value(VVA, abs_env(env)))), "value")
    for x in ("V1", "V2"):
        # the identity on x's stored keys, bit for bit
        got = as_dict(plan.layout("d" + x), host(out["d" + x]), coords)
        compare(got, ref.jacobian_tensorized(VVA, env, x), None, "d" + x, exact=True)


@pytest.mark.parametrize("s", [0.0, -1.25, 3.0])
def test_vsm_value_and_jacobians(S, s):
    rng = np.random.default_rng(7)
    keys, val = sparse_vector(rng, 2000, 300)
    prog = S.compile(VSM, V=S.SparseVec(2000), s=S.Dense())
    V = svec(2000, keys, val)
    plan = prog.plan(("s", "V"))
    out = plan.execute({"V": V, "s": real(s)})
    env = {"V": vec_env(keys, val), "s": s}
    coords = {"V": (keys,)}
    compare(as_dict(plan.layout("value"), host(out["value"]), coords),
            dict(ref.leaves(ref.value(VSM, env))),
            dict(ref.leaves(ref.value(VSM, abs_env(env)))), "value")
    for x in ("s", "V"):
        compare(as_dict(plan.layout("d" + x), host(out["d" + x]), coords),
                ref.jacobian_tensorized(VSM, env, x),
                ref.jacobian_tensorized(VSM, abs_env(env), x), "d" + x)


def test_matvec_jacobians_are_the_matrix_and_the_gathered_vector(S):
    A, rowptr, colind, val, rows = matrix(3)
    x = np.random.default_rng(3).standard_normal(A.ncols).astype(np.float32)
    prog = S.compile(MATVEC, M=S.Sparse(A.nrows, A.ncols), x=S.Dense(A.ncols))
    plan = prog.plan(("x", "M"))
    out = plan.execute({"M": A, "x": dev(x)})
    env = {"M": ref.csr_dict(rowptr, colind, val.astype(np.float64)), "x": ref.dense_dict(x)}
    coords = {"M": (rows, colind)}
    for w in ("x", "M"):
        # dx = M on its keys, dM(i, i, j) = x(j): exact copies
        compare(as_dict(plan.layout("d" + w), host(out["d" + w]), coords),
                ref.jacobian_tensorized(MATVEC, env, w), None, "d" + w, exact=True)


@pytest.mark.parametrize("s", [0.5, -2.0])
def test_matrix_valued_program_and_its_jacobians(S, s):
    A, rowptr, colind, val, rows = matrix(4)
    x = np.random.default_rng(4).standard_normal(A.ncols).astype(np.float32)
    prog = S.compile(MATSQ, M=S.Sparse(A.nrows, A.ncols), x=S.Dense(A.ncols), s=S.Dense())
    plan = prog.plan(("M", "x", "s"))
    out = plan.execute({"M": A, "x": dev(x), "s": real(s)})
    env = {"M": ref.csr_dict(rowptr, colind, val.astype(np.float64)), "x": ref.dense_dict(x),
           "s": s}
    aenv = abs_env(env)
    coords = {"M": (rows, colind)}
    compare(as_dict(plan.layout("value"), host(out["value"]), coords),
            dict(ref.leaves(ref.value(MATSQ, env))),
            dict(ref.leaves(ref.value(MATSQ, aenv))), "value")
    for w in ("M", "x", "s"):
        compare(as_dict(plan.layout("d" + w), host(out["d" + w]), coords),
                ref.jacobian_tensorized(MATSQ, env, w),
                ref.jacobian_tensorized(MATSQ, aenv, w), "d" + w)


def test_trace_value_and_gradient_through_the_front_end(S):
    from paper_2303_07030_amd.operand import DeviceCsr
    rng = np.random.default_rng(9)
    n = 400
    rowptr = [0]
    cols = []
    for i in range(n):
        c = set(rng.choice(n, size=int(rng.integers(0, 6)), replace=False).tolist())
        if i % 3 == 0:
            c.add(i)  # a third of the diagonal keys are stored
        cols.extend(sorted(c))
        rowptr.append(len(cols))
    rowptr, colind = np.array(rowptr, np.int32), np.array(cols, np.int32)
    val = rng.standard_normal(len(colind)).astype(np.float32)
    prog = S.compile(TRACE, M=S.Sparse(n, n))
    out = prog.run({"M": DeviceCsr(n, n, rowptr, colind, val)}, grads=("M",))
    env = {"M": ref.csr_dict(rowptr, colind, val.astype(np.float64))}
    env_abs = {"M": ref.csr_dict(rowptr, colind, np.abs(val).astype(np.float64))}
    assert_mag_close(host(out["value"])[0], ref.value(TRACE, env), ref.value(TRACE, env_abs),
                     what="trace")
    want = ref.gradient_tensorized(TRACE, env, "M")
    rows = np.repeat(np.arange(n), np.diff(rowptr))
    assert np.array_equal(host(out["dM"]), np.array(
        [want[(int(r), int(c))] for r, c in zip(rows, colind)], dtype=np.float32))


# ------------------------------------------------ J V, batches of tangents


def batch_dict(V, coords=None):
    """Tangents [m, ...] as the interpreter's tau levels: for a sparse input
    its stored keys (coords) then t; for a dense one its index then t; for a
    real just t."""
    m = V.shape[0]
    out = {}
    if V.ndim == 1:
        return {t: float(V[t]) for t in range(m)}
    if coords is not None:
        for e in range(V.shape[1]):
            d = out
            key = [int(c[e]) for c in coords]
            for k in key[:-1]:
                d = d.setdefault(k, {})
            d[key[-1]] = {t: float(V[t, e]) for t in range(m)}
        return out
    for idx in np.ndindex(*V.shape[1:]):
        d = out
        for k in idx[:-1]:
            d = d.setdefault(int(k), {})
        d[int(idx[-1])] = {t: float(V[(t,) + idx]) for t in range(m)}
    return out


def tangent_result(layout, tan, coords):
    """{output key + (t,): value} of a batch of tangents [m, ...]."""
    out = {}
    for t in range(tan.shape[0]):
        for k, v in as_dict(layout, tan[t], coords).items():
            out[k + (t,)] = v
    return out


def test_jvp_of_the_vector_kernels(S):
    rng = np.random.default_rng(21)
    n, m = 3000, 5
    k1, v1 = sparse_vector(rng, n, 400)
    k2, v2 = sparse_vector(rng, n, 250)
    V1, V2 = svec(n, k1, v1), svec(n, k2, v2)
    prog = S.compile(VVA, V1=S.SparseVec(n), V2=S.SparseVec(n))
    T1 = rng.standard_normal((m, len(k1))).astype(np.float32)
    T2 = rng.standard_normal((m, len(k2))).astype(np.float32)
    out = prog.jvp({"V1": V1, "V2": V2}, {"V1": dev(T1), "V2": dev(T2)})
    env = {"V1": vec_env(k1, v1), "V2": vec_env(k2, v2)}
    tans = {"V1": batch_dict(T1, (k1,)), "V2": batch_dict(T2, (k2,))}
    want = ref.jvp_tensorized(VVA, env, tans)
    wmag = ref.jvp_tensorized(VVA, abs_env(env), {x: ref._replace_leaves(v, lambda _, y: abs(y))
                                                 for x, v in tans.items()})
    lay = prog.jvp_plan(("V1", "V2")).layout("tangent")
    compare(tangent_result(lay, host(out["tangent"]), {}), want, wmag, "VVA tangent")
    # VSM along s and V at once
    keys, val = sparse_vector(rng, n, 300)
    V = svec(n, keys, val)
    prog = S.compile(VSM, V=S.SparseVec(n), s=S.Dense())
    Ts = rng.standard_normal(m)
    TV = rng.standard_normal((m, len(keys))).astype(np.float32)
    out = prog.jvp({"V": V, "s": real(0.7)}, {"s": dev(Ts), "V": dev(TV)})
    env = {"V": vec_env(keys, val), "s": 0.7}
    tans = {"s": batch_dict(Ts), "V": batch_dict(TV, (keys,))}
    want = ref.jvp_tensorized(VSM, env, tans)
    wmag = ref.jvp_tensorized(VSM, abs_env(env), {x: ref._replace_leaves(v, lambda _, y: abs(y))
                                                 for x, v in tans.items()})
    lay = prog.jvp_plan(("s", "V")).layout("tangent")
    compare(tangent_result(lay, host(out["tangent"]), {"V": (keys,)}), want, wmag,
            "VSM tangent")


def test_jvp_of_a_matrix_valued_program(S):
    A, rowptr, colind, val, rows = matrix(5)
    rng = np.random.default_rng(5)
    x = rng.standard_normal(A.ncols).astype(np.float32)
    m = 3
    prog = S.compile(MATSQ, M=S.Sparse(A.nrows, A.ncols), x=S.Dense(A.ncols), s=S.Dense())
    TM = rng.standard_normal((m, A.nnz)).astype(np.float32)
    Tx = rng.standard_normal((m, A.ncols)).astype(np.float32)
    Ts = rng.standard_normal(m)
    out = prog.jvp({"M": A, "x": dev(x), "s": real(1.5)},
                   {"M": dev(TM), "x": dev(Tx), "s": dev(Ts)})
    env = {"M": ref.csr_dict(rowptr, colind, val.astype(np.float64)), "x": ref.dense_dict(x),
           "s": 1.5}
    tans = {"M": batch_dict(TM, (rows, colind)), "x": batch_dict(Tx), "s": batch_dict(Ts)}
    want = ref.jvp_tensorized(MATSQ, env, tans)
    wmag = ref.jvp_tensorized(MATSQ, abs_env(env), {x_: ref._replace_leaves(v, lambda _, y: abs(y))
                                                   for x_, v in tans.items()})
    lay = prog.jvp_plan(("M", "x", "s")).layout("tangent")
    compare(tangent_result(lay, host(out["tangent"]), {"M": (rows, colind)}), want, wmag,
            "MATSQ tangent")
    compare(as_dict(lay, host(out["value"]), {"M": (rows, colind)}),
            dict(ref.leaves(ref.value(MATSQ, env))),
            dict(ref.leaves(ref.value(MATSQ, abs_env(env)))), "value")


@pytest.mark.parametrize("k", [1, 8, 33])
def test_jvp_of_a_sampled_product(S, k):
    # J V over the SDDMM kernel: tangents of A(i,j) <X(i), Y(j)> on A's keys
    # along A, X and Y at once, against the batched forward mode
    A, rowptr, colind, val, rows = matrix(7)
    rng = np.random.default_rng(70 + k)
    X = rng.standard_normal((A.nrows, k)).astype(np.float32)
    Y = rng.standard_normal((A.ncols, k)).astype(np.float32)
    m = 3
    prog = S.compile(SAMPLED, A=S.Sparse(A.nrows, A.ncols), X=S.Dense(A.nrows, k),
                     Y=S.Dense(A.ncols, k))
    TA = rng.standard_normal((m, A.nnz)).astype(np.float32)
    TX = rng.standard_normal((m, A.nrows, k)).astype(np.float32)
    TY = rng.standard_normal((m, A.ncols, k)).astype(np.float32)
    out = prog.jvp({"A": A, "X": dev(X), "Y": dev(Y)},
                   {"A": dev(TA), "X": dev(TX), "Y": dev(TY)})
    env = {"A": ref.csr_dict(rowptr, colind, val.astype(np.float64)), "X": ref.dense_dict(X),
           "Y": ref.dense_dict(Y)}
    tans = {"A": batch_dict(TA, (rows, colind)), "X": batch_dict(TX), "Y": batch_dict(TY)}
    want = ref.jvp_tensorized(SAMPLED, env, tans)
    wmag = ref.jvp_tensorized(SAMPLED, abs_env(env),
                              {x: ref._replace_leaves(v, lambda _, y: abs(y))
                               for x, v in tans.items()})
    lay = prog.jvp_plan(("A", "X", "Y")).layout("tangent")
    coords = {"A": (rows, colind)}
    compare(tangent_result(lay, host(out["tangent"]), coords), want, wmag, "tangent")
    compare(as_dict(lay, host(out["value"]), coords), dict(ref.leaves(ref.value(SAMPLED, env))),
            dict(ref.leaves(ref.value(SAMPLED, abs_env(env)))), "value")


@pytest.mark.parametrize("wrt", [("A", "B"), ("A",), ("B",)])
@pytest.mark.parametrize("k", [1, 3, 64, 70])
def test_jvp_of_the_matrix_product(S, orc, wrt, k):
    # fused (one batched call) and term by term, against the C oracle's
    # forward-mode tangent of C = A B, one tangent at a time
    A, rowptr, colind, val, rows = matrix(6, 700, 900)
    rng = np.random.default_rng(k)
    m = 6
    B = rng.standard_normal((A.ncols, k) if k > 1 else (A.ncols,)).astype(np.float32)
    text = SPMM if k > 1 else MATVEC.replace("M", "A").replace("x(j)", "B(j)")
    prog = S.compile(text, A=S.Sparse(A.nrows, A.ncols),
                     B=S.Dense(A.ncols, k) if k > 1 else S.Dense(A.ncols))
    TA = rng.standard_normal((m, A.nnz)).astype(np.float32)
    TB = rng.standard_normal((m,) + B.shape).astype(np.float32)
    tans = {x: dev(TA if x == "A" else TB) for x in wrt}
    fused = prog.jvp({"A": A, "B": dev(B)}, tans)
    assert not prog.jvp_plan(wrt).per_tangent
    unfused = prog.jvp({"A": A, "B": dev(B)}, tans, fuse=False)
    D = orc.Dok((A.nrows, A.ncols), (rows, colind), val)
    B2 = B.reshape(A.ncols, k)
    for t in range(m):
        dA = TA[t] if "A" in wrt else np.zeros(A.nnz, np.float32)
        dB = TB[t].reshape(A.ncols, k) if "B" in wrt else np.zeros_like(B2)
        C, Cm, dC, dCm = orc.spmm_jvp(D, orc.Dok((A.nrows, A.ncols), (rows, colind), dA), B2,
                                      dB, k)
        for name, got in (("fused", fused), ("term by term", unfused)):
            assert_mag_close(host(got["tangent"][t]).reshape(A.nrows, k), dC, dCm,
                             what=f"{name} dC[{t}]")
        if t == 0:
            assert_mag_close(host(fused["value"]).reshape(A.nrows, k), C, Cm, what="C")


def test_jvp_of_real_valued_losses_is_the_gradient_along_each_tangent(S, orc):
    # forward mode against reverse mode: the tangent of a loss along v is
    # <grad L, v> (Section 6, the differential), with the gradients from
    # the C oracle; the magnitude is sum |terms of grad| * |v|
    from test_sdql import FROB, GNN
    A, rowptr, colind, val, rows = matrix(9, 700, 900)
    rng = np.random.default_rng(9)
    k, m = 16, 4
    D = orc.Dok((A.nrows, A.ncols), (rows, colind), val)
    TA = rng.standard_normal((m, A.nnz)).astype(np.float32)
    # 1/2 ||A B||^2 along A and B
    B = rng.standard_normal((A.ncols, k)).astype(np.float32)
    TB = rng.standard_normal((m, A.ncols, k)).astype(np.float32)
    prog = S.compile(FROB, A=S.Sparse(A.nrows, A.ncols), B=S.Dense(A.ncols, k))
    got = host(prog.jvp({"A": A, "B": dev(B)}, {"A": dev(TA), "B": dev(TB)})["tangent"])
    C, Cm = orc.spmm(D, B, k)
    gA, gAm = orc.sddmm(D, C, B, k, rows, colind, Xmag=Cm)
    gB, gBm = orc.spmm_t(D, C, k, Gmag=Cm)
    for t in range(m):
        want = gA @ TA[t].astype(np.float64) + np.sum(gB * TB[t])
        mag = gAm @ np.abs(TA[t]).astype(np.float64) + np.sum(gBm * np.abs(TB[t]))
        assert_mag_close(got[t], want, mag, what=f"frob tangent {t}")
    # the GNN layer's loss along A, H and G
    H = rng.standard_normal((A.ncols, k)).astype(np.float32)
    G = rng.standard_normal((A.nrows, k)).astype(np.float32)
    TH = rng.standard_normal((m, A.ncols, k)).astype(np.float32)
    TG = rng.standard_normal((m, A.nrows, k)).astype(np.float32)
    prog = S.compile(GNN, A=S.Sparse(A.nrows, A.ncols), H=S.Dense(A.ncols, k),
                     G=S.Dense(A.nrows, k))
    got = host(prog.jvp({"A": A, "H": dev(H), "G": dev(G)},
                        {"A": dev(TA), "H": dev(TH), "G": dev(TG)})["tangent"])
    gA, gAm = orc.sddmm(D, G, H, k, rows, colind)
    gH, gHm = orc.spmm_t(D, G, k)
    gG, gGm = orc.spmm(D, H, k)
    for t in range(m):
        want = (gA @ TA[t].astype(np.float64) + np.sum(gH * TH[t]) + np.sum(gG * TG[t]))
        mag = (gAm @ np.abs(TA[t]).astype(np.float64) + np.sum(gHm * np.abs(TH[t]))
               + np.sum(gGm * np.abs(TG[t])))
        assert_mag_close(got[t], want, mag, what=f"gnn tangent {t}")


# ------------------------------------------------ the C-ABI entry points


def run_jvp_batch(nsd, A, m, TA, B, TB, k, want_C=True):
    C = torch.full((A.nrows, k), np.nan, dtype=torch.float32, device="cuda") if want_C else None
    dC = torch.full((max(m, 1), A.nrows, k), np.nan, dtype=torch.float32, device="cuda")
    ws = torch.empty(nsd.nsd_spmm_jvp_batch_workspace_size(A.desc, k), dtype=torch.uint8,
                     device="cuda")
    nsd.nsd_spmm_jvp_batch(A.desc, m, None if TA is None else dev(TA), dev(B),
                           None if TB is None else dev(TB), k, C, dC, ws)
    return (host(C) if want_C else None), host(dC)[:m]


@pytest.mark.parametrize("m,k,has_dA,has_dB,want_C", [
    (0, 3, True, True, True), (1, 3, True, True, True), (4, 64, True, True, False),
    (5, 1, True, False, True), (9, 70, False, True, True), (6, 256, True, True, True),
    (3, 13, True, True, True),
])
def test_spmm_jvp_batch_against_the_oracle_and_single_tangents(nsd, orc, m, k, has_dA, has_dB,
                                                               want_C):
    A, rowptr, colind, val, rows = matrix(8, 700, 900)
    rng = np.random.default_rng(m * 100 + k)
    B = rng.standard_normal((A.ncols, k)).astype(np.float32)
    TA = rng.standard_normal((m, A.nnz)).astype(np.float32) if has_dA else None
    TB = rng.standard_normal((m, A.ncols, k)).astype(np.float32) if has_dB else None
    C, dC = run_jvp_batch(nsd, A, m, TA, B, TB, k, want_C)
    D = orc.Dok((A.nrows, A.ncols), (rows, colind), val)
    zA, zB = np.zeros(A.nnz, np.float32), np.zeros((A.ncols, k), np.float32)
    for t in range(max(m, 1)):
        dA = TA[t] if has_dA and m else zA
        dB = TB[t] if has_dB and m else zB
        Co, Cm, dCo, dCm = orc.spmm_jvp(D, orc.Dok((A.nrows, A.ncols), (rows, colind), dA), B,
                                        dB, k)
        if want_C and t == 0:
            assert_mag_close(C, Co, Cm, what="C")
        if t >= m:
            break
        assert_mag_close(dC[t], dCo, dCm, what=f"dC[{t}]")
        # the same sums in the same order as the one-tangent kernel
        C1 = torch.empty((A.nrows, k), dtype=torch.float32, device="cuda")
        dC1 = torch.empty((A.nrows, k), dtype=torch.float32, device="cuda")
        nsd.nsd_spmm_jvp(A.desc, dev(dA), dev(B), dev(dB), k, C1, dC1, A.workspace(2 * k))
        assert np.array_equal(host(dC1), dC[t]), f"dC[{t}] differs from nsd_spmm_jvp"
        if want_C:
            assert np.array_equal(host(C1), C)


def test_spmm_jvp_batch_empty_and_errors(nsd):
    from paper_2303_07030_amd.operand import DeviceCsr
    A = DeviceCsr(5, 4, np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    B = np.ones((4, 3), np.float32)
    C, dC = run_jvp_batch(nsd, A, 3, np.zeros((3, 0), np.float32), B,
                          np.ones((3, 4, 3), np.float32), 3)
    assert np.all(C == 0) and np.all(dC == 0)
    with pytest.raises(nsd.NsdError):
        nsd.nsd_spmm_jvp_batch(A.desc, -1, None, dev(B), None, 3, None, None,
                               torch.empty(1 << 16, dtype=torch.uint8, device="cuda"))
    with pytest.raises(nsd.NsdError):
        nsd.nsd_spmm_jvp_batch(A.desc, 1, None, dev(B), None, 3, None, None,
                               torch.empty(1, dtype=torch.uint8, device="cuda"))


@pytest.mark.parametrize("n", [0, 1, 1000, 300_000])
def test_scale_against_double_products(nsd, n):
    rng = np.random.default_rng(n)
    x1 = rng.standard_normal(n).astype(np.float32)
    x2 = rng.standard_normal(3 * n + 1).astype(np.float32)
    idx = rng.integers(0, 3 * n + 1, size=n).astype(np.int32)
    s1, s2 = 1.7, -0.3
    y0 = rng.standard_normal(n).astype(np.float32)
    want = (2.0 * s1 * s2 * x1.astype(np.float64) * x2[idx].astype(np.float64)
            + 0.5 * y0.astype(np.float64)).astype(np.float32)
    y = dev(y0)
    nsd.nsd_scale(n, 2.0, real(s1), real(s2), dev(x1), dev(x2), dev(idx), 0.5, y)
    assert np.array_equal(host(y), want)
    # beta 0 does not read y (NaN stays out); scatter to distinct indices
    out = torch.full((2 * n + 1,), np.nan, dtype=torch.float32, device="cuda")
    dst = rng.permutation(2 * n + 1)[:n].astype(np.int32)
    nsd.nsd_scale(n, 1.0, None, None, dev(x1), None, None, 0.0, out, dev(dst))
    got = host(out)
    assert np.array_equal(got[dst], x1)
    rest = np.setdiff1d(np.arange(2 * n + 1), dst)
    assert np.all(np.isnan(got[rest]))


def test_scale_real(nsd):
    y = real(4.0)
    nsd.nsd_scale_real(3.0, real(2.0), real(-0.5), real(1.25), 0.5, y)
    assert host(y)[0] == 3.0 * 2.0 * -0.5 * 1.25 + 0.5 * 4.0
    nsd.nsd_scale_real(2.0, None, None, None, 0.0, y)
    assert host(y)[0] == 2.0
