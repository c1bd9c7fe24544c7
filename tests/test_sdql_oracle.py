"""Pins for the reference interpreter of Logical SDQLite (oracle/sdql.py).

Its values are tied to numpy (dot and matrix products, Examples 1 and 2 and
the matrix product of Section 3), to the semi-ring dictionary laws of
Section 2 (absent keys read as zero, insertion adds), and to the fp64 C
oracle's losses; its forward-mode gradients are tied to closed forms and to
central finite differences, which share nothing with the dual numbers.
"""
import numpy as np
import pytest

from oracle import sdql as ref


def rand_csr(rng, nr, nc, nnz, empty_row=None):
    cells = np.arange(nr * nc)
    if empty_row is not None:
        cells = cells[cells // nc != empty_row]
    keys = np.sort(rng.choice(cells, size=nnz, replace=False))
    row, col = keys // nc, keys % nc
    rowptr = np.zeros(nr + 1, dtype=np.int64)
    np.add.at(rowptr, row + 1, 1)
    val = rng.standard_normal(nnz).astype(np.float32).astype(np.float64)
    return np.cumsum(rowptr), col, val


def dense(nr, nc, rowptr, colind, val):
    D = np.zeros((nr, nc))
    for i in range(nr):
        D[i, colind[rowptr[i]:rowptr[i + 1]]] = val[rowptr[i]:rowptr[i + 1]]
    return D


# ----------------------------------------------------------------- syntax


@pytest.mark.parametrize("text,want", [
    ("1 + 2 * 3", 7),
    ("(1 + 2) * 3", 9),
    ("-2 * 3 + 1", -5),
    ("let x = 2 in let y = x * x in y + x", 6),
    ("let x = 2 in (let x = 5 in x) + x", 7),
    ("if 1 = 1 then 4", 4),
    ("if not (1 = 1) then 4 + 0", ref.ZERO),
    ("{3 -> 2.5}(3)", 2.5),
])
def test_expressions(text, want):
    assert ref.evaluate(text, {}) == want


def test_sum_body_extends_to_the_right():
    V = {0: 1.0, 3: 2.0}
    assert ref.evaluate("2 * sum(<i,a> in V) a + 1", {"V": V}) == 2 * ((1 + 1) + (2 + 1))


# ------------------------------------------------------ dictionary semantics


def test_absent_key_reads_zero_and_is_the_identity():
    V = {0: 1.0, 3: 2.0}
    assert ref.evaluate("V(1)", {"V": V}) is ref.ZERO
    assert ref.evaluate("V(1) + 4", {"V": V}) == 4
    assert ref.evaluate("V(1) * 4", {"V": V}) is ref.ZERO
    assert ref.evaluate("{} + V", {"V": V}) == V
    assert ref.evaluate("sum(<i,a> in W) a", {"W": {}}) is ref.ZERO


def test_insertion_adds_values_of_equal_keys():
    V = {0: 1.0, 3: 2.0, 5: 4.0}
    assert ref.evaluate("sum(<i,a> in V) {0 -> a}", {"V": V}) == {0: 7.0}


def test_map_over_values():
    V = {0: 1.0, 3: 2.0}
    assert ref.evaluate("sum(<k,v> in V) {k -> 2 * v}", {"V": V}) == {0: 2.0, 3: 4.0}


def test_scalar_vector_product_is_scaling():
    # Example 2: s * V
    v = np.array([1.0, -2.0, 0.5])
    out = ref.evaluate("s * V", {"s": 3.0, "V": ref.dense_dict(v)})
    np.testing.assert_array_equal(ref.to_array(out, (3,)), 3 * v)


def test_outer_product_of_vectors():
    a, b = np.array([1.0, 2.0]), np.array([3.0, -1.0, 5.0])
    out = ref.evaluate("a * b", {"a": ref.dense_dict(a), "b": ref.dense_dict(b)})
    np.testing.assert_array_equal(ref.to_array(out, (2, 3)), np.outer(a, b))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_dot_product_both_variants(seed):
    # Example 1: iterate either vector; a sparse V1 stores a subset of keys
    rng = np.random.default_rng(seed)
    v1 = rng.standard_normal(9)
    keep = rng.random(9) < 0.5
    v2 = rng.standard_normal(9)
    V1 = {i: float(v1[i]) for i in range(9) if keep[i]}
    env = {"V1": V1, "V2": ref.dense_dict(v2)}
    want = float(np.dot(np.where(keep, v1, 0.0), v2))
    assert ref.evaluate("sum(<i, a> in V1) a * V2(i)", env) == pytest.approx(want, rel=1e-14)
    assert ref.evaluate("sum(<i, a> in V2) V1(i) * a", env) == pytest.approx(want, rel=1e-14)


MATMUL = ("sum(<i,row> in M1) { i -> sum(<j, v1> in row) sum(<k, v2> in M2(j)) "
          "{ k -> v1 * v2 } }")


@pytest.mark.parametrize("seed", [0, 1])
def test_matrix_product(seed):
    # the matrix product of Section 3, with a sparse M1 that has an empty row
    rng = np.random.default_rng(seed)
    rowptr, colind, val = rand_csr(rng, 5, 4, 9, empty_row=2)
    B = rng.standard_normal((4, 3))
    out = ref.evaluate(MATMUL, {"M1": ref.csr_dict(rowptr, colind, val),
                                "M2": ref.dense_dict(B)})
    assert 2 not in out                      # no stored row, no key
    np.testing.assert_allclose(ref.to_array(out, (5, 3)), dense(5, 4, rowptr, colind, val) @ B,
                               rtol=1e-13, atol=1e-14)


# ---------------------------------------------------- against the C oracle


SMVM = "sum(<i,r> in A) sum(<j,a> in r) a * x(j)"
FROB = ("let C = sum(<i,row> in A) { i -> sum(<j,a> in row) sum(<c,b> in B(j)) { c -> a * b } }"
        " in 0.5 * sum(<i,r> in C) sum(<c,v> in r) v * v")
GNN = "sum(<i,r> in A) sum(<j,a> in r) sum(<c,h> in H(j)) a * h * G(i)(c)"
MF = ("let R = sum(<i,r> in A) {i -> sum(<j,a> in r) {j -> a + -1 * sum(<c,u> in U(i)) "
      "u * V(j)(c)}} in sum(<i,r> in R) sum(<j,v> in r) v * v")


def test_losses_agree_with_the_c_oracle(orc):
    rng = np.random.default_rng(4)
    nr, nc, k = 7, 6, 3
    rowptr, colind, val = rand_csr(rng, nr, nc, 15, empty_row=3)
    A = orc.Dok.from_csr(nr, nc, rowptr, colind, val.astype(np.float32))
    Ad = ref.csr_dict(rowptr, colind, val)
    x = rng.standard_normal(nc)
    B, H = rng.standard_normal((nc, k)), rng.standard_normal((nc, k))
    G, U = rng.standard_normal((nr, k)), rng.standard_normal((nr, k))
    V = rng.standard_normal((nc, k))
    dd = ref.dense_dict
    got = ref.value(SMVM, {"A": Ad, "x": dd(x)})
    assert got == pytest.approx(orc.loss_sum_spmv(A, x)[0], rel=1e-12)
    C, Cmag = orc.spmm(A, B, k)
    got = ref.value(FROB, {"A": Ad, "B": dd(B)})
    assert got == pytest.approx(orc.loss_half_sq(C, Cmag)[0], rel=1e-12)
    got = ref.value(GNN, {"A": Ad, "H": dd(H), "G": dd(G)})
    assert got == pytest.approx(orc.loss_bilinear(A, G, H, k)[0], rel=1e-12)
    got = ref.value(MF, {"A": Ad, "U": dd(U), "V": dd(V)})
    assert got == pytest.approx(orc.mf_loss(A, U, V, k)[0], rel=1e-12)


# -------------------------------------------------------------- gradients


def test_dot_product_gradient_is_the_other_vector():
    # Example 1 (cont.): d(V1 . V2)/dV2 = V1 on V2's keys
    v1, v2 = np.array([1.0, 0.0, -2.0, 4.0]), np.array([3.0, 1.0, 2.0, -1.0])
    env = {"V1": {0: 1.0, 2: -2.0, 3: 4.0}, "V2": ref.dense_dict(v2)}
    g = ref.gradient("sum(<i, a> in V1) a * V2(i)", env, "V2")
    assert g == {(0,): 1.0, (1,): 0.0, (2,): -2.0, (3,): 4.0}
    g = ref.gradient("sum(<i, a> in V1) a * V2(i)", env, "V1")
    assert g == {(0,): 3.0, (2,): 2.0, (3,): -1.0}


def test_trace_gradient_is_one_on_the_diagonal():
    # Example 3: d trace(M)/dM is 1 on the stored diagonal keys, 0 elsewhere
    M = {0: {0: 2.0, 2: 1.0}, 1: {0: 5.0}, 2: {2: -1.0, 1: 3.0}}
    g = ref.gradient("sum(<i,r> in M) r(i)", {"M": M}, "M")
    assert g == {(0, 0): 1.0, (0, 2): 0.0, (1, 0): 0.0, (2, 1): 0.0, (2, 2): 1.0}


def test_gradients_closed_forms():
    rng = np.random.default_rng(7)
    nr, nc, k = 6, 5, 3
    rowptr, colind, val = rand_csr(rng, nr, nc, 12, empty_row=1)
    D = dense(nr, nc, rowptr, colind, val)
    mask = dense(nr, nc, rowptr, colind, np.ones_like(val)) > 0
    Ad = ref.csr_dict(rowptr, colind, val)
    x, B = rng.standard_normal(nc), rng.standard_normal((nc, k))
    U, V = rng.standard_normal((nr, k)), rng.standard_normal((nc, k))

    def at_keys(g, shape):
        out = np.full(shape, np.nan)
        for key, v in g.items():
            out[key] = v
        return out

    env = {"A": Ad, "x": ref.dense_dict(x)}
    gA = at_keys(ref.gradient(SMVM, env, "A"), (nr, nc))
    np.testing.assert_allclose(gA[mask], np.broadcast_to(x, (nr, nc))[mask], rtol=1e-14)
    np.testing.assert_allclose(at_keys(ref.gradient(SMVM, env, "x"), (nc,)), D.sum(0),
                               rtol=1e-13, atol=1e-15)
    env = {"A": Ad, "B": ref.dense_dict(B)}
    C = D @ B
    np.testing.assert_allclose(at_keys(ref.gradient(FROB, env, "B"), (nc, k)), D.T @ C,
                               rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(at_keys(ref.gradient(FROB, env, "A"), (nr, nc))[mask],
                               (C @ B.T)[mask], rtol=1e-12, atol=1e-13)
    env = {"A": Ad, "U": ref.dense_dict(U), "V": ref.dense_dict(V)}
    R = np.where(mask, D - U @ V.T, 0.0)
    np.testing.assert_allclose(at_keys(ref.gradient(MF, env, "U"), (nr, k)), -2 * R @ V,
                               rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(at_keys(ref.gradient(MF, env, "V"), (nc, k)), -2 * R.T @ U,
                               rtol=1e-12, atol=1e-13)


NONLINEAR = [
    "sum(<i,a> in V) exp(a) * a",
    "sum(<i,a> in V) sin(a * W(i)) + W(i) * W(i) * a",
    "let s = sum(<i,a> in V) a * a in s * s + sum(<j,b> in W) cos(b) * s",
    "sum(<i,r> in M) sum(<j,a> in r) let t = a * V(j) in sqrt(t * t + 1)",
]


@pytest.mark.parametrize("text", NONLINEAR)
def test_gradients_match_central_differences(text):
    rng = np.random.default_rng(11)
    v, w = rng.standard_normal(4), rng.standard_normal(4)
    M = {0: {1: 0.5, 3: -1.2}, 2: {0: 2.0}, 3: {2: 0.7, 3: 0.1}}
    env = {"V": ref.dense_dict(v), "W": ref.dense_dict(w), "M": M}
    h = 1e-5
    for wrt in ("V", "W", "M"):
        g = ref.gradient(text, env, wrt)
        for key, got in g.items():
            def shifted(dx):
                e2 = dict(env)
                src = env[wrt]
                e2[wrt] = ref._replace_leaves(src, lambda kk, val: val + dx if kk == key else val)
                return ref.value(text, e2)

            fd = (shifted(h) - shifted(-h)) / (2 * h)
            assert got == pytest.approx(fd, rel=1e-6, abs=1e-8), (wrt, key)


# ----------------------------------- gradient API, evaluated literally


TENSORIZED_PROGRAMS = [
    "sum(<i, a> in V1) a * V2(i)",
    "sum(<i, a> in V2) V1(i) * a",
    "sum(<i,r> in M) r(i)",
    SMVM, FROB, GNN, MF,
    "sum(<i,r> in A) sum(<j,a> in r) let d = a + -1 * sum(<c,u> in U(i)) u * V(j)(c) in d * d",
    "sum(<i,a> in V1) exp(a) * a + sin(V2(i)) * a * a",
]


def tiny_env(rng):
    rowptr, colind, val = rand_csr(rng, 5, 4, 9, empty_row=1)
    Mp, Mc, Mv = rand_csr(rng, 4, 4, 7)
    k = 3
    dd = ref.dense_dict
    return {
        "A": ref.csr_dict(rowptr, colind, val), "M": ref.csr_dict(Mp, Mc, Mv),
        "V1": {0: 0.7, 2: -1.1, 3: 0.4}, "V2": dd(rng.standard_normal(4)),
        "x": dd(rng.standard_normal(4)), "B": dd(rng.standard_normal((4, k))),
        "H": dd(rng.standard_normal((4, k))), "G": dd(rng.standard_normal((5, k))),
        "U": dd(rng.standard_normal((5, k))), "V": dd(rng.standard_normal((4, k))),
    }, (rowptr, colind, val)


@pytest.mark.parametrize("text", TENSORIZED_PROGRAMS)
def test_tensorized_gradient_equals_scalar_forward_mode(text):
    # two independent differentiations: the tensorized rules applied to the
    # program (one evaluation) and dual numbers (one evaluation per key)
    env, _ = tiny_env(np.random.default_rng(3))
    used = {n for n in env if n in text.replace("(", " ").replace(")", " ").split()}
    env = {n: env[n] for n in used}
    for wrt in sorted(used):
        a = ref.gradient_tensorized(text, env, wrt)
        b = ref.gradient(text, env, wrt)
        assert a.keys() == b.keys()
        for key in a:
            assert a[key] == pytest.approx(b[key], rel=1e-12, abs=1e-13), (wrt, key)


def test_tensorized_examples_1_and_3():
    env = {"V1": {0: 1.0, 2: -2.0, 3: 4.0}, "V2": ref.dense_dict([3.0, 1.0, 2.0, -1.0])}
    assert ref.gradient_tensorized("sum(<i, a> in V1) a * V2(i)", env, "V2") == \
        {(0,): 1.0, (1,): 0.0, (2,): -2.0, (3,): 4.0}
    M = {0: {0: 2.0, 2: 1.0}, 1: {0: 5.0}, 2: {2: -1.0, 1: 3.0}}
    assert ref.gradient_tensorized("sum(<i,r> in M) r(i)", {"M": M}, "M") == \
        {(0, 0): 1.0, (0, 2): 0.0, (1, 0): 0.0, (2, 1): 0.0, (2, 2): 1.0}


def test_tensorized_gradients_equal_the_c_oracle(orc):
    # the interpreter's `gradient e x` against the fp64 C oracle's
    # hand-derived gradients: same keys (the stored pattern), same values
    env, (rowptr, colind, val) = tiny_env(np.random.default_rng(9))
    nr, nc, k = 5, 4, 3
    A = orc.Dok.from_csr(nr, nc, rowptr, colind, val.astype(np.float32))
    rows = np.repeat(np.arange(nr, dtype=np.int32), np.diff(rowptr)).astype(np.int32)
    cols = np.asarray(colind, dtype=np.int32)
    arr = {n: ref.to_array(env[n], (4,) if n == "x" else ((5 if n in "GU" else 4), k))
           for n in ("x", "B", "H", "G", "U", "V")}

    def on_pattern(g):
        return np.array([g[(int(i), int(j))] for i, j in zip(rows, cols)])

    def dense_grad(g, shape):
        out = np.zeros(shape)
        for key, v in g.items():
            out[key] = v
        return out

    e = {"A": env["A"], "x": env["x"]}
    ref_dA, _ = orc.sddmm(A, None, arr["x"].reshape(-1, 1), 1, rows, cols)
    np.testing.assert_allclose(on_pattern(ref.gradient_tensorized(SMVM, e, "A")), ref_dA,
                               rtol=1e-12, atol=1e-13)
    ref_dx, _ = orc.spmm_t(A, None, 1)
    np.testing.assert_allclose(dense_grad(ref.gradient_tensorized(SMVM, e, "x"), (nc,)),
                               ref_dx[:, 0], rtol=1e-12, atol=1e-13)
    e = {"A": env["A"], "B": env["B"]}
    C, Cm = orc.spmm(A, arr["B"], k)
    ref_dA, _ = orc.sddmm(A, C, arr["B"], k, rows, cols, Xmag=Cm)
    np.testing.assert_allclose(on_pattern(ref.gradient_tensorized(FROB, e, "A")), ref_dA,
                               rtol=1e-11, atol=1e-12)
    ref_dB, _ = orc.spmm_t(A, C, k, Gmag=Cm)
    np.testing.assert_allclose(dense_grad(ref.gradient_tensorized(FROB, e, "B"), (nc, k)),
                               ref_dB, rtol=1e-11, atol=1e-12)
    e = {"A": env["A"], "U": env["U"], "V": env["V"]}
    for mode, (w, shape) in enumerate([("U", (nr, k)), ("V", (nc, k))]):
        g, _ = orc.mf_grad(A, arr["U"], arr["V"], k, mode)
        np.testing.assert_allclose(dense_grad(ref.gradient_tensorized(MF, e, w), shape), g,
                                   rtol=1e-11, atol=1e-12)
    e = {"A": env["A"], "H": env["H"], "G": env["G"]}
    ref_dA, _ = orc.sddmm(A, arr["G"], arr["H"], k, rows, cols)
    np.testing.assert_allclose(on_pattern(ref.gradient_tensorized(GNN, e, "A")), ref_dA,
                               rtol=1e-11, atol=1e-12)
    ref_dH, _ = orc.spmm_t(A, arr["G"], k)
    np.testing.assert_allclose(dense_grad(ref.gradient_tensorized(GNN, e, "H"), (nc, k)),
                               ref_dH, rtol=1e-11, atol=1e-12)


# ------------------------- Jacobians of tensor-valued programs (vector kernels)

VVA = "sum(<i,v> in V1) {i -> v} + sum(<i,v> in V2) {i -> v}"
VSM = "sum(<i,v> in V) {i -> v * s * s}"
MATVEC = "sum(<i,r> in M) {i -> sum(<j,a> in r) a * x(j)}"


def sparse_vector(rng, n, nnz):
    keys = np.sort(rng.choice(n, size=nnz, replace=False))
    return {int(k): float(v) for k, v in zip(keys, rng.standard_normal(nnz))}


def both_jacobians(text, env, wrt):
    j1 = ref.jacobian(text, env, wrt)
    j2 = ref.jacobian_tensorized(text, env, wrt)
    assert set(j1) == {k for k, v in j2.items() if v != 0.0}
    for key, v in j1.items():
        assert j2[key] == pytest.approx(v, rel=1e-12, abs=1e-14), key
    return j1


@pytest.mark.parametrize("seed", range(3))
def test_vector_addition_jacobian_is_the_identity_on_the_stored_keys(seed):
    # the VVA kernel of the evaluation (Section 7.1): d(V1 + V2)/dV1 is 1 at
    # (k, k) for every stored key k of V1 and nothing else, whatever V2 stores
    rng = np.random.default_rng(seed)
    env = {"V1": sparse_vector(rng, 40, 9), "V2": sparse_vector(rng, 40, 11)}
    assert both_jacobians(VVA, env, "V1") == {(k, k): 1.0 for k in env["V1"]}


@pytest.mark.parametrize("seed", range(3))
def test_vector_scalar_product_jacobian_is_2sV(seed):
    # the VSM kernel of the evaluation: f(i) = V(i) s s, df/ds = 2 s V on V's keys
    rng = np.random.default_rng(10 + seed)
    s = float(rng.standard_normal())
    env = {"V": sparse_vector(rng, 50, 13), "s": s}
    J = both_jacobians(VSM, env, "s")
    assert J == pytest.approx({(k,): 2 * s * v for k, v in env["V"].items() if v != 0.0})
    # and with respect to V: the diagonal s^2 on V's keys
    J = both_jacobians(VSM, env, "V")
    assert J == pytest.approx({(k, k): s * s for k in env["V"]})


def test_matrix_vector_product_jacobian_is_the_matrix():
    rng = np.random.default_rng(20)
    M = {i: sparse_vector(rng, 7, int(rng.integers(1, 5))) for i in range(6) if i != 3}
    env = {"M": M, "x": ref.dense_dict(rng.standard_normal(7))}
    J = both_jacobians(MATVEC, env, "x")
    assert J == pytest.approx({(i, j): a for i, r in M.items() for j, a in r.items()})


def test_jacobian_of_a_real_valued_program_is_its_gradient():
    rng = np.random.default_rng(21)
    M = {i: sparse_vector(rng, 5, 3) for i in range(5)}
    for i in (0, 2):
        M[i][i] = float(rng.standard_normal())  # some stored diagonal keys
    env = {"M": M}
    trace = "sum(<i,r> in M) r(i)"
    assert both_jacobians(trace, env, "M") == {(i, i): 1.0 for i in M if i in M[i]}
    g = ref.gradient(trace, env, "M")
    assert {k: v for k, v in g.items() if v != 0.0} == ref.jacobian(trace, env, "M")


def test_jacobian_matches_central_differences():
    # a nonlinear vector program: each column of the Jacobian against central
    # differences of the output dictionary
    text = "sum(<i,v> in V) {i -> sin(v * W(i)) + v * v * W(i)}"
    rng = np.random.default_rng(22)
    env = {"V": sparse_vector(rng, 12, 6), "W": ref.dense_dict(rng.standard_normal(12))}
    h = 1e-5
    for wrt in ("V", "W"):
        J = both_jacobians(text, env, wrt)
        for key, _ in ref.leaves(env[wrt]):
            def shifted(dx):
                e2 = dict(env)
                e2[wrt] = ref._replace_leaves(env[wrt],
                                              lambda kk, val: val + dx if kk == key else val)
                return dict(ref.leaves(ref.value(text, e2)))

            hi, lo = shifted(h), shifted(-h)
            for out in hi:
                fd = (hi[out] - lo[out]) / (2 * h)
                assert J.get(out + key, 0.0) == pytest.approx(fd, rel=1e-6, abs=1e-8), (wrt, key)


# ------------------------------------- batched tangents (J V, Section 4.2)


def _batch_tangent(rng, x, m):
    """Random tangents of a dictionary x: its key paths, then the batch key."""
    out = {}
    for path, _ in ref.leaves(x):
        leaf = {t: float(rng.standard_normal()) for t in range(m)}
        d = out
        for k in path[:-1]:
            d = d.setdefault(k, {})
        if path:
            d[path[-1]] = leaf
        else:
            out = leaf
    return out


def test_batched_tangents_match_central_differences():
    # the tangent along each direction of the batch against central
    # differences of the output dictionary along that direction
    text = "sum(<i,v> in V) {i -> sin(v * W(i)) + v * v * W(i)}"
    rng = np.random.default_rng(60)
    env = {"V": sparse_vector(rng, 12, 6), "W": ref.dense_dict(rng.standard_normal(12))}
    m, h = 3, 1e-5
    tans = {"V": _batch_tangent(rng, env["V"], m), "W": _batch_tangent(rng, env["W"], m)}
    got = ref.jvp_tensorized(text, env, tans)
    for t in range(m):
        def moved(eps):
            e2 = {n: ref._replace_leaves(env[n], lambda key, v, n=n: v + eps * _at(tans[n], key)[t])
                  for n in env}
            return dict(ref.leaves(ref.value(text, e2)))

        hi, lo = moved(h), moved(-h)
        for out in hi:
            fd = (hi[out] - lo[out]) / (2 * h)
            assert got.get(out + (t,), 0.0) == pytest.approx(fd, rel=1e-6, abs=1e-8), (out, t)


def _at(d, key):
    for k in key:
        d = d[k]
    return d


def test_batched_tangents_equal_the_one_key_jacobian_times_V():
    # J V from the per-key forward mode (one evaluation per stored key of
    # each input, then contracted with the batch) for a matrix program
    rng = np.random.default_rng(61)
    M = {i: sparse_vector(rng, 7, int(rng.integers(1, 5))) for i in range(6) if i != 2}
    env = {"M": M, "x": ref.dense_dict(rng.standard_normal(7)), "s": 0.75}
    text = "sum(<i,r> in M) {i -> sum(<j,a> in r) {j -> a * a * x(j) * s}}"
    m = 4
    tans = {n: _batch_tangent(rng, env[n], m) for n in ("M", "x", "s")}
    got = ref.jvp_tensorized(text, env, tans)
    want = {}
    for n in ("M", "x", "s"):
        for key, v in ref.jacobian(text, env, n).items():
            # the output keys (i, j), then n's key (none for the real s)
            for t in range(m):
                out = key[:2] + (t,)
                want[out] = want.get(out, 0.0) + v * _at(tans[n], key[2:])[t]
    assert set(want) == set(got)
    for key, v in want.items():
        assert got.get(key, 0.0) == pytest.approx(v, rel=1e-12, abs=1e-14), key


def test_batched_tangents_are_linear_in_the_tangents():
    rng = np.random.default_rng(62)
    env = {"V": sparse_vector(rng, 20, 7), "s": -1.3}
    text = "sum(<i,v> in V) {i -> v * s * s}"
    a, b = _batch_tangent(rng, env["V"], 2), _batch_tangent(rng, env["V"], 2)
    ab = {k: {t: a[k][t] + 2.0 * b[k][t] for t in range(2)} for k in a}
    ga, gb = ref.jvp_tensorized(text, env, {"V": a}), ref.jvp_tensorized(text, env, {"V": b})
    gab = ref.jvp_tensorized(text, env, {"V": ab})
    for key in gab:
        assert gab[key] == pytest.approx(ga[key] + 2.0 * gb[key], rel=1e-12, abs=1e-14)
