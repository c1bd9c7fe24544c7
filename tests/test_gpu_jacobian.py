"""Jacobians of the vector kernels (VVA, VSM) and the trace gradient through
the library, against the oracle's Jacobians of the same programs (one-key
forward mode and the literal gradient API).  Indices and the constant
Jacobians are bit-exact; scaled values within the parity tolerance."""
import numpy as np
import pytest
import torch

from helpers import assert_mag_close
from oracle import sdql as ref

pytestmark = pytest.mark.gpu

VVA = "sum(<i,v> in V1) {i -> v} + sum(<i,v> in V2) {i -> v}"
VSM = "sum(<i,v> in V) {i -> v * s * s}"
TRACE = "sum(<i,r> in M) r(i)"


@pytest.fixture(scope="module")
def J():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import jacobian
    return jacobian


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def sparse_vector(rng, n, nnz):
    keys = np.sort(rng.choice(n, size=nnz, replace=False)).astype(np.int32)
    return keys, rng.standard_normal(nnz).astype(np.float32)


@pytest.mark.parametrize("n,nnz", [(1, 1), (300, 37), (5000, 700)])
def test_vva_jacobian_is_the_identity_on_v1s_keys(J, n, nnz):
    rng = np.random.default_rng(n)
    k1, v1 = sparse_vector(rng, n, nnz)
    k2, v2 = sparse_vector(rng, n, max(1, nnz // 2))
    A = J.vva_jacobian(n, torch.from_numpy(k1).cuda())
    env = {"V1": dict(zip(k1.tolist(), v1.astype(np.float64).tolist())),
           "V2": dict(zip(k2.tolist(), v2.astype(np.float64).tolist()))}
    # the literal gradient API: one evaluation (the one-key forward mode it
    # is pinned against is quadratic in the keys)
    want = ref.jacobian_tensorized(VVA, env, "V1")
    rowptr, colind, val = host(A.rowptr), host(A.colind), host(A.val)
    rows = np.repeat(np.arange(n), np.diff(rowptr))
    got = {(int(r), int(c)): float(v) for r, c, v in zip(rows, colind, val)}
    assert got == want


@pytest.mark.parametrize("s", [0.0, -1.25, 3.0])
def test_vsm_jacobians(J, s):
    rng = np.random.default_rng(7)
    keys, val = sparse_vector(rng, 2000, 300)
    env = {"V": dict(zip(keys.tolist(), val.astype(np.float64).tolist())), "s": s}
    env_abs = {"V": {k: abs(v) for k, v in env["V"].items()}, "s": abs(s)}
    out = torch.full((len(keys),), np.nan, dtype=torch.float32, device="cuda")
    J.vsm_jacobian_s(torch.from_numpy(val).cuda(), s, out)
    want, mag = ref.jacobian_tensorized(VSM, env, "s"), ref.jacobian_tensorized(VSM, env_abs, "s")
    assert_mag_close(host(out), np.array([want.get((k,), 0.0) for k in keys.tolist()]),
                     np.array([mag.get((k,), 0.0) for k in keys.tolist()]), what="df/ds")
    J.vsm_jacobian_v(len(keys), s, out)
    want = ref.jacobian(VSM, env, "V")
    assert np.array_equal(host(out), np.array([want.get((k, k), 0.0) for k in keys.tolist()],
                                              dtype=np.float32))


def test_trace_value_and_gradient_through_the_front_end(J):
    from paper_2303_07030_amd import sdql as S
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
