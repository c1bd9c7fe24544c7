"""Hot-path entry points captured in a HIP graph.

A hot-path call issues kernel launches only (no copy, fill, allocation or
host synchronisation), so one call can be captured and replayed.  Each case
runs the call eagerly, captures it once, then replays the graph three times
with unrelated eager work and a synchronisation between replays and with
every output overwritten by NaN before each replay; every replay must equal
the eager result bit for bit (the calls are deterministic and write their
outputs in full).
"""
import numpy as np
import pytest
import torch

from test_gpu_parity import edge_pattern

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def nsd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import nsd as m
    return m


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def out(*shape, dtype=torch.float32):
    return torch.full(shape, float("nan"), dtype=dtype, device="cuda")


def csr(k=None):
    from paper_2303_07030_amd.operand import DeviceCsr
    nrows, ncols, rowptr, colind, val = edge_pattern(31)
    return DeviceCsr(nrows, ncols, rowptr, colind, val, k_hint=k)


def rand(*shape, seed=0, scale=1.0):
    g = np.random.default_rng(seed)
    return dev((scale * g.standard_normal(shape)).astype(np.float32))


def case_frob(nsd, k=64):
    A = csr(k)
    B, ws = rand(A.ncols, k), A.workspace(k)
    o = [out(A.nrows, k), out(1, dtype=torch.float64), out(A.nnz), out(A.ncols, k)]
    return (lambda: nsd.nsd_loss_frob_spmm(A.desc, A.csc, B, k, 1.0, o[0], o[1], o[2], o[3], ws)), o


def case_bilinear(nsd, k=16):
    A = csr(k)
    H, G, ws = rand(A.ncols, k, seed=1), rand(A.nrows, k, seed=2), A.workspace(k)
    o = [out(1, dtype=torch.float64), out(A.nnz), out(A.ncols, k)]
    return (lambda: nsd.nsd_loss_bilinear(A.desc, A.csc, H, G, k, 1.0, *o, ws)), o


def case_mf(nsd, k=32):
    A = csr(k)
    valT = A.values_in_csc_order()
    U, V = rand(A.nrows, k, seed=3, scale=0.3), rand(A.ncols, k, seed=4, scale=0.3)
    ws = A.workspace(k)
    o = [out(1, dtype=torch.float64), out(A.nrows, k), out(A.ncols, k)]
    return (lambda: nsd.nsd_loss_mf(A.desc, A.csc, valT, U, V, k, 1.0, *o, ws)), o


def case_sum_spmv(nsd):
    A = csr(1)
    x, ws = rand(A.ncols, seed=5), A.workspace(1)
    o = [out(1, dtype=torch.float64), out(A.nnz), out(A.ncols)]
    return (lambda: nsd.nsd_loss_sum_spmv(A.desc, A.csc, x, 1.0, *o, ws)), o


def case_spmm_t(nsd, k=64):
    A = csr(k)
    G, ws = rand(A.nrows, k, seed=6), A.workspace(k)
    o = [out(A.ncols, k)]
    return (lambda: nsd.nsd_spmm_t(A.desc, A.csc, G, k, 1.0, o[0], ws)), o


def case_jvp(nsd, k=64):
    A = csr(k)
    dval, B, dB = rand(A.nnz, seed=7), rand(A.ncols, k, seed=8), rand(A.ncols, k, seed=9)
    ws = A.workspace(2 * k)
    o = [out(A.nrows, k), out(A.nrows, k)]
    return (lambda: nsd.nsd_spmm_jvp(A.desc, dval, B, dB, k, o[0], o[1], ws)), o


def case_cp(nsd):
    from paper_2303_07030_amd import synth
    from paper_2303_07030_amd.operand import DeviceCoo3
    d = synth.make("cp", "small")
    R = d["rank"]
    X = DeviceCoo3(d["dims"], d["i"], d["j"], d["k"], d["val"], rank_hint=R)
    F = [dev(d[f]) for f in ("F1", "F2", "F3")]
    ws = X.workspace(R)
    o = [out(1, dtype=torch.float64), out(X.nnz)] + [out(X.dims[m], R) for m in range(3)]
    return (lambda: nsd.nsd_loss_cp(X.desc, *F, R, 1.0, *o, ws)), o


def case_cpn(nsd):
    from paper_2303_07030_amd.operand import DeviceCooN
    rng = np.random.default_rng(10)
    dims, nnz, R = (40, 30, 20, 25), 20_000, 16
    flat = rng.choice(int(np.prod(dims)), size=nnz, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(flat, dims)]
    X = DeviceCooN(dims, coords, rng.standard_normal(nnz).astype(np.float32), rank_hint=R)
    F = [rand(n, R, seed=11 + m, scale=0.5) for m, n in enumerate(dims)]
    ws = X.workspace(R)
    o = [out(1, dtype=torch.float64), out(nnz)] + [out(n, R) for n in dims]
    return (lambda: nsd.nsd_loss_cpn(X.desc, F, R, 1.0, o[0], o[1], o[2:], ws)), o


def case_bilinear_moves(nsd, k=64):
    # the bilinear layer with the two-pass permutation moves (a pattern
    # given the CSC's perm plans): two moves around the column pass
    from paper_2303_07030_amd.operand import DeviceCsr
    nrows, ncols, rowptr, colind, val = edge_pattern(32)
    A = DeviceCsr(nrows, ncols, rowptr, colind, val, k_hint=k, perm_plans=True)
    H, G, ws = rand(A.ncols, k, seed=12), rand(A.nrows, k, seed=13), A.workspace(k)
    o = [out(1, dtype=torch.float64), out(A.nnz), out(A.ncols, k)]
    return (lambda: nsd.nsd_loss_bilinear(A.desc, A.csc, H, G, k, 1.0, *o, ws)), o


def case_bilinear_wide(nsd, k=300):
    # a width beyond a fused slot: SDDMM and the gather-reduce
    A = csr(k)
    H, G, ws = rand(A.ncols, k, seed=14), rand(A.nrows, k, seed=15), A.workspace(k)
    o = [out(1, dtype=torch.float64), out(A.nnz), out(A.ncols, k)]
    return (lambda: nsd.nsd_loss_bilinear(A.desc, A.csc, H, G, k, 1.0, *o, ws)), o


def case_mf_wide(nsd, k=300):
    # the factorisation beyond a fused slot: residual once, two gather-reduces
    A = csr(k)
    U, V = rand(A.nrows, k, seed=16, scale=0.1), rand(A.ncols, k, seed=17, scale=0.1)
    ws = A.workspace(k)
    o = [out(1, dtype=torch.float64), out(A.nrows, k), out(A.ncols, k)]
    return (lambda: nsd.nsd_loss_mf(A.desc, A.csc, None, U, V, k, 1.0, *o, ws)), o


def case_jvp_batch(nsd, k=64, m=5):
    A = csr(k)
    dval, B = rand(m, A.nnz, seed=18), rand(A.ncols, k, seed=19)
    dB = rand(m, A.ncols, k, seed=20)
    ws = torch.empty(nsd.nsd_spmm_jvp_batch_workspace_size(A.desc, k), dtype=torch.uint8,
                     device="cuda")
    o = [out(A.nrows, k), out(m, A.nrows, k)]
    return (lambda: nsd.nsd_spmm_jvp_batch(A.desc, m, dval, B, dB, k, o[0], o[1], ws)), o


def case_scale(nsd, n=100_000):
    g = np.random.default_rng(21)
    x1, x2 = rand(n, seed=22), rand(3 * n, seed=23)
    idx = dev(g.integers(0, 3 * n, n).astype(np.int32))
    s1 = torch.tensor([1.5], dtype=torch.float64, device="cuda")
    o = [out(n)]
    return (lambda: nsd.nsd_scale(n, 2.0, s1, None, x1, x2, idx, 0.0, o[0])), o


CASES = {
    "frob": case_frob, "bilinear": case_bilinear, "mf": case_mf, "sum_spmv": case_sum_spmv,
    "spmm_t": case_spmm_t, "jvp": case_jvp, "cp": case_cp, "cpn": case_cpn,
    "bilinear_moves": case_bilinear_moves, "bilinear_wide": case_bilinear_wide,
    "mf_wide": case_mf_wide, "jvp_batch": case_jvp_batch, "scale": case_scale,
}


@pytest.mark.parametrize("name", list(CASES))
def test_graph_replays_equal_eager(nsd, name):
    step, outs = CASES[name](nsd)
    torch.cuda.synchronize()
    step()
    torch.cuda.synchronize()
    want = [t.cpu().numpy().copy() for t in outs]
    for w in want:
        assert not np.isnan(w).any()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # the call once on the capturing stream
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    other = torch.randn(512, 512, device="cuda")
    for r in range(3):
        for t in outs:
            t.fill_(float("nan"))
        other = other @ other.T / 512.0   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (t, w) in enumerate(zip(outs, want)):
            got = t.cpu().numpy()
            assert np.array_equal(got, w), f"{name}: replay {r}, output {i}"
