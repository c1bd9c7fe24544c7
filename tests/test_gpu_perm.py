"""The two-pass value permutation (nsd_perm_plan_build / nsd_permute_f32)
against its definition, dst[q] = src[perm[q]] (and the inverse form),
bit for bit; and the bilinear layer, the SpMM VJP and the Frobenius loss
through a CSC that carries the two-pass forms of its permutation against
the same calls without them."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def nsd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import nsd as m
    return m


def run_perm(nsd, perm, src, inverse):
    from paper_2303_07030_amd.operand import build_perm_plan
    n = len(perm)
    p = torch.from_numpy(perm.astype(np.int32)).cuda()
    plan = build_perm_plan(n, p, inverse, "cuda")
    s = torch.from_numpy(src).cuda()
    d = torch.full((max(n, 1),), np.nan, dtype=torch.float32, device="cuda")
    staging = torch.empty(max(n, 1), dtype=torch.float32, device="cuda")
    nsd.nsd_permute_f32(plan, s, d, staging)
    torch.cuda.synchronize()
    return d.cpu().numpy()[:n]


@pytest.mark.parametrize("n", [0, 1, 5, 32767, 32768, 32769, 100_000, 1_000_003])
@pytest.mark.parametrize("inverse", [0, 1])
def test_permute_matches_definition(nsd, n, inverse):
    rng = np.random.default_rng(n + inverse)
    perm = rng.permutation(n)
    src = rng.standard_normal(n).astype(np.float32)
    src[::7] = -0.0  # signed zeros and NaNs travel bit for bit
    if n > 3:
        src[3] = np.nan
    got = run_perm(nsd, perm, src, inverse)
    want = np.empty_like(src)
    if inverse:
        want[perm] = src
    else:
        want = src[perm]
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_permute_csr_to_csc_and_back(nsd):
    """The CSC permutation of a power-law pattern (long rows whose entries
    spread over all columns) both ways: values into CSC order and back."""
    from test_gpu_parity import make_csr
    from paper_2303_07030_amd.operand import DeviceCsr
    rng = np.random.default_rng(3)
    nrows, ncols = 5000, 80_000
    lengths = np.minimum((20 * rng.pareto(1.05, nrows)).astype(np.int64), ncols)
    rowptr, colind, val = make_csr(rng, nrows, ncols, lengths)
    A = DeviceCsr(nrows, ncols, rowptr, colind, val, perm_plans=True)
    perm = A.perm.cpu().numpy()
    got = run_perm(nsd, perm, val, 0)
    assert np.array_equal(got.view(np.uint32), val[perm].view(np.uint32))
    back = run_perm(nsd, perm, got, 1)
    assert np.array_equal(back.view(np.uint32), val.view(np.uint32))


def test_perm_plan_rejects_non_permutations(nsd):
    from paper_2303_07030_amd.operand import build_perm_plan
    for bad in ([0, 1, 1, 3], [0, 1, 2, 4], [-1, 0, 1, 2]):
        with pytest.raises(nsd.NsdError) as e:
            build_perm_plan(4, torch.tensor(bad, dtype=torch.int32, device="cuda"), 0, "cuda")
        assert e.value.status == nsd.NSD_ERR_BAD_FORMAT


@pytest.mark.parametrize("k", [256, 64, 300])
def test_bilinear_with_perm_plans_equals_without(nsd, orc, k):
    """Values moved to CSC order and the sparse gradient moved back by the
    two-pass permutations give the bits of the pass that reads and writes
    through perm."""
    from test_gpu_parity import make_csr
    from paper_2303_07030_amd.operand import DeviceCsr
    rng = np.random.default_rng(k)
    nrows, ncols = 3000, 2500
    lengths = np.minimum((25 * rng.pareto(1.05, nrows)).astype(np.int64), ncols)
    lengths[rng.random(nrows) < 0.1] = 0
    rowptr, colind, val = make_csr(rng, nrows, ncols, lengths, hot_col=7)
    H = torch.from_numpy(rng.standard_normal((ncols, k)).astype(np.float32)).cuda()
    G = torch.from_numpy(rng.standard_normal((nrows, k)).astype(np.float32)).cuda()
    out = []
    for plans in (False, True):
        A = DeviceCsr(nrows, ncols, rowptr, colind, val, k_hint=k, perm_plans=plans)
        assert (A.csc.to_csc.n == A.nnz) == plans
        loss = torch.empty(1, dtype=torch.float64, device="cuda")
        dA = torch.full((A.nnz,), np.nan, dtype=torch.float32, device="cuda")
        dH = torch.full((ncols, k), np.nan, dtype=torch.float32, device="cuda")
        nsd.nsd_loss_bilinear(A.desc, A.csc, H, G, k, 0.75, loss, dA, dH, A.workspace(k))
        torch.cuda.synchronize()
        out.append([t.cpu().numpy() for t in (loss, dA, dH)])
    for a, b in zip(*out):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
    from helpers import assert_mag_close
    D = orc.Dok.from_csr(nrows, ncols, rowptr, colind, val)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    ref, mag = orc.sddmm(D, G.cpu().numpy(), H.cpu().numpy(), k, rows, colind, alpha=0.75)
    assert_mag_close(out[1][1], ref, mag, what="dA")


@pytest.mark.parametrize("k", [1, 64])
def test_vjp_and_frob_with_perm_plans_equal_without(nsd, k):
    """The SpMM VJP and the Frobenius loss take the same moves around their
    column pass: the same bits as through perm."""
    from test_gpu_parity import make_csr
    from paper_2303_07030_amd.operand import DeviceCsr
    rng = np.random.default_rng(100 + k)
    nrows, ncols = 2500, 3000
    lengths = np.minimum((25 * rng.pareto(1.05, nrows)).astype(np.int64), ncols)
    lengths[rng.random(nrows) < 0.1] = 0
    rowptr, colind, val = make_csr(rng, nrows, ncols, lengths, hot_col=3)
    X = torch.from_numpy(rng.standard_normal((ncols, k)).astype(np.float32)).cuda()
    G = torch.from_numpy(rng.standard_normal((nrows, k)).astype(np.float32)).cuda()
    out = []
    for plans in (False, True):
        A = DeviceCsr(nrows, ncols, rowptr, colind, val, k_hint=k, perm_plans=plans)
        assert (A.csc.to_csc.n == A.nnz) == plans
        dA = torch.full((A.nnz,), np.nan, dtype=torch.float32, device="cuda")
        dX = torch.full((ncols, k), np.nan, dtype=torch.float32, device="cuda")
        nsd.nsd_spmm_vjp(A.desc, A.csc, X, G, k, dA, dX, A.workspace(k))
        loss = torch.empty(1, dtype=torch.float64, device="cuda")
        C = torch.full((nrows, k), np.nan, dtype=torch.float32, device="cuda")
        fA = torch.full((A.nnz,), np.nan, dtype=torch.float32, device="cuda")
        fB = torch.full((ncols, k), np.nan, dtype=torch.float32, device="cuda")
        nsd.nsd_loss_frob_spmm(A.desc, A.csc, X, k, 1.0, C, loss, fA, fB, A.workspace(k))
        torch.cuda.synchronize()
        out.append([t.cpu().numpy() for t in (dA, dX, loss, C, fA, fB)])
    for a, b in zip(*out):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
    assert not np.isnan(out[1][0]).any() and not np.isnan(out[1][4]).any()

