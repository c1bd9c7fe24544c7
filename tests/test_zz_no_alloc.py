"""The bilinear layer's entry point that allocates nothing (its scratch is a
static device array) against the entry point with a workspace: same results
bit for bit and within the parity bar of the oracle, on two calls in a row,
the second on a smaller operand; an operand needing more scratch than the
array holds is refused before any launch."""
import numpy as np
import pytest
import torch

from helpers import assert_mag_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def nsd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2303_07030_amd import nsd as m
    return m


def case(seed, nrows, ncols, k):
    from test_gpu_parity import make_csr
    rng = np.random.default_rng(seed)
    lengths = np.minimum((30 * rng.pareto(1.1, nrows)).astype(np.int64), ncols)
    lengths[rng.random(nrows) < 0.1] = 0
    rowptr, colind, val = make_csr(rng, nrows, ncols, lengths, hot_col=3)
    H = rng.standard_normal((ncols, k)).astype(np.float32)
    G = rng.standard_normal((nrows, k)).astype(np.float32)
    return rowptr, colind, val, H, G


def run_both(nsd, nrows, ncols, rowptr, colind, val, H, G, k, item_len=None):
    from paper_2303_07030_amd.operand import DeviceCsr
    A = DeviceCsr(nrows, ncols, rowptr, colind, val, k_hint=k, item_len=item_len)
    Hd, Gd = torch.from_numpy(H).cuda(), torch.from_numpy(G).cuda()
    out = []
    for noalloc in (False, True):
        loss = torch.full((1,), np.nan, dtype=torch.float64, device="cuda")
        dA = torch.full((max(A.nnz, 1),), np.nan, dtype=torch.float32, device="cuda")
        dH = torch.full((ncols, k), np.nan, dtype=torch.float32, device="cuda")
        if noalloc:
            nsd.nsd_loss_bilinear_noalloc(A.desc, A.csc, Hd, Gd, k, 0.5, loss, dA, dH)
        else:
            nsd.nsd_loss_bilinear(A.desc, A.csc, Hd, Gd, k, 0.5, loss, dA, dH, A.workspace(k))
        torch.cuda.synchronize()
        out.append((loss.cpu().numpy(), dA.cpu().numpy()[: A.nnz], dH.cpu().numpy()))
    return out


@pytest.mark.parametrize("k", [256, 64, 300, 13])
def test_noalloc_equals_workspace_entry_point(nsd, orc, k):
    # the first call on a larger operand (long columns: chunk partials in the
    # scratch), the second on a smaller one: the scratch keeps the first
    # call's contents, which must not leak into the second
    for seed, nrows, ncols, L in ((k, 3000, 2000, 16), (k + 1, 700, 500, None)):
        rowptr, colind, val, H, G = case(seed, nrows, ncols, k)
        ref, got = run_both(nsd, nrows, ncols, rowptr, colind, val, H, G, k, item_len=L)
        for a, b in zip(ref, got):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
        D = orc.Dok.from_csr(nrows, ncols, rowptr, colind, val)
        rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
        L_, Lm = orc.loss_bilinear(D, G, H, k)
        dA, dAm = orc.sddmm(D, G, H, k, rows, colind, alpha=0.5)
        dH, dHm = orc.spmm_t(D, G, k, alpha=0.5)
        assert_mag_close(got[0][0], L_, Lm, what="loss")
        assert_mag_close(got[1], dA, dAm, what="dA")
        assert_mag_close(got[2], dH, dHm, what="dH")


def test_noalloc_refuses_operands_beyond_the_scratch(nsd):
    # two columns of 600,000 entries cut into 16-entry chunks: 75,000 chunk
    # partial rows of 1 KiB, more than the 64 MiB scratch
    from paper_2303_07030_amd.operand import DeviceCsr
    nrows, ncols, k = 600_000, 2, 256
    rowptr = np.arange(0, 2 * nrows + 1, 2, dtype=np.int32)
    colind = np.tile(np.array([0, 1], np.int32), nrows)
    val = np.ones(2 * nrows, np.float32)
    A = DeviceCsr(nrows, ncols, rowptr, colind, val, k_hint=k, item_len=16)
    H = torch.zeros((ncols, k), device="cuda")
    G = torch.zeros((nrows, k), device="cuda")
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    dA = torch.zeros(A.nnz, device="cuda")
    dH = torch.full((ncols, k), 7.0, device="cuda")
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_loss_bilinear_noalloc(A.desc, A.csc, H, G, k, 1.0, loss, dA, dH)
    assert e.value.status == nsd.NSD_ERR_WORKSPACE
    assert "static scratch" in nsd.nsd_last_error()
    torch.cuda.synchronize()
    assert torch.all(dH == 7.0)  # nothing was launched
