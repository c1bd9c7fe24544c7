"""Parity of the HIP path with the fp64 oracle, called through the C ABI.

Index and pattern outputs must equal the oracle bit for bit; floating-point
outputs must satisfy |got - ref| <= 1e-4 * mag (mag: the oracle's evaluation
on absolute values), with exact zeros where mag is 0.
"""
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


@pytest.fixture(scope="module")
def operand(nsd):
    from paper_2303_07030_amd.operand import DeviceCsr
    return DeviceCsr


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def make_csr(rng, nrows, ncols, lengths, hot_col=None):
    """Sorted unique columns per row; hot_col (if given) joins every other row."""
    rowptr = np.zeros(nrows + 1, np.int64)
    cols = []
    for r in range(nrows):
        L = int(lengths[r])
        c = rng.choice(ncols, size=L, replace=False) if L else np.empty(0, np.int64)
        if hot_col is not None and r % 2 == 0 and L and hot_col not in c:
            c[0] = hot_col
        c = np.sort(c)
        cols.append(c)
        rowptr[r + 1] = rowptr[r] + L
    colind = np.concatenate(cols).astype(np.int32) if cols else np.empty(0, np.int32)
    val = rng.standard_normal(colind.shape[0]).astype(np.float32)
    return rowptr.astype(np.int32), colind, val


def edge_pattern(seed=0, nrows=700, ncols=900):
    """Power-law rows, empty rows at the start, middle and end, one row of
    850 entries spanning many slots, and a column present in half the rows."""
    rng = np.random.default_rng(seed)
    lengths = np.minimum((40 * rng.pareto(1.2, nrows)).astype(np.int64), 300)
    lengths[[0, 1, 350, 351, nrows - 3, nrows - 2, nrows - 1]] = 0
    lengths[123] = 850
    return nrows, ncols, *make_csr(rng, nrows, ncols, lengths, hot_col=5)


def oracle_dok(orc, nrows, ncols, rowptr, colind, val):
    return orc.Dok.from_csr(nrows, ncols, rowptr, colind, val)


# ------------------------------------------------------------------ builders

def test_expand_rows_bit_exact(nsd, operand):
    nrows, ncols, rowptr, colind, val = edge_pattern(1)
    A = operand(nrows, ncols, rowptr, colind, val, build_csc=False)
    ref = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    assert np.array_equal(host(A.rowidx), ref)


@pytest.mark.parametrize("seed", [0, 1])
def test_csr_to_csc_bit_exact(nsd, operand, orc, seed):
    nrows, ncols, rowptr, colind, val = edge_pattern(seed)
    A = operand(nrows, ncols, rowptr, colind, val)
    segptr, skey, perm = orc.stable_sort_by_key(colind, ncols)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    assert np.array_equal(host(A.colptr), segptr)
    assert np.array_equal(host(A.colidx), skey)
    assert np.array_equal(host(A.perm), perm)
    assert np.array_equal(host(A.rowind), rows[perm])


def test_csr_to_csc_full_size_spmm_workload(nsd, operand, orc):
    from paper_2303_07030_amd import synth
    d = synth.make("spmm")
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    segptr, skey, perm = orc.stable_sort_by_key(d["colind"], d["ncols"])
    assert np.array_equal(host(A.colptr), segptr)
    assert np.array_equal(host(A.perm), perm)
    assert np.array_equal(host(A.colidx), skey)


@pytest.mark.parametrize("seed", [0, 3])
def test_coo_to_csr_sums_duplicates(nsd, orc, seed):
    rng = np.random.default_rng(seed)
    nr, nc, n = 300, 517, 20000
    keys = rng.choice(nr * nc, size=n - 3000, replace=False)
    keys = np.concatenate([keys, rng.choice(keys, size=3000)])
    rng.shuffle(keys)
    row, col = (keys // nc).astype(np.int32), (keys % nc).astype(np.int32)
    val = rng.standard_normal(n).astype(np.float32)
    ws = torch.empty(nsd.nsd_build_workspace_size(n, max(nr, nc)), dtype=torch.uint8, device="cuda")
    out = [torch.empty(m, dtype=t, device="cuda") for m, t in
           [(nr + 1, torch.int32), (n, torch.int32), (n, torch.int32), (n, torch.float32),
            (n, torch.int32)]]
    nuniq = nsd.nsd_coo_to_csr(nr, nc, n, dev(row), dev(col), dev(val), nsd.NSD_DUP_SUM, *out, ws)
    rowptr_r, colind_r, val_r, first_r = orc.coo_to_csr(orc.Dok((nr, nc), (row, col), val))
    assert nuniq == len(colind_r)
    rowptr, rowidx, colind, vout, perm = [host(t) for t in out]
    assert np.array_equal(rowptr, rowptr_r)
    assert np.array_equal(colind[:nuniq], colind_r)
    assert np.array_equal(perm[:nuniq], first_r)
    assert np.array_equal(rowidx[:nuniq], np.repeat(np.arange(nr), np.diff(rowptr_r)))
    # values: the fp32 sum of the duplicates; bit-exact where there is only one
    counts = np.bincount(np.searchsorted(np.unique(keys), keys), minlength=nuniq)
    single = counts == 1
    assert np.array_equal(vout[:nuniq][single], val[first_r[single]])
    mag = np.zeros(nuniq)
    np.add.at(mag, np.searchsorted(np.unique(keys), keys), np.abs(val.astype(np.float64)))
    assert_mag_close(vout[:nuniq], val_r, mag, what="merged values")


@pytest.mark.parametrize("nrows,ncols", [(1, 1), (3, 2), (1, 1 << 24), (1 << 21, 3),
                                         (256, 256), (257, 255), (70_000, 65_536),
                                         (1_000_003, 300_007), (1 << 20, (1 << 31) - 1)])
def test_coo_to_csr_pair_key_widths(nsd, nrows, ncols):
    """The sort by the pair (row, col) over the combined bits of both
    coordinates (2 to 51 of them: digits straddling the two words, a last
    pass of few bits) against a stable lexicographic sort, duplicates
    merged."""
    rng = np.random.default_rng(nrows ^ ncols)
    n = 30_000
    row = rng.integers(0, nrows, n).astype(np.int32)
    col = rng.integers(0, ncols, n).astype(np.int32)
    row[:50], col[:50] = nrows - 1, ncols - 1  # the largest coordinates, repeated
    val = rng.standard_normal(n).astype(np.float32)
    ws = torch.empty(nsd.nsd_build_workspace_size(n, max(nrows, ncols)), dtype=torch.uint8,
                     device="cuda")
    rowptr = torch.empty(nrows + 1, dtype=torch.int32, device="cuda")
    out = [rowptr] + [torch.empty(n, dtype=t, device="cuda")
                      for t in (torch.int32, torch.int32, torch.float32, torch.int32)]
    m = nsd.nsd_coo_to_csr(nrows, ncols, n, dev(row), dev(col), dev(val), nsd.NSD_DUP_SUM, *out,
                           ws)
    order = np.lexsort((col, row))
    r, c = row[order], col[order]
    head = np.ones(n, bool)
    head[1:] = (r[1:] != r[:-1]) | (c[1:] != c[:-1])
    assert m == int(head.sum())
    _, rowidx, colind, _, perm = [host(t) for t in out]
    assert np.array_equal(rowidx[:m], r[head])
    assert np.array_equal(colind[:m], c[head])
    assert np.array_equal(perm[:m], order[head])
    assert np.array_equal(host(rowptr), np.searchsorted(r[head], np.arange(nrows + 1)))


def test_coo_to_csr_errors(nsd):
    row = dev(np.array([0, 1, 1, 2], np.int32))
    col = dev(np.array([0, 2, 2, 1], np.int32))
    val = dev(np.ones(4, np.float32))
    ws = torch.empty(nsd.nsd_build_workspace_size(4, 3), dtype=torch.uint8, device="cuda")
    outs = [torch.empty(m, dtype=t, device="cuda") for m, t in
            [(4, torch.int32), (4, torch.int32), (4, torch.int32), (4, torch.float32),
             (4, torch.int32)]]
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_coo_to_csr(3, 3, 4, row, col, val, nsd.NSD_DUP_ERROR, *outs, ws)
    assert e.value.status == nsd.NSD_ERR_DUPLICATE
    bad = dev(np.array([0, 1, 5, 2], np.int32))
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_coo_to_csr(3, 3, 4, row, bad, val, nsd.NSD_DUP_SUM, *outs, ws)
    assert e.value.status == nsd.NSD_ERR_BAD_FORMAT
    for r, c in (([0, 3, 1, 2], [0, 2, 2, 1]), ([0, 1, 1, 2], [0, -1, 2, 1]),
                 ([-5, 1, 1, 2], [0, 2, 2, 1])):  # a row past the end, negative indices
        with pytest.raises(nsd.NsdError) as e:
            nsd.nsd_coo_to_csr(3, 3, 4, dev(np.array(r, np.int32)), dev(np.array(c, np.int32)),
                               val, nsd.NSD_DUP_SUM, *outs, ws)
        assert e.value.status == nsd.NSD_ERR_BAD_FORMAT
    assert nsd.nsd_coo_to_csr(3, 3, 4, row, col, val, nsd.NSD_DUP_SUM, *outs, ws) == 3


def test_csc_and_mode_index_reject_out_of_range(nsd, operand):
    """A column (or mode key) outside its range is refused, whichever
    position holds it; the builders stay usable afterwards."""
    n = 5000
    ws = torch.empty(nsd.nsd_build_workspace_size(n, 64), dtype=torch.uint8, device="cuda")
    i32 = lambda m: torch.empty(max(m, 1), dtype=torch.int32, device="cuda")  # noqa: E731
    rng = np.random.default_rng(4)
    for bad in (64, -1, 1 << 30):
        for at in (0, 2047, n - 1):
            key = rng.integers(0, 64, n).astype(np.int32)
            key[at] = bad
            with pytest.raises(nsd.NsdError) as e:
                nsd.nsd_coo_mode_index(n, 64, dev(key), i32(65), i32(n), i32(n), ws)
            assert e.value.status == nsd.NSD_ERR_BAD_FORMAT
            rowptr = np.arange(0, n + 1, 5, dtype=np.int32)  # rows of 5 entries
            colind = key.copy()
            A = nsd.csr_desc(len(rowptr) - 1, 64, dev(rowptr),
                             dev(np.repeat(np.arange(len(rowptr) - 1), 5).astype(np.int32)),
                             dev(colind), dev(np.ones(n, np.float32)))
            with pytest.raises(nsd.NsdError) as e:
                nsd.nsd_csr_to_csc(A, i32(65), i32(n), i32(n), i32(n), ws)
            assert e.value.status == nsd.NSD_ERR_BAD_FORMAT
    key = rng.integers(0, 64, n).astype(np.int32)
    segptr, segidx, perm = i32(65), i32(n), i32(n)
    nsd.nsd_coo_mode_index(n, 64, dev(key), segptr, segidx, perm, ws)
    assert np.array_equal(host(perm)[:n], np.argsort(key, kind="stable"))


def test_mode_index_bit_exact(nsd, orc):
    from paper_2303_07030_amd import synth
    d = synth.make("cp", "small")
    n = len(d["val"])
    ws = torch.empty(nsd.nsd_build_workspace_size(n, d["dims"][0]), dtype=torch.uint8,
                     device="cuda")
    for key in (d["i"], d["j"], d["k"]):
        segptr = torch.empty(d["dims"][0] + 1, dtype=torch.int32, device="cuda")
        segidx = torch.empty(n, dtype=torch.int32, device="cuda")
        perm = torch.empty(n, dtype=torch.int32, device="cuda")
        nsd.nsd_coo_mode_index(n, d["dims"][0], dev(key), segptr, segidx, perm, ws)
        rs, rk, rp = orc.stable_sort_by_key(key, d["dims"][0])
        assert np.array_equal(host(segptr), rs)
        assert np.array_equal(host(segidx), rk)
        assert np.array_equal(host(perm), rp)


def test_gather_is_exact_copy(nsd):
    rng = np.random.default_rng(2)
    src = rng.standard_normal(5000).astype(np.float32)
    perm = rng.permutation(5000).astype(np.int32)
    dst = torch.empty(5000, dtype=torch.float32, device="cuda")
    nsd.nsd_gather_f32(5000, dev(perm), dev(src), dst)
    assert np.array_equal(host(dst), src[perm])


def test_validate_csr(nsd, operand):
    nrows, ncols, rowptr, colind, val = edge_pattern(4)
    A = operand(nrows, ncols, rowptr, colind, val, build_csc=False)
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    nsd.nsd_validate_csr(A.desc, 1, ws)
    bad = colind.copy()
    r = 123
    bad[rowptr[r]], bad[rowptr[r] + 1] = bad[rowptr[r] + 1], bad[rowptr[r]]
    B = operand(nrows, ncols, rowptr, bad, val, build_csc=False)
    nsd.nsd_validate_csr(B.desc, 0, ws)  # order not checked
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_validate_csr(B.desc, 1, ws)
    assert e.value.status == nsd.NSD_ERR_BAD_FORMAT and "order" in str(e.value)
    bad2 = colind.copy()
    bad2[10] = ncols + 3
    Cm = operand(nrows, ncols, rowptr, bad2, val, build_csc=False)
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_validate_csr(Cm.desc, 0, ws)
    assert "column-range" in str(e.value)


@pytest.mark.parametrize("L", [4, 16, 64, 256])
def test_plan_invariants(nsd, L):
    # a plan is an implementation device, checked by its defining properties:
    # items tile the entries of the non-empty segments in order, never split a
    # short segment (at most S = L + min(L, 32) entries), cut long ones into
    # chunks of L, and list empty segments
    from paper_2303_07030_amd.operand import build_plan
    nrows, ncols, rowptr, colind, val = edge_pattern(5)
    lens = np.diff(rowptr)
    plan = build_plan(nrows, len(colind), dev(rowptr), L, "cuda")
    n_it, n_long, n_empty = plan.nitems, plan.nlong, plan.nempty
    kp = plan._keep
    item_ptr = host(kp["item_ptr"])[: n_it + 1]
    long_first = host(kp["long_first"])[:n_long]
    long_seg = host(kp["long_seg"])[:n_long]
    huge = host(kp["huge_idx"])[: plan.nhuge]
    chunks = host(kp["chunk_item"])[: plan.nchunks]
    empty = host(kp["empty_seg"])[:n_empty]
    assert item_ptr[0] == 0 and item_ptr[-1] == len(colind)
    assert np.all(np.diff(item_ptr) > 0)
    assert np.array_equal(empty, np.nonzero(lens == 0)[0])
    S = L + min(L, 32)
    long_rows = np.nonzero(lens > S)[0]
    assert n_long == len(long_rows) and np.array_equal(long_seg, long_rows)
    nch_all = -(-lens[long_rows] // L)
    assert np.array_equal(huge, np.nonzero(nch_all > 64)[0])
    assert plan.nchunks == nch_all.sum()
    assert plan.longest_chunks == (nch_all.max() if n_long else 0)
    assert np.array_equal(chunks, np.concatenate(
        [long_first[i] + np.arange(nch_all[i]) for i in range(n_long)]) if n_long else chunks)
    starts = set(item_ptr[:-1].tolist())
    for r in np.nonzero((lens > 0) & (lens <= S))[0]:
        # a short row lies inside one item: no item starts strictly inside it
        inner = [q for q in range(rowptr[r] + 1, rowptr[r + 1]) if q in starts]
        assert not inner
    for i, r in enumerate(long_rows):
        s0 = long_first[i]
        nch = -(-lens[r] // L)
        assert np.array_equal(item_ptr[s0:s0 + nch + 1][:-1], rowptr[r] + L * np.arange(nch))
        assert item_ptr[s0 + nch] == rowptr[r + 1]
    # bounded work: an item of short rows holds at most L + S entries
    assert np.diff(item_ptr).max() <= L + S
    # compact partial rows: a chunk item's row is its position in chunk_item
    ord_ = host(kp["chunk_ord"])[:n_it]
    want = np.full(n_it, -1, np.int32)
    want[chunks] = np.arange(plan.nchunks)
    assert np.array_equal(ord_, want)


# ---------------------------------------------------------------- primitives

KS = [1, 3, 4, 8, 16, 32, 64, 100, 128, 256, 264]


@pytest.fixture(scope="module")
def edge_A(operand, orc):
    nrows, ncols, rowptr, colind, val = edge_pattern(7)
    A = operand(nrows, ncols, rowptr, colind, val)
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    return A, D, rows, colind


@pytest.mark.parametrize("k", KS)
def test_spmm(nsd, orc, edge_A, k):
    A, D, _, _ = edge_A
    rng = np.random.default_rng(k)
    B = rng.standard_normal((A.ncols, k)).astype(np.float32)
    Cg = torch.full((A.nrows, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm(A.desc, dev(B), k, Cg, A.workspace(k))
    ref, mag = orc.spmm(D, B, k)
    assert_mag_close(host(Cg), ref, mag, what=f"spmm k={k}")


def test_spmv(nsd, orc, edge_A):
    A, D, _, _ = edge_A
    x = np.random.default_rng(0).standard_normal(A.ncols).astype(np.float32)
    y = torch.full((A.nrows,), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmv(A.desc, dev(x), y, A.workspace(1))
    ref, mag = orc.spmm(D, x.reshape(-1, 1), 1)
    assert_mag_close(host(y), ref[:, 0], mag[:, 0], what="spmv")


@pytest.mark.parametrize("k", KS)
def test_sddmm(nsd, orc, edge_A, k):
    A, D, rows, cols = edge_A
    rng = np.random.default_rng(100 + k)
    X = rng.standard_normal((A.nrows, k)).astype(np.float32)
    Y = rng.standard_normal((A.ncols, k)).astype(np.float32)
    out = torch.full((A.nnz,), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_sddmm(A.desc, dev(X), dev(Y), k, -0.75, out)
    ref, mag = orc.sddmm(D, X, Y, k, rows, cols, alpha=-0.75)
    assert_mag_close(host(out), ref, mag, what=f"sddmm k={k}")


@pytest.mark.parametrize("k", KS)
def test_spmm_t(nsd, orc, edge_A, k):
    A, D, _, _ = edge_A
    rng = np.random.default_rng(200 + k)
    G = rng.standard_normal((A.nrows, k)).astype(np.float32)
    out = torch.full((A.ncols, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm_t(A.desc, A.csc, dev(G), k, 1.5, out, A.workspace(k))
    ref, mag = orc.spmm_t(D, G, k, alpha=1.5)
    assert_mag_close(host(out), ref, mag, what=f"spmm_t k={k}")


def chunk_offsets_pattern():
    """Rows for item length 4: long rows whose first chunk falls at every
    offset within a group of 8 slots (3 to 39 chunks, ragged last chunks),
    a row of 75 chunks (a huge plan segment with few partial rows) and one of
    750 chunks (more than 64 partial rows even after the in-wave sums),
    between short and empty rows."""
    rng = np.random.default_rng(41)
    lengths = [1, 0, 2] + [4 * c - (c % 3) for c in range(3, 40)] + [1] * 5
    lengths += [300, 0, 3000, 9, 17, 1, 0]
    nrows, ncols = len(lengths), 4000
    return nrows, ncols, *make_csr(rng, nrows, ncols, np.array(lengths), hot_col=7)


@pytest.mark.parametrize("k", [1, 8, 12, 64, 256])
def test_chunk_partials_at_every_group_offset(nsd, operand, orc, k):
    nrows, ncols, rowptr, colind, val = chunk_offsets_pattern()
    A = operand(nrows, ncols, rowptr, colind, val, item_len=4, k_hint=k)
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    rng = np.random.default_rng(300 + k)
    B = rng.standard_normal((ncols, k)).astype(np.float32)
    G = rng.standard_normal((nrows, k)).astype(np.float32)
    Cg = torch.full((nrows, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm(A.desc, dev(B), k, Cg, A.workspace(k))
    ref, mag = orc.spmm(D, B, k)
    assert_mag_close(host(Cg), ref, mag, what=f"spmm k={k}")
    out = torch.full((ncols, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm_t(A.desc, A.csc, dev(G), k, 1.0, out, A.workspace(k))
    ref, mag = orc.spmm_t(D, G, k)
    assert_mag_close(host(out), ref, mag, what=f"spmm_t k={k}")
    if k % 4 == 0 and k <= 256:
        got = run_frob(nsd, A, B, k)
        check_frob(orc, nrows, ncols, rowptr, colind, val, B, k, got)


def test_spmm_t_ones_is_column_sums(nsd, orc, edge_A):
    A, D, _, _ = edge_A
    out = torch.full((A.ncols, 1), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm_t(A.desc, A.csc, None, 1, 1.0, out, A.workspace(1))
    ref, mag = orc.spmm_t(D, None, 1)
    assert_mag_close(host(out), ref, mag, what="column sums")


# ------------------------------------------------------------ fused losses

def run_frob(nsd, A, B, k, seed=1.0):
    Cg = torch.empty((A.nrows, k), dtype=torch.float32, device="cuda")
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dA = torch.empty(A.nnz, dtype=torch.float32, device="cuda")
    dB = torch.empty((A.ncols, k), dtype=torch.float32, device="cuda")
    nsd.nsd_loss_frob_spmm(A.desc, A.csc, dev(B), k, seed, Cg, loss, dA, dB, A.workspace(k))
    return host(Cg), host(loss)[0], host(dA), host(dB)


def check_frob(orc, nrows, ncols, rowptr, colind, val, B, k, got, seed=1.0):
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    rows = np.repeat(np.arange(nrows, dtype=np.int32), np.diff(rowptr))
    Cref, Cmag = orc.spmm(D, B, k)
    L, Lmag = orc.loss_half_sq(Cref, Cmag)
    dA, dAm = orc.sddmm(D, Cref, B, k, rows, colind, alpha=seed, Xmag=Cmag)
    dB, dBm = orc.spmm_t(D, Cref, k, alpha=seed, Gmag=Cmag)
    Cg, Lg, dAg, dBg = got
    assert_mag_close(Cg, Cref, Cmag, what="C")
    assert_mag_close(Lg, L, Lmag, what="loss")
    assert_mag_close(dAg, dA, dAm, what="dA")
    assert_mag_close(dBg, dB, dBm, what="dB")


def test_loss_sum_spmv_full_workload(nsd, operand, orc):
    from paper_2303_07030_amd import synth
    d = synth.make("spmv")
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dA = torch.empty(A.nnz, dtype=torch.float32, device="cuda")
    dx = torch.empty(A.ncols, dtype=torch.float32, device="cuda")
    nsd.nsd_loss_sum_spmv(A.desc, A.csc, dev(d["x"]), 1.0, loss, dA, dx, A.workspace(1))
    D = oracle_dok(orc, d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    L, Lm = orc.loss_sum_spmv(D, d["x"])
    assert_mag_close(host(loss)[0], L, Lm, what="loss")
    # closed forms: dA = x[col] exactly, dx = column sums
    assert np.array_equal(host(dA), d["x"][d["colind"]])
    ref, mag = orc.spmm_t(D, None, 1)
    assert_mag_close(host(dx), ref[:, 0], mag[:, 0], what="dx")


@pytest.mark.parametrize("size", ["small", "full"])
def test_loss_frob_spmm_workload(nsd, operand, orc, size):
    from paper_2303_07030_amd import synth
    d = synth.make("spmm", size)
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    got = run_frob(nsd, A, d["B"], d["k"])
    check_frob(orc, d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"], d["B"], d["k"], got)


@pytest.mark.parametrize("k", [1, 12, 64, 128])
def test_loss_frob_spmm_edge(nsd, operand, orc, k):
    nrows, ncols, rowptr, colind, val = edge_pattern(11)
    A = operand(nrows, ncols, rowptr, colind, val)
    B = np.random.default_rng(k).standard_normal((ncols, k)).astype(np.float32)
    got = run_frob(nsd, A, B, k, seed=0.5)
    check_frob(orc, nrows, ncols, rowptr, colind, val, B, k, got, seed=0.5)


def run_bilinear(nsd, A, H, G, k, seed=1.0):
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dA = torch.empty(A.nnz, dtype=torch.float32, device="cuda")
    dH = torch.empty((A.ncols, k), dtype=torch.float32, device="cuda")
    nsd.nsd_loss_bilinear(A.desc, A.csc, dev(H), dev(G), k, seed, loss, dA, dH, A.workspace(k))
    return host(loss)[0], host(dA), host(dH)


def test_loss_bilinear_small_workload(nsd, operand, orc):
    from paper_2303_07030_amd import synth
    d = synth.make("gnn", "small")
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    Lg, dAg, dHg = run_bilinear(nsd, A, d["H"], d["G"], d["k"])
    D = oracle_dok(orc, d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    rows = np.repeat(np.arange(d["nrows"], dtype=np.int32), np.diff(d["rowptr"]))
    L, Lm = orc.loss_bilinear(D, d["G"], d["H"], d["k"])
    dA, dAm = orc.sddmm(D, d["G"], d["H"], d["k"], rows, d["colind"])
    dH, dHm = orc.spmm_t(D, d["G"], d["k"])
    assert_mag_close(Lg, L, Lm, what="loss")
    assert_mag_close(dAg, dA, dAm, what="dA")
    assert_mag_close(dHg, dH, dHm, what="dH")


def run_mf(nsd, A, U, V, k, seed=1.0, with_valT=True):
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dU = torch.full((A.nrows, k), np.nan, dtype=torch.float32, device="cuda")
    dV = torch.full((A.ncols, k), np.nan, dtype=torch.float32, device="cuda")
    valT = A.values_in_csc_order() if with_valT else None
    nsd.nsd_loss_mf(A.desc, A.csc, valT, dev(U), dev(V), k, seed, loss, dU, dV, A.workspace(k))
    return host(loss)[0], host(dU), host(dV)


def check_mf(orc, D, U, V, k, got, seed=1.0):
    L, Lm = orc.mf_loss(D, U, V, k)
    dU, dUm = orc.mf_grad(D, U, V, k, 0)
    dV, dVm = orc.mf_grad(D, U, V, k, 1)
    Lg, dUg, dVg = got
    assert_mag_close(Lg, L, Lm, what="loss")
    assert_mag_close(dUg, seed * dU, abs(seed) * dUm, what="dU")
    assert_mag_close(dVg, seed * dV, abs(seed) * dVm, what="dV")


def test_loss_mf_small_workload_from_coo(nsd, operand, orc):
    from paper_2303_07030_amd import synth
    d = synth.make("mf", "small")
    A = operand.from_coo(d["nrows"], d["ncols"], d["row"], d["col"], d["val"], k_hint=d["k"])
    got = run_mf(nsd, A, d["U"], d["V"], d["k"])
    D = orc.Dok((d["nrows"], d["ncols"]), (d["row"], d["col"]), d["val"])
    check_mf(orc, D, d["U"], d["V"], d["k"], got)
    # the column pass reading values through perm gives the same bits
    got2 = run_mf(nsd, A, d["U"], d["V"], d["k"], with_valT=False)
    for x, y in zip(got, got2):
        assert np.array_equal(np.asarray(x), np.asarray(y))


@pytest.mark.parametrize("k", [1, 5, 12, 64, 128, 256])
def test_loss_mf_edge(nsd, operand, orc, k):
    nrows, ncols, rowptr, colind, val = edge_pattern(13)
    val = (1 + 4 * np.abs(val)).astype(np.float32)
    A = operand(nrows, ncols, rowptr, colind, val, k_hint=k)
    rng = np.random.default_rng(k)
    U = (0.1 * rng.standard_normal((nrows, k))).astype(np.float32)
    V = (0.1 * rng.standard_normal((ncols, k))).astype(np.float32)
    got = run_mf(nsd, A, U, V, k, seed=0.5)
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    check_mf(orc, D, U, V, k, got, seed=0.5)


def run_cp(nsd, X, F, rank, seed=1.0):
    from paper_2303_07030_amd.operand import DeviceCoo3  # noqa: F401
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dX = torch.full((X.nnz,), np.nan, dtype=torch.float32, device="cuda")
    dF = [torch.full((X.dims[m], rank), np.nan, dtype=torch.float32, device="cuda")
          for m in range(3)]
    nsd.nsd_loss_cp(X.desc, *[dev(f) for f in F], rank, seed, loss, dX, *dF, X.workspace(rank))
    return host(loss)[0], in_input_order(X, host(dX)), [host(t) for t in dF]


def in_input_order(X, stored):
    """A value array on X's keys, from X's stored (lexicographic) order back
    to the order of the input coordinates."""
    out = np.full(X.nnz, np.nan, dtype=stored.dtype)
    out[host(X.coo_perm)] = stored[: X.nnz]
    return out


def check_cp(orc, dims, i, j, l, val, F, rank, got, seed=1.0):
    D = orc.Dok(dims, (i, j, l), val)
    L, Lm = orc.cp_loss(D, *F, rank)
    R, Rm = orc.cp_resid(D, *F, rank, i, j, l)
    Lg, dXg, dFg = got
    assert_mag_close(Lg, L, Lm, what="loss")
    assert_mag_close(dXg, seed * R, abs(seed) * Rm, what="residual")
    for m in range(3):
        g, gm = orc.cp_grad(D, *F, rank, m)
        assert_mag_close(dFg[m], seed * g, abs(seed) * gm, what=f"dF{m + 1}")


@pytest.mark.parametrize("order", [3, 4, 6])
def test_coo_stored_in_lexicographic_order(nsd, order):
    # the operand's storage order is the stable lexicographic sort of the
    # input coordinates, built by the library's mode index (bit-exact)
    from paper_2303_07030_amd.operand import DeviceCoo3, DeviceCooN
    rng = np.random.default_rng(order)
    dims = (9, 40, 3, 17, 2, 5)[:order]
    nnz = 3000
    coords = [rng.integers(0, d, nnz).astype(np.int32) for d in dims]  # duplicates too
    val = rng.standard_normal(nnz).astype(np.float32)
    X = DeviceCoo3(dims, *coords, val) if order == 3 else DeviceCooN(dims, coords, val)
    want = np.lexsort(coords[::-1])
    assert np.array_equal(host(X.coo_perm), want)
    for m in range(order):
        assert np.array_equal(host(X.coords[m]), coords[m][want])
    assert np.array_equal(host(X.val), val[want])


def test_loss_cp_small_workload(nsd, orc):
    from paper_2303_07030_amd import synth
    from paper_2303_07030_amd.operand import DeviceCoo3
    d = synth.make("cp", "small")
    X = DeviceCoo3(d["dims"], d["i"], d["j"], d["k"], d["val"], rank_hint=d["rank"])
    F = [d["F1"], d["F2"], d["F3"]]
    got = run_cp(nsd, X, F, d["rank"])
    check_cp(orc, d["dims"], d["i"], d["j"], d["k"], d["val"], F, d["rank"], got)


@pytest.mark.parametrize("rank,dims", [(32, (7, 300, 45)), (8, (50, 3, 200)), (5, (20, 20, 20)),
                                       (64, (1, 40, 40))])
def test_loss_cp_shapes(nsd, orc, rank, dims):
    # skewed mode sizes: long slices (a mode of size 1 or 3), short ones, and
    # empty slices; odd rank takes the scalar lane layout
    from paper_2303_07030_amd.operand import DeviceCoo3
    rng = np.random.default_rng(rank)
    total = dims[0] * dims[1] * dims[2]
    nnz = min(4000, total // 2)
    keys = rng.choice(total, size=nnz, replace=False)
    i = (keys // (dims[1] * dims[2])).astype(np.int32)
    j = ((keys // dims[2]) % dims[1]).astype(np.int32)
    l = (keys % dims[2]).astype(np.int32)
    val = rng.standard_normal(nnz).astype(np.float32)
    F = [(0.3 * rng.standard_normal((dims[m], rank))).astype(np.float32) for m in range(3)]
    X = DeviceCoo3(dims, i, j, l, val, rank_hint=rank, item_len=16)
    got = run_cp(nsd, X, F, rank, seed=2.0)
    check_cp(orc, dims, i, j, l, val, F, rank, got, seed=2.0)


@pytest.mark.parametrize("dims,nnz", [((60, 60, 60), 25_000), ((5, 7, 300), 2_000),
                                       ((40, 30, 1), 500)])
def test_ttv_and_vjp(nsd, orc, dims, nnz):
    from paper_2303_07030_amd.operand import DeviceTtv
    rng = np.random.default_rng(nnz)
    keys = rng.choice(dims[0] * dims[1] * dims[2], size=nnz, replace=False)
    i = (keys // (dims[1] * dims[2])).astype(np.int32)
    j = ((keys // dims[2]) % dims[1]).astype(np.int32)
    l = (keys % dims[2]).astype(np.int32)
    x = rng.standard_normal(nnz).astype(np.float32)
    v = rng.standard_normal(dims[2]).astype(np.float32)
    T = DeviceTtv(dims, [i, j, l])
    D = orc.Dok(dims, (i, j, l), x)
    yi, yj, y, ym = orc.ttv(D, v)
    assert T.ny == len(yi)
    assert np.array_equal(host(T.ykey[0])[:T.ny], yi)
    assert np.array_equal(host(T.ykey[1])[:T.ny], yj)
    ws = T.workspace()
    yg = torch.full((T.ny,), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_ttv(T.desc, dev(x), dev(v), yg, ws)
    assert_mag_close(host(yg), y, ym, what="Y")
    gy = rng.standard_normal(T.ny).astype(np.float32)
    dx = torch.full((nnz,), np.nan, dtype=torch.float32, device="cuda")
    dv = torch.full((dims[2],), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_ttv_vjp(T.desc, dev(x), dev(v), dev(gy), dx, dv, ws)
    gY = orc.Dok((dims[0], dims[1]), (yi, yj), gy)
    rdx, rdxm, rdv, rdvm = orc.ttv_vjp(D, v, gY, i, j, l)
    assert_mag_close(host(dx), rdx, rdxm, what="dX")
    assert_mag_close(host(dv), rdv, rdvm, what="dv")


@pytest.mark.parametrize("R", [1, 3, 8, 32, 64, 100])
@pytest.mark.parametrize("dims,nnz", [((30, 40, 50), 6000), ((3, 4, 2000), 5000)])
def test_ttm_and_vjp(nsd, orc, dims, nnz, R):
    # TTM along mode 3 on the projected keys and its VJP; the second shape
    # gives few projected keys holding long l-fibres (chunked segments)
    from paper_2303_07030_amd.operand import DeviceTtv
    rng = np.random.default_rng(nnz + R)
    keys = rng.choice(dims[0] * dims[1] * dims[2], size=nnz, replace=False)
    i = (keys // (dims[1] * dims[2])).astype(np.int32)
    j = ((keys // dims[2]) % dims[1]).astype(np.int32)
    l = (keys % dims[2]).astype(np.int32)
    x = rng.standard_normal(nnz).astype(np.float32)
    U = rng.standard_normal((dims[2], R)).astype(np.float32)
    T = DeviceTtv(dims, [i, j, l])
    D = orc.Dok(dims, (i, j, l), x)
    yi, yj, y, ym = orc.ttm(D, U, R)
    assert T.ny == len(yi)
    ws = T.ttm_workspace(R)
    Y = torch.full((T.ny, R), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_ttm(T.desc, dev(x), dev(U), R, Y, ws)
    assert_mag_close(host(Y), y, ym, what="Y")
    gY = rng.standard_normal((T.ny, R)).astype(np.float32)
    dx = torch.full((nnz,), np.nan, dtype=torch.float32, device="cuda")
    dU = torch.full((dims[2], R), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_ttm_vjp(T.desc, dev(x), dev(U), R, dev(gY), dx, dU, ws)
    rdx, rdxm, rdU, rdUm = orc.ttm_vjp(D, U, R, gY, i, j, l)
    assert_mag_close(host(dx), rdx, rdxm, what="dX")
    assert_mag_close(host(dU), rdU, rdUm, what="dU")


@pytest.mark.parametrize("dims,R", [((20, 30, 25), 7), ((6, 5, 4, 7), 16), ((4, 5, 3, 6, 2), 3),
                                    ((3, 4, 2, 5, 2, 3), 64), ((2, 300, 3), 100)])
def test_mode_products_every_mode(nsd, orc, dims, R):
    """TTM (and TTV, its width-1 case) along every mode of orders 3 to 6,
    with the VJPs: projected keys bit for bit, values against the oracle's
    mode product (the 2 x 300 x 3 shape gives long fibres in mode 1)."""
    from paper_2303_07030_amd.operand import DeviceTtv
    N = len(dims)
    rng = np.random.default_rng(sum(dims) * R)
    size = int(np.prod(dims))
    nnz = min(size // 2, 6000)
    keys = rng.choice(size, size=nnz, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(keys, dims)]
    perm = rng.permutation(nnz)  # input order not sorted
    coords = [c[perm] for c in coords]
    x = rng.standard_normal(nnz).astype(np.float32)
    D = orc.Dok(dims, coords, x)
    for n in range(N):
        T = DeviceTtv(dims, coords, mode=n)
        U = rng.standard_normal((dims[n], R)).astype(np.float32)
        yk, y, ym = orc.ttmn(D, n, U, R)
        assert T.ny == len(yk[0])
        for o in range(N - 1):
            assert np.array_equal(host(T.ykey[o])[:T.ny], yk[o]), f"mode {n} key {o}"
        ws = T.ttm_workspace(R)
        Y = torch.full((T.ny, R), np.nan, dtype=torch.float32, device="cuda")
        nsd.nsd_ttm(T.desc, dev(x), dev(U), R, Y, ws)
        assert_mag_close(host(Y), y, ym, what=f"Y mode {n}")
        gY = rng.standard_normal((T.ny, R)).astype(np.float32)
        dx = torch.full((nnz,), np.nan, dtype=torch.float32, device="cuda")
        dU = torch.full((dims[n], R), np.nan, dtype=torch.float32, device="cuda")
        nsd.nsd_ttm_vjp(T.desc, dev(x), dev(U), R, dev(gY), dx, dU, ws)
        rdx, rdxm, rdU, rdUm = orc.ttmn_vjp(D, n, U, R, gY, coords)
        assert_mag_close(host(dx), rdx, rdxm, what=f"dX mode {n}")
        assert_mag_close(host(dU), rdU, rdUm, what=f"dU mode {n}")
        # TTV along the same mode: the first column of U
        v = U[:, 0].copy()
        yv = torch.full((max(T.ny, 1),), np.nan, dtype=torch.float32, device="cuda")
        nsd.nsd_ttv(T.desc, dev(x), dev(v), yv, T.workspace())
        _, y1, ym1 = orc.ttmn(D, n, v.reshape(-1, 1), 1)
        assert_mag_close(host(yv)[:T.ny], y1[:, 0], ym1[:, 0], what=f"TTV mode {n}")


def test_mode_product_builder_rejects_out_of_range(nsd):
    from paper_2303_07030_amd.operand import DeviceTtv
    c = [np.array([0, 1, 2], np.int32), np.array([0, 5, 1], np.int32),
         np.array([1, 1, 1], np.int32), np.array([0, 0, 0], np.int32)]
    with pytest.raises(nsd.NsdError) as e:
        DeviceTtv((3, 4, 2, 1), c, mode=1)   # 5 >= dims[1]
    assert e.value.status == nsd.NSD_ERR_BAD_FORMAT


# ------------------------------------------------------- edge cases

def test_empty_matrix_writes_zeros(nsd, operand):
    nrows, ncols, k = 50, 40, 64
    A = operand(nrows, ncols, np.zeros(nrows + 1, np.int32), np.empty(0, np.int32),
                np.empty(0, np.float32))
    B = np.ones((ncols, k), np.float32)
    Cg, Lg, dAg, dBg = run_frob(nsd, A, B, k)
    assert Lg == 0.0 and dAg.size == 0
    assert np.all(Cg == 0) and np.all(dBg == 0)
    Lb, _, dH = run_bilinear(nsd, A, B, np.ones((nrows, k), np.float32), k)
    assert Lb == 0.0 and np.all(dH == 0)


def test_single_entry_and_single_dense_row(nsd, operand, orc):
    for nrows, ncols, lengths in [(3, 4, [0, 1, 0]), (5, 3000, [0, 0, 3000, 0, 0])]:
        rng = np.random.default_rng(nrows)
        rowptr, colind, val = make_csr(rng, nrows, ncols, lengths)
        A = operand(nrows, ncols, rowptr, colind, val)
        B = rng.standard_normal((ncols, 64)).astype(np.float32)
        got = run_frob(nsd, A, B, 64)
        check_frob(orc, nrows, ncols, rowptr, colind, val, B, 64, got)


def test_single_dense_column(nsd, operand, orc):
    nrows, ncols = 4000, 6
    rowptr = np.arange(nrows + 1, dtype=np.int32)
    colind = np.full(nrows, 2, np.int32)
    val = np.random.default_rng(9).standard_normal(nrows).astype(np.float32)
    A = operand(nrows, ncols, rowptr, colind, val)
    G = np.random.default_rng(10).standard_normal((nrows, 32)).astype(np.float32)
    out = torch.empty((ncols, 32), dtype=torch.float32, device="cuda")
    nsd.nsd_spmm_t(A.desc, A.csc, dev(G), 32, 1.0, out, A.workspace(32))
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    ref, mag = orc.spmm_t(D, G, 32)
    assert_mag_close(host(out), ref, mag, what="dense column")


# ---------------------------------------------------------- invariants

def test_bitwise_deterministic(nsd, operand):
    from paper_2303_07030_amd import synth
    d = synth.make("spmm", "small")
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    a = run_frob(nsd, A, d["B"], d["k"])
    b = run_frob(nsd, A, d["B"], d["k"])
    for x, y in zip(a, b):
        assert np.array_equal(np.asarray(x), np.asarray(y))


def test_seed_scales_gradients_exactly(nsd, operand):
    from paper_2303_07030_amd import synth
    d = synth.make("spmm", "small")
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    C1, L1, dA1, dB1 = run_frob(nsd, A, d["B"], d["k"], seed=1.0)
    C2, L2, dA2, dB2 = run_frob(nsd, A, d["B"], d["k"], seed=4.0)
    assert L1 == L2 and np.array_equal(C1, C2)
    assert np.array_equal(dA2, 4 * dA1) and np.array_equal(dB2, 4 * dB1)


def test_bilinear_dA_ignores_values_and_dH_ignores_H(nsd, operand):
    from paper_2303_07030_amd import synth
    d = synth.make("gnn", "small")
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"])
    A2 = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], 2 * d["val"] + 1)
    _, dA1, dH1 = run_bilinear(nsd, A, d["H"], d["G"], d["k"])
    _, dA2, _ = run_bilinear(nsd, A2, d["H"], d["G"], d["k"])
    _, _, dH3 = run_bilinear(nsd, A, 3 * d["H"] - 1, d["G"], d["k"])
    assert np.array_equal(dA1, dA2)   # the gradient on the pattern does not read A's values
    assert np.array_equal(dH1, dH3)   # a linear loss: dH does not depend on H


# ---------------------------------------------------------- BATAX Jacobian

def run_batax(nsd, A, beta):
    """J = beta A^T A through the C ABI: (rowptr, colind, val) on the host."""
    ws0 = torch.empty(256, dtype=torch.uint8, device="cuda")
    P = nsd.nsd_batax_pairs(A.desc, ws0)
    ws = torch.empty(nsd.nsd_batax_workspace_size(A.desc, P), dtype=torch.uint8, device="cuda")
    jrowptr = torch.full((A.ncols + 1,), -1, dtype=torch.int32, device="cuda")
    jcol = torch.full((max(P, 1),), -1, dtype=torch.int32, device="cuda")
    jval = torch.full((max(P, 1),), np.nan, dtype=torch.float32, device="cuda")
    nk = nsd.nsd_batax_jacobian(A.desc, beta, P, jrowptr, jcol, jval, ws)
    return host(jrowptr), host(jcol)[:nk], host(jval)[:nk]


def check_batax(orc, nrows, ncols, rowptr, colind, val, beta, got):
    D = oracle_dok(orc, nrows, ncols, rowptr, colind, val)
    rp, ci, v, m = orc.batax_jacobian(D, beta)
    grp, gci, gv = got
    assert np.array_equal(grp, rp), "J row pointers"
    assert np.array_equal(gci, ci), "J columns"
    assert_mag_close(gv, v, m, what="J values")


def test_batax_jacobian_edge(nsd, operand, orc):
    # power-law rows (one of 850 entries: 722K products), empty rows, a hot
    # column shared by half the rows, and a stored zero
    nrows, ncols, rowptr, colind, val = edge_pattern(17)
    val[10] = 0.0
    A = operand(nrows, ncols, rowptr, colind, val, build_csc=False)
    check_batax(orc, nrows, ncols, rowptr, colind, val, 0.75,
                run_batax(nsd, A, 0.75))


def test_batax_jacobian_small_workload(nsd, operand, orc):
    from paper_2303_07030_amd import synth
    d = synth.make("batax", "small")
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"], build_csc=False)
    got = run_batax(nsd, A, d["beta"])
    check_batax(orc, d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"], d["beta"], got)
    again = run_batax(nsd, A, d["beta"])  # bitwise reproducible
    for x, y in zip(got, again):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("case", ["empty", "no_entries", "single", "dense_row"])
def test_batax_jacobian_degenerate(nsd, operand, orc, case):
    rng = np.random.default_rng(3)
    if case == "empty":
        nrows, ncols = 0, 0
        rowptr, colind, val = np.zeros(1, np.int32), np.empty(0, np.int32), np.empty(0, np.float32)
    elif case == "no_entries":
        nrows, ncols = 5, 4
        rowptr, colind, val = np.zeros(6, np.int32), np.empty(0, np.int32), np.empty(0, np.float32)
    elif case == "single":
        nrows, ncols = 3, 5
        rowptr = np.array([0, 0, 1, 1], np.int32)
        colind, val = np.array([4], np.int32), np.array([-2.5], np.float32)
    else:
        nrows, ncols = 4, 300
        lengths = np.array([0, 300, 3, 0])
        rowptr, colind, val = make_csr(rng, nrows, ncols, lengths)
    A = operand(nrows, ncols, rowptr, colind, val, build_csc=False)
    got = run_batax(nsd, A, 2.0)
    if nrows == 0:
        assert np.array_equal(got[0], np.zeros(1, np.int32)) and len(got[1]) == 0
        return
    check_batax(orc, nrows, ncols, rowptr, colind, val, 2.0, got)


def max_row_terms(ncols, rowptr, colind):
    """Largest number of terms of a row of J = A^T A (the rows of A storing
    column j, their lengths summed)."""
    lens = np.diff(rowptr).astype(np.int64)
    rows = np.repeat(np.arange(len(lens)), lens)
    t = np.zeros(max(ncols, 1), np.int64)
    np.add.at(t, colind, lens[rows])
    return int(t.max()) if len(colind) else 0


def boundary_pattern(rng, terms):
    """Two rows of terms // 2 and terms - terms // 2 entries on columns
    [0, 1000), both storing column 0, and 300 sparse rows on columns
    [1000, 2000): the longest row of J (column 0's) has exactly `terms` terms."""
    ncols = 2000
    rows = []
    for n in (terms // 2, terms - terms // 2):
        c = rng.choice(np.arange(1, 1000), size=n - 1, replace=False)
        rows.append(np.sort(np.concatenate([[0], c])))
    for _ in range(300):
        rows.append(np.sort(rng.choice(np.arange(1000, 2000), size=int(rng.integers(0, 6)),
                                       replace=False)))
    rowptr = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32)
    colind = np.concatenate(rows).astype(np.int32)
    val = rng.standard_normal(len(colind)).astype(np.float32)
    return len(rows), ncols, rowptr, colind, val


def many_rows_pattern(rng):
    """40 rows of 12 entries sharing column 0 (column 0's row of J gathers 40
    rows, 480 terms) and sparse rows elsewhere."""
    rows = []
    for _ in range(40):
        rows.append(np.sort(np.concatenate([[0], rng.choice(np.arange(1, 2000), size=11,
                                                             replace=False)])))
    for _ in range(200):
        rows.append(np.sort(rng.choice(np.arange(1, 2000), size=int(rng.integers(0, 4)),
                                       replace=False)))
    rowptr = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32)
    colind = np.concatenate(rows).astype(np.int32)
    return len(rows), 2000, rowptr, colind, rng.standard_normal(len(colind)).astype(np.float32)


@pytest.mark.parametrize("case", ["small_workload", "edge", "dense_row", "cap", "cap_plus_one",
                                  "many_rows", "tall_column", "wide"])
def test_batax_row_path_equals_sort_path(nsd, operand, orc, case):
    """J built row by row in LDS (when no row of J has more than 512 terms)
    and by the two global sorts (forced with NSD_BATAX_ROW_CAP=0): the same
    bits, and the oracle's keys; likewise from a CSR descriptor without its
    row index (the row path derives it from rowptr)."""
    import os
    from paper_2303_07030_amd import synth
    rng = np.random.default_rng(31)
    if case == "small_workload":
        d = synth.make("batax", "small")
        nrows, ncols, rowptr, colind, val = d["nrows"], d["ncols"], d["rowptr"], d["colind"], \
            d["val"]
    elif case == "edge":
        nrows, ncols, rowptr, colind, val = edge_pattern(19)
    elif case == "dense_row":
        nrows, ncols = 4, 300
        rowptr, colind, val = make_csr(rng, nrows, ncols, np.array([0, 300, 3, 0]))
    elif case == "many_rows":
        # a row of J gathering 40 rows of A
        nrows, ncols, rowptr, colind, val = many_rows_pattern(rng)
        assert np.bincount(colind).max() == 40
    elif case == "tall_column":
        # column 5 stored by 150 short rows: a row of J gathering more rows
        # of A than a wave has lanes (still at most 512 terms)
        nrows, ncols = 300, 400
        rows = []
        for r in range(nrows):
            c = rng.choice(np.arange(6, ncols), size=int(rng.integers(0, 3)), replace=False)
            if r % 2 == 0:
                c = np.concatenate([c, [5]])
            rows.append(np.sort(c))
        rowptr = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32)
        colind = np.concatenate(rows).astype(np.int32)
        val = rng.standard_normal(len(colind)).astype(np.float32)
        assert np.bincount(colind)[5] == 150
    elif case == "wide":
        # 2^23 + 5 columns: the row path's 64-bit sort keys
        nrows, ncols = 300, (1 << 23) + 5
        hot = rng.integers(0, ncols, 40)  # columns shared by several rows
        rows = [np.unique(np.concatenate([rng.choice(hot, 3), rng.integers(0, ncols, 4)]))
                for _ in range(nrows)]
        rows[-1] = np.unique(np.concatenate([rows[-1], [ncols - 1]]))
        rowptr = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32)
        colind = np.concatenate(rows).astype(np.int32)
        val = rng.standard_normal(len(colind)).astype(np.float32)
    else:
        nrows, ncols, rowptr, colind, val = boundary_pattern(rng, 512 if case == "cap" else 513)
    mx = max_row_terms(ncols, rowptr, colind)
    if case == "cap":
        assert mx == 512
    if case in ("edge", "cap_plus_one"):
        assert mx > 512  # these take the sort path either way
    A = operand(nrows, ncols, rowptr, colind, val, build_csc=False)
    default = run_batax(nsd, A, 1.25)
    os.environ["NSD_BATAX_ROW_CAP"] = "0"
    try:
        forced = run_batax(nsd, A, 1.25)
    finally:
        del os.environ["NSD_BATAX_ROW_CAP"]
    for x, y in zip(default, forced):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))

    class Bare:  # rowptr, colind, val only
        desc = nsd.csr_desc(A.nrows, A.ncols, A.rowptr, None, A.colind, A.val)
    Bare.ncols = A.ncols
    bare = run_batax(nsd, Bare, 1.25)
    for x, y in zip(default, bare):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
    check_batax(orc, nrows, ncols, rowptr, colind, val, 1.25, default)


@pytest.mark.parametrize("row_cap", [None, "0"])
def test_batax_jacobian_rejects_wrong_pair_count(nsd, operand, row_cap, monkeypatch):
    """A wrong npairs is refused on the row path and on the sort path."""
    if row_cap is not None:
        monkeypatch.setenv("NSD_BATAX_ROW_CAP", row_cap)
    nrows, ncols, rowptr, colind, val = edge_pattern(18)
    A = operand(nrows, ncols, rowptr, colind, val, build_csc=False)
    ws0 = torch.empty(256, dtype=torch.uint8, device="cuda")
    P = nsd.nsd_batax_pairs(A.desc, ws0)
    assert P == int(np.sum(np.diff(rowptr).astype(np.int64) ** 2))
    ws = torch.empty(nsd.nsd_batax_workspace_size(A.desc, P + 1), dtype=torch.uint8,
                     device="cuda")
    jr = torch.empty(ncols + 1, dtype=torch.int32, device="cuda")
    jc = torch.empty(P + 1, dtype=torch.int32, device="cuda")
    jv = torch.empty(P + 1, dtype=torch.float32, device="cuda")
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_batax_jacobian(A.desc, 1.0, P + 1, jr, jc, jv, ws)
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG


# ------------------------------------------------- forward-mode tangent

def run_spmm_jvp(nsd, A, dAval, B, dB, k):
    C = torch.full((A.nrows, k), np.nan, dtype=torch.float32, device="cuda")
    dC = torch.full((A.nrows, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm_jvp(A.desc, dev(dAval), dev(B), dev(dB), k, C, dC, A.workspace(2 * k))
    return host(C), host(dC)


@pytest.mark.parametrize("k", [1, 3, 16, 64, 128, 256, 264])
def test_spmm_jvp(nsd, orc, edge_A, k):
    A, D, rows, colind = edge_A
    rng = np.random.default_rng(100 + k)
    dval = rng.standard_normal(A.nnz).astype(np.float32)
    B = rng.standard_normal((A.ncols, k)).astype(np.float32)
    dB = rng.standard_normal((A.ncols, k)).astype(np.float32)
    Cg, dCg = run_spmm_jvp(nsd, A, dval, B, dB, k)
    dD = orc.Dok((A.nrows, A.ncols), (rows, colind), dval)
    C, Cm, dC, dCm = orc.spmm_jvp(D, dD, B, dB, k)
    assert_mag_close(Cg, C, Cm, what="C")
    assert_mag_close(dCg, dC, dCm, what="dC")


def test_spmm_jvp_full_workload(nsd, operand, orc):
    from paper_2303_07030_amd import synth
    d = synth.make("spmm")
    k = d["k"]
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"], build_csc=False,
                k_hint=k)
    rng = np.random.default_rng(7)
    dval = rng.standard_normal(A.nnz).astype(np.float32)
    dB = rng.standard_normal(d["B"].shape).astype(np.float32)
    Cg, dCg = run_spmm_jvp(nsd, A, dval, d["B"], dB, k)
    rows = np.repeat(np.arange(d["nrows"], dtype=np.int32), np.diff(d["rowptr"]))
    D = orc.Dok((d["nrows"], d["ncols"]), (rows, d["colind"]), d["val"])
    dD = orc.Dok((d["nrows"], d["ncols"]), (rows, d["colind"]), dval)
    C, Cm, dC, dCm = orc.spmm_jvp(D, dD, d["B"], dB, k)
    assert_mag_close(Cg, C, Cm, what="C")
    assert_mag_close(dCg, dC, dCm, what="dC")


def test_spmm_jvp_batch_full_workload(nsd, operand, orc):
    # J V for five tangents on the full SpMM workload (a group of four and a
    # group of one): each tangent bit for bit the one-tangent kernel's, and
    # the last one against the oracle
    from paper_2303_07030_amd import synth
    d = synth.make("spmm")
    k, m = d["k"], 5
    A = operand(d["nrows"], d["ncols"], d["rowptr"], d["colind"], d["val"], build_csc=False,
                k_hint=k)
    rng = np.random.default_rng(8)
    TA = rng.standard_normal((m, A.nnz), dtype=np.float32)
    TB = rng.standard_normal((m,) + d["B"].shape, dtype=np.float32)
    C = torch.full((A.nrows, k), np.nan, dtype=torch.float32, device="cuda")
    dC = torch.full((m, A.nrows, k), np.nan, dtype=torch.float32, device="cuda")
    ws = torch.empty(nsd.nsd_spmm_jvp_batch_workspace_size(A.desc, k), dtype=torch.uint8,
                     device="cuda")
    nsd.nsd_spmm_jvp_batch(A.desc, m, dev(TA), dev(d["B"]), dev(TB), k, C, dC, ws)
    dC = host(dC)
    for t in range(m):
        Cg, dCg = run_spmm_jvp(nsd, A, TA[t], d["B"], TB[t], k)
        assert np.array_equal(dCg, dC[t]), f"tangent {t}"
    assert np.array_equal(Cg, host(C))
    rows = np.repeat(np.arange(d["nrows"], dtype=np.int32), np.diff(d["rowptr"]))
    D = orc.Dok((d["nrows"], d["ncols"]), (rows, d["colind"]), d["val"])
    dD = orc.Dok((d["nrows"], d["ncols"]), (rows, d["colind"]), TA[m - 1])
    _, _, dCo, dCm = orc.spmm_jvp(D, dD, d["B"], TB[m - 1], k)
    assert_mag_close(dC[m - 1], dCo, dCm, what="dC[4]")


# --------------------------------------------------- order-N CP gradient

def run_cpn(nsd, X, F, rank, seed=1.0):
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    dX = torch.full((max(X.nnz, 1),), np.nan, dtype=torch.float32, device="cuda")
    dF = [torch.full((d, rank), np.nan, dtype=torch.float32, device="cuda") for d in X.dims]
    nsd.nsd_loss_cpn(X.desc, [dev(f) for f in F], rank, seed, loss, dX, dF, X.workspace(rank))
    return host(loss)[0], in_input_order(X, host(dX)), [host(t) for t in dF]


def check_cpn(orc, dims, coords, val, F, rank, got, seed=1.0):
    D = orc.Dok(dims, coords, val)
    L, Lm = orc.cpn_loss(D, F, rank)
    R, Rm = orc.cpn_resid(D, F, rank, coords)
    Lg, dXg, dFg = got
    assert_mag_close(Lg, L, Lm, what="loss")
    assert_mag_close(dXg, seed * R, abs(seed) * Rm, what="residual")
    for m in range(len(dims)):
        g, gm = orc.cpn_grad(D, F, rank, m)
        assert_mag_close(dFg[m], seed * g, abs(seed) * gm, what=f"dF{m + 1}")


def test_loss_cpn_small_order4_workload(nsd, orc):
    from paper_2303_07030_amd import synth
    from paper_2303_07030_amd.operand import DeviceCooN
    d = synth.make("cp4", "small")
    X = DeviceCooN(d["dims"], d["coords"], d["val"], rank_hint=d["rank"])
    got = run_cpn(nsd, X, d["F"], d["rank"])
    check_cpn(orc, d["dims"], d["coords"], d["val"], d["F"], d["rank"], got)


@pytest.mark.parametrize("fibers", [True, False])
@pytest.mark.parametrize("dims,rank", [((9, 7, 5), 12), ((6, 5, 4, 7, 3), 8),
                                       ((4, 3, 5, 2, 3, 4), 5), ((40, 3, 2, 50), 64),
                                       ((30, 2, 2, 2), 256), ((3, 4, 200, 5), 32)])
def test_loss_cpn_orders_and_ranks(nsd, orc, dims, rank, fibers):
    # skewed and tiny modes (long slices, chunked), scalar ranks (5), wide
    # ranks (256: a full wave per slot), empty slices
    from paper_2303_07030_amd.operand import DeviceCooN
    rng = np.random.default_rng(len(dims) * 100 + rank)
    size = int(np.prod(dims))
    nnz = min(size // 2, 4000)
    keys = rng.choice(size, size=nnz, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(keys, dims)]
    val = rng.standard_normal(nnz).astype(np.float32)
    F = [(0.3 * rng.standard_normal((dd, rank))).astype(np.float32) for dd in dims]
    X = DeviceCooN(dims, coords, val, rank_hint=rank, item_len=16, fibers=fibers)
    got = run_cpn(nsd, X, F, rank, seed=0.5)
    check_cpn(orc, dims, coords, val, F, rank, got, seed=0.5)


def test_loss_cpn_fibers_in_any_entry_order(nsd, orc):
    """The fiber level regroups by runs of equal coordinate, so entries in an
    order with short runs (mode indexes built over an unsorted input, not the
    operand's lexicographic storage) give the same values to the bar."""
    from paper_2303_07030_amd.operand import DeviceCooN
    rng = np.random.default_rng(77)
    dims, rank = (6, 5, 40, 7), 16
    size = int(np.prod(dims))
    keys = rng.choice(size, size=2500, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(keys, dims)]
    val = rng.standard_normal(2500).astype(np.float32)
    F = [(0.3 * rng.standard_normal((d, rank))).astype(np.float32) for d in dims]
    X = DeviceCooN(dims, coords, val, rank_hint=rank, item_len=8, fibers=True)
    # scramble the entry order of every mode index within its slices: the
    # per-entry arrays are permuted together, slices (and the plans) stay
    keep = []
    for m in range(len(dims)):
        md, arrs = X.desc.mode[m], X.modes[m]
        segptr = host(arrs["segptr"])
        pi = np.concatenate([segptr[i] + rng.permutation(segptr[i + 1] - segptr[i])
                             for i in range(dims[m])]).astype(np.int64)
        new = {f: dev(host(arrs[f])[: X.nnz][pi]) for f in ("perm", "val")}
        new["idx"] = [dev(host(t)[: X.nnz][pi]) for t in arrs["idx"]]
        md.perm, md.val = new["perm"].data_ptr(), new["val"].data_ptr()
        for o, t in enumerate(new["idx"]):
            md.idx[o] = t.data_ptr()
        keep.append(new)
    got = run_cpn(nsd, X, F, rank)
    check_cpn(orc, dims, coords, val, F, rank, got)


def test_loss_cpn_order3_equals_cp(nsd, orc):
    """The order-N path on an order-3 tensor gives the order-3 path's bits
    where both use the same plans (same summation orders)."""
    from paper_2303_07030_amd import synth
    from paper_2303_07030_amd.operand import DeviceCoo3, DeviceCooN
    d = synth.make("cp", "small")
    F = [d["F1"], d["F2"], d["F3"]]
    X3 = DeviceCoo3(d["dims"], d["i"], d["j"], d["k"], d["val"], item_len=24)
    XN = DeviceCooN(d["dims"], [d["i"], d["j"], d["k"]], d["val"], item_len=24, fibers=False)
    a = run_cp(nsd, X3, F, d["rank"])
    b = run_cpn(nsd, XN, F, d["rank"])
    check_cpn(orc, d["dims"], [d["i"], d["j"], d["k"]], d["val"], F, d["rank"], b)
    assert np.array_equal(a[1], b[1])
    for x, y in zip(a[2], b[2]):
        assert np.array_equal(x, y)


# --------------------------------------------------- VJP of the product

@pytest.mark.parametrize("k,ones", [(1, False), (1, True), (16, False), (64, False),
                                    (300, False)])
def test_spmm_vjp(nsd, orc, edge_A, k, ones):
    # k = 300 is beyond the fused column pass: SDDMM then A^T G
    A, D, rows, cols = edge_A
    rng = np.random.default_rng(300 + k)
    X = rng.standard_normal((A.ncols, k)).astype(np.float32)
    G = None if ones else rng.standard_normal((A.nrows, k)).astype(np.float32)
    dA = torch.full((A.nnz,), np.nan, dtype=torch.float32, device="cuda")
    dX = torch.full((A.ncols, k), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmm_vjp(A.desc, A.csc, dev(X), None if G is None else dev(G), k, dA, dX,
                     A.workspace(k))
    ref, mag = orc.sddmm(D, G, X, k, rows, cols)
    assert_mag_close(host(dA), ref, mag, what=f"dA k={k}")
    ref, mag = orc.spmm_t(D, G, k)
    assert_mag_close(host(dX), ref, mag, what=f"dX k={k}")


def test_spmv_vjp(nsd, orc, edge_A):
    A, D, rows, cols = edge_A
    rng = np.random.default_rng(5)
    x = rng.standard_normal(A.ncols).astype(np.float32)
    gy = rng.standard_normal(A.nrows).astype(np.float32)
    dA = torch.full((A.nnz,), np.nan, dtype=torch.float32, device="cuda")
    dx = torch.full((A.ncols,), np.nan, dtype=torch.float32, device="cuda")
    nsd.nsd_spmv_vjp(A.desc, A.csc, dev(x), dev(gy), dA, dx, A.workspace(1))
    ref, mag = orc.sddmm(D, gy.reshape(-1, 1), x.reshape(-1, 1), 1, rows, cols)
    assert_mag_close(host(dA), ref, mag, what="dA")
    ref, mag = orc.spmm_t(D, gy.reshape(-1, 1), 1)
    assert_mag_close(host(dx), ref[:, 0], mag[:, 0], what="dx")


# ---------------------------------------------------------- COO validator

@pytest.mark.parametrize("order", [2, 3, 6])
def test_validate_coo(nsd, order):
    rng = np.random.default_rng(order)
    dims = (7, 300, 5, 11, 3, 4)[:order]
    size = int(np.prod(dims))
    nnz = min(size // 2, 5000)
    keys = rng.choice(size, size=nnz, replace=False)
    coords = [c.astype(np.int32) for c in np.unravel_index(keys, dims)]

    def check(cs, unique=True):
        ws = torch.empty(nsd.nsd_validate_coo_workspace_size(dims, len(cs[0])),
                         dtype=torch.uint8, device="cuda")
        nsd.nsd_validate_coo(dims, len(cs[0]), [dev(c) for c in cs], unique, ws)

    check(coords)                                   # distinct keys in range
    dup = [np.concatenate([c, c[[17]]]) for c in coords]
    with pytest.raises(nsd.NsdError) as e:
        check(dup)
    assert e.value.status == nsd.NSD_ERR_DUPLICATE
    check(dup, unique=False)                        # duplicates allowed when not asked
    bad = [c.copy() for c in coords]
    bad[order - 1][123] = dims[order - 1]
    with pytest.raises(nsd.NsdError) as e:
        check(bad)
    assert e.value.status == nsd.NSD_ERR_BAD_FORMAT
    bad[order - 1][123] = -1
    with pytest.raises(nsd.NsdError) as e:
        check(bad, unique=False)
    assert e.value.status == nsd.NSD_ERR_BAD_FORMAT
    check([c[:1] for c in coords])                  # a single entry


@pytest.mark.parametrize("order", [3, 4])
def test_loss_cp_empty_tensor(nsd, order):
    # no stored entries: the loss is 0 and every factor gradient is 0
    from paper_2303_07030_amd.operand import DeviceCoo3, DeviceCooN
    dims = (5, 7, 3, 4)[:order]
    rank = 8
    empty = np.empty(0, np.int32)
    F = [np.ones((d, rank), np.float32) for d in dims]
    if order == 3:
        X = DeviceCoo3(dims, empty, empty, empty, np.empty(0, np.float32), rank_hint=rank)
        L, dX, dF = run_cp(nsd, X, F, rank)
    else:
        X = DeviceCooN(dims, [empty] * order, np.empty(0, np.float32), rank_hint=rank)
        L, dX, dF = run_cpn(nsd, X, F, rank)
    assert L == 0.0 and dX.size == 0
    for g in dF:
        assert np.array_equal(g, np.zeros_like(g))
