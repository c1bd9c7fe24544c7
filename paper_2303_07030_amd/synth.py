"""Seeded synthetic inputs shaped like the paper's sparse workloads.

This module only *draws inputs*: sparsity patterns, values and dense operands.
It holds none of the gradient arithmetic, so the oracle and the HIP path can
both be fed from it without sharing any of the method.

The paper evaluates on SuiteSparse matrices and on random matrices of varying
density and dimension (Section "Experimental Results", Table of real-world
matrices and the synthetic sweeps).  Those matrices are not available here, so
every workload is synthetic, at the shapes below:

  spmv  1,000 x 1,000 CSR, 10,000 uniform-random positions, values N(0,1);
        dense x (1,000) N(0,1).
  spmm  100,000 x 100,000 CSR, 1M nnz, row lengths from a Zipf(s=1.1) profile
        capped at 5,000, uniform columns, values N(0,1); dense B 100,000 x 64.
  mf    1,000,000 x 500,000 COO, 50M unique (row, col) pairs drawn i.i.d. from
        truncated Zipf(1.1) on each axis, values U(1,5); U, V with 128 columns
        ~ N(0, 0.1^2).
  cp    10,000^3 COO 3-tensor, 20M unique uniform coordinates, values N(0,1);
        three 10,000 x 32 factors ~ N(0, 0.1^2).
  gnn   2,400,000-node power-law graph, 60M edges (out-degree Zipf profile
        s=1.05), weights U[0,1); H and G 2,400,000 x 256 ~ N(0,1).
  cp4   1,000^4 COO 4-tensor, 20M distinct uniform coordinates, values
        N(0,1); four 1,000 x 32 factors ~ N(0, 0.1^2) (the CP workload at
        order 4).
  batax 100,000 x 100,000 CSR, 1M entries at uniform random positions
        (multinomial row lengths, distinct uniform columns), values N(0,1),
        beta = 1.5 (the Jacobian beta A^T A of Example 5's kernel).

Seeds: numpy PCG64 streams from SeedSequence(entropy=230307030,
spawn_key=(workload id, replicate)); each workload spawns five child streams
used in a fixed order: pattern, values, dense 1, dense 2, dense 3.

Zipf readings (the workload text only says "Zipf(s)"):
  * row-length profiles: l_r = min(cap, floor(c * r^-s)) over ranks
    r = 1..nrows with c found by bisection so that the lengths sum to nnz;
    the remainder goes +1 to the uncapped ranks with the largest fractional
    part; ranks map to row ids through a seeded permutation.
  * per-entry indices (mf): i.i.d. draws from the truncated discrete Zipf on
    ranks 1..N by inverse CDF, with a seeded rank -> id permutation per axis;
    pairs are deduplicated by first occurrence.
  * N(0, 0.1) means standard deviation 0.1.
"""
from __future__ import annotations

import sys
import time

import numpy as np

ENTROPY = 230307030
VERBOSE = False  # progress lines on stderr for the multi-minute workloads


def _say(msg):
    if VERBOSE:
        print(f"[synth {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)
WORKLOAD_IDS = {"spmv": 1, "spmm": 2, "mf": 3, "cp": 4, "gnn": 5, "batax": 6, "cp4": 7}

# Full-size workloads and smaller variants of the same recipes that the
# oracle finishes in seconds (they still span many tiles and ragged tails).
PRESETS = {
    "spmv": {"full": dict(nrows=1000, ncols=1000, nnz=10_000)},
    "spmm": {
        "full": dict(n=100_000, nnz=1_000_000, s=1.1, cap=5000, k=64),
        "small": dict(n=3000, nnz=30_000, s=1.1, cap=600, k=64),
    },
    "mf": {
        "full": dict(nrows=1_000_000, ncols=500_000, nnz=50_000_000, s=1.1, k=128),
        "small": dict(nrows=4000, ncols=2500, nnz=60_000, s=1.1, k=128),
    },
    "cp": {
        "full": dict(dim=10_000, nnz=20_000_000, rank=32),
        "small": dict(dim=60, nnz=25_000, rank=32),
    },
    "gnn": {
        "full": dict(n=2_400_000, nnz=60_000_000, s=1.05, k=256),
        "small": dict(n=5000, nnz=70_000, s=1.05, k=256),
    },
    "batax": {
        "full": dict(n=100_000, nnz=1_000_000, beta=1.5),
        "small": dict(n=2000, nnz=20_000, beta=1.5),
    },
    "cp4": {
        "full": dict(dims=(1000, 1000, 1000, 1000), nnz=20_000_000, rank=32),
        "small": dict(dims=(24, 20, 16, 30), nnz=30_000, rank=32),
    },
}


def streams(workload: str, replicate: int = 0):
    """Five independent generators: pattern, values, dense1, dense2, dense3."""
    ss = np.random.SeedSequence(entropy=ENTROPY,
                                spawn_key=(WORKLOAD_IDS[workload], replicate))
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(5)]


def zipf_lengths(nrows: int, nnz: int, s: float, cap: int) -> np.ndarray:
    """Row-length profile by rank: min(cap, floor(c r^-s)) summing to nnz."""
    if cap * nrows < nnz:
        raise ValueError("cap * nrows < nnz")
    w = np.arange(1, nrows + 1, dtype=np.float64) ** (-s)

    def total(c):
        return np.minimum(cap, c * w).sum()

    lo, hi = 0.0, cap / w[-1]
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if total(mid) <= nnz:
            lo = mid
        else:
            hi = mid
    real = np.minimum(cap, lo * w)
    lens = np.floor(real).astype(np.int64)
    rem = nnz - int(lens.sum())
    uncapped = np.nonzero(real < cap)[0]
    frac = real[uncapped] - lens[uncapped]
    order = np.lexsort((uncapped, -frac))  # largest fraction first, then rank
    lens[uncapped[order[:rem]]] += 1
    assert int(lens.sum()) == nnz and lens.max() <= cap
    return lens


def _rows_without_replacement(rng, lengths: np.ndarray, ncols: int):
    """Sorted, distinct uniform columns for each row; returns rowptr, colind."""
    nrows = lengths.shape[0]
    rowptr = np.zeros(nrows + 1, dtype=np.int64)
    np.cumsum(lengths, out=rowptr[1:])
    colind = np.empty(int(rowptr[-1]), dtype=np.int32)
    big = min(4096, max(1, ncols // 8))
    small_rows = np.nonzero((lengths > 0) & (lengths <= big))[0]
    big_rows = np.nonzero(lengths > big)[0]
    # short rows: all at once, redraw collisions until every row is distinct;
    # after the first round only the rows that had a collision are re-checked
    ls = lengths[small_rows]
    rows_rep = np.repeat(small_rows.astype(np.int64), ls)
    cols = rng.integers(0, ncols, size=rows_rep.shape[0], dtype=np.int64)
    active = np.arange(rows_rep.shape[0], dtype=np.int64)
    while active.shape[0]:
        key = rows_rep[active] * ncols + cols[active]
        order = np.argsort(key, kind="stable")
        ks = key[order]
        dup = np.zeros(active.shape[0], dtype=bool)
        dup[order[1:][ks[1:] == ks[:-1]]] = True
        ndup = int(dup.sum())
        if ndup == 0:
            break
        pos = active[dup]
        cols[pos] = rng.integers(0, ncols, size=ndup, dtype=np.int64)
        bad = np.zeros(nrows, dtype=bool)
        bad[rows_rep[pos]] = True
        active = np.nonzero(bad[rows_rep])[0]
    key = rows_rep * ncols + cols
    cols_sorted = (np.sort(key) % ncols).astype(np.int32)
    starts = np.zeros(small_rows.shape[0], dtype=np.int64)
    if ls.shape[0] > 1:
        np.cumsum(ls[:-1], out=starts[1:])
    offs = np.arange(rows_rep.shape[0], dtype=np.int64) - np.repeat(starts, ls)
    pos = np.repeat(rowptr[small_rows], ls) + offs
    colind[pos] = cols_sorted
    _say(f"short rows placed; {len(big_rows)} long rows to draw")
    # long rows one by one (numpy picks a set-based or permutation method)
    for r in big_rows:
        c = rng.choice(ncols, size=int(lengths[r]), replace=False)
        c.sort()
        colind[rowptr[r]:rowptr[r + 1]] = c
    return rowptr.astype(np.int32), colind


def _power_law_csr(rng, n: int, nnz: int, s: float, cap: int):
    lens_by_rank = zipf_lengths(n, nnz, s, cap)
    row_of_rank = rng.permutation(n)
    lengths = np.empty(n, dtype=np.int64)
    lengths[row_of_rank] = lens_by_rank
    return _rows_without_replacement(rng, lengths, n)


def _normal(rng, shape, std=1.0):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def _zipf_cdf(N: int, s: float):
    """Truncated Zipf CDF over ranks 1..N plus a guide table for inversion."""
    cdf = np.cumsum(np.arange(1, N + 1, dtype=np.float64) ** (-s))
    cdf /= cdf[-1]
    # guide[b] = first rank index whose CDF exceeds b / M (M a power of two,
    # so u * M and b / M are exact and the bracket below is exact)
    M = 1 << 22
    guide = np.searchsorted(cdf, np.arange(M + 1, dtype=np.float64) / M, side="right")
    return cdf, guide


def _zipf_ids(rng, u_count: int, table, rank_to_id: np.ndarray):
    """Inverse-CDF draws: the first rank whose CDF exceeds u (bracketed by
    the guide table, then bisected), mapped through rank_to_id."""
    cdf, guide = table
    N = cdf.shape[0]
    M = guide.shape[0] - 1
    u = rng.random(u_count)
    b = (u * M).astype(np.int64)
    lo, hi = guide[b], guide[b + 1]
    act = np.nonzero(lo < hi)[0]
    while act.shape[0]:
        l, h = lo[act], hi[act]
        mid = (l + h) >> 1
        right = cdf[mid] <= u[act]
        lo[act] = np.where(right, mid + 1, l)
        hi[act] = np.where(right, h, mid)
        act = act[lo[act] < hi[act]]
    return rank_to_id[np.minimum(lo, N - 1)]


def _first_unique(keys: np.ndarray):
    """np.unique(keys, return_index=True) (sorted distinct keys and the index
    of each one's first occurrence) via one sort of (key, index) packed into
    a uint64 when both fit."""
    n = keys.shape[0]
    ib = max(1, int(n - 1).bit_length())
    if n == 0 or int(keys.min()) < 0 or int(keys.max()).bit_length() + ib > 64:
        return np.unique(keys, return_index=True)
    c = (keys.astype(np.uint64) << np.uint64(ib)) | np.arange(n, dtype=np.uint64)
    c.sort()
    k = (c >> np.uint64(ib)).astype(np.int64)
    head = np.ones(n, dtype=bool)
    head[1:] = k[1:] != k[:-1]
    first = (c[head] & np.uint64((1 << ib) - 1)).astype(np.int64)
    return k[head], first


def _dedupe_first(draw_batch, nnz: int):
    """Keep the first nnz distinct int64 keys in first-occurrence order."""
    seen = np.empty(0, dtype=np.int64)
    out = []
    count = 0
    while count < nnz:
        _say(f"distinct keys {count}/{nnz}")
        keys = draw_batch()
        uk, first = _first_unique(keys)
        if seen.shape[0]:
            pos = np.minimum(np.searchsorted(seen, uk), seen.shape[0] - 1)
            new = seen[pos] != uk
            uk, first = uk[new], first[new]
        take = min(uk.shape[0], nnz - count)
        order = np.argsort(first, kind="stable")[:take]
        out.append(uk[order])
        count += take
        if count < nnz:
            seen = np.sort(np.concatenate([seen, uk[order]]), kind="stable")
    return np.concatenate(out)


# ---------------------------------------------------------------- workloads

def make_spmv(nrows=1000, ncols=1000, nnz=10_000, replicate=0):
    g_pat, g_val, g_d1, _, _ = streams("spmv", replicate)
    keys = np.sort(g_pat.choice(nrows * ncols, size=nnz, replace=False))
    row = (keys // ncols).astype(np.int32)
    colind = (keys % ncols).astype(np.int32)
    rowptr = np.zeros(nrows + 1, dtype=np.int32)
    np.cumsum(np.bincount(row, minlength=nrows), out=rowptr[1:])
    return dict(workload="spmv", nrows=nrows, ncols=ncols, rowptr=rowptr,
                colind=colind, val=_normal(g_val, nnz), x=_normal(g_d1, ncols))


def make_spmm(n=100_000, nnz=1_000_000, s=1.1, cap=5000, k=64, replicate=0):
    g_pat, g_val, g_d1, _, _ = streams("spmm", replicate)
    rowptr, colind = _power_law_csr(g_pat, n, nnz, s, cap)
    return dict(workload="spmm", nrows=n, ncols=n, rowptr=rowptr, colind=colind,
                val=_normal(g_val, nnz), B=_normal(g_d1, (n, k)), k=k)


def make_mf(nrows=1_000_000, ncols=500_000, nnz=50_000_000, s=1.1, k=128,
            replicate=0, batch=20_000_000):
    g_pat, g_val, g_d1, g_d2, _ = streams("mf", replicate)
    row_ids = g_pat.permutation(nrows)
    col_ids = g_pat.permutation(ncols)
    batch = min(batch, max(4 * nnz, 1024))

    cdf_r, cdf_c = _zipf_cdf(nrows, s), _zipf_cdf(ncols, s)

    def draw():
        r = _zipf_ids(g_pat, batch, cdf_r, row_ids).astype(np.int64)
        c = _zipf_ids(g_pat, batch, cdf_c, col_ids).astype(np.int64)
        return r * ncols + c

    keys = _dedupe_first(draw, nnz)
    val = (np.float32(1.0) + np.float32(4.0) * g_val.random(nnz, dtype=np.float32))
    return dict(workload="mf", nrows=nrows, ncols=ncols,
                row=(keys // ncols).astype(np.int32),
                col=(keys % ncols).astype(np.int32), val=val,
                U=_normal(g_d1, (nrows, k), 0.1), V=_normal(g_d2, (ncols, k), 0.1),
                k=k)


def make_cp(dim=10_000, nnz=20_000_000, rank=32, replicate=0):
    g_pat, g_val, g_d1, g_d2, g_d3 = streams("cp", replicate)
    draws = nnz + nnz // 20 + 64

    def draw():
        i = g_pat.integers(0, dim, size=draws, dtype=np.int64)
        j = g_pat.integers(0, dim, size=draws, dtype=np.int64)
        kk = g_pat.integers(0, dim, size=draws, dtype=np.int64)
        return (i * dim + j) * dim + kk

    keys = _dedupe_first(draw, nnz)
    return dict(workload="cp", dims=(dim, dim, dim),
                i=(keys // (dim * dim)).astype(np.int32),
                j=((keys // dim) % dim).astype(np.int32),
                k=(keys % dim).astype(np.int32),
                val=_normal(g_val, nnz),
                F1=_normal(g_d1, (dim, rank), 0.1), F2=_normal(g_d2, (dim, rank), 0.1),
                F3=_normal(g_d3, (dim, rank), 0.1), rank=rank)


def make_gnn(n=2_400_000, nnz=60_000_000, s=1.05, k=256, replicate=0):
    g_pat, g_val, g_d1, g_d2, _ = streams("gnn", replicate)
    rowptr, colind = _power_law_csr(g_pat, n, nnz, s, n)
    return dict(workload="gnn", nrows=n, ncols=n, rowptr=rowptr, colind=colind,
                val=g_val.random(nnz, dtype=np.float32),
                H=_normal(g_d1, (n, k)), G=_normal(g_d2, (n, k)), k=k)


def make_batax(n=100_000, nnz=1_000_000, beta=1.5, replicate=0):
    """A square CSR with entries at uniform random positions (each entry's
    row uniform, distinct uniform columns per row), values N(0,1)."""
    g_pat, g_val, g_d1, _, _ = streams("batax", replicate)
    lengths = g_pat.multinomial(nnz, np.full(n, 1.0 / n))
    rowptr, colind = _rows_without_replacement(g_pat, lengths.astype(np.int64), n)
    return dict(workload="batax", nrows=n, ncols=n, rowptr=rowptr, colind=colind,
                val=_normal(g_val, nnz), x=_normal(g_d1, n), beta=beta)


def make_cpn(dims, nnz, rank, workload="cp4", replicate=0):
    """An order-N tensor with distinct uniform coordinates (first occurrence
    of uniform draws), values N(0,1), factors N(0, 0.1^2); the order-N form of
    the CP workload."""
    g_pat, g_val, g_d1, g_d2, _ = streams(workload, replicate)
    dims = tuple(int(x) for x in dims)
    draws = nnz + nnz // 20 + 64

    def draw():
        key = np.zeros(draws, dtype=np.int64)
        for d in dims:
            key = key * d + g_pat.integers(0, d, size=draws, dtype=np.int64)
        return key

    keys = _dedupe_first(draw, nnz)
    coords = []
    for d in reversed(dims):
        coords.append((keys % d).astype(np.int32))
        keys = keys // d
    coords = coords[::-1]
    F = [_normal(g_d1 if n % 2 == 0 else g_d2, (d, rank), 0.1) for n, d in enumerate(dims)]
    return dict(workload=workload, dims=dims, coords=coords, val=_normal(g_val, nnz), F=F,
                rank=rank)


def make_cp4(dims=(1000, 1000, 1000, 1000), nnz=20_000_000, rank=32, replicate=0):
    return make_cpn(dims, nnz, rank, "cp4", replicate)


MAKERS = {"spmv": make_spmv, "spmm": make_spmm, "mf": make_mf, "cp": make_cp,
          "gnn": make_gnn, "batax": make_batax, "cp4": make_cp4}


def make(workload: str, size: str = "full", replicate: int = 0, **over):
    params = dict(PRESETS[workload][size])
    params.update(over)
    _say(f"generating {workload} ({size})")
    d = MAKERS[workload](replicate=replicate, **params)
    _say(f"generated {workload} ({size})")
    return d
