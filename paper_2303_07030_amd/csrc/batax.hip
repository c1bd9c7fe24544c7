// Jacobian of the BATAX kernel f(j) = sum_{i,k} beta A(i,j) A(i,k) x(k) with
// respect to x:  J = beta A^T A, a sparse matrix whose pattern is not an
// input's (Example 5; the matrix-kernel benchmarks of Section 7).
//
// The paper's differentiated, normalised program inserts, for every stored
// row r of A, the outer product r x r into the result dictionary.  Here that
// is expand / sort / reduce:
//   1. every ordered pair (p, q) of stored entries of one row becomes a term
//      (j, k, beta * a_p * a_q) with j = col(p), k = col(q); rows are laid
//      out in order, pairs row-major inside a row;
//   2. the terms are sorted stably by k, then stably by j (two radix sorts),
//      so a run of equal (j, k) keeps its terms in row order;
//   3. runs become the keys of J (run heads, a scan); J's row pointers come
//      from the runs' j, its columns from their k;
//   4. the values are the run sums, one thread per run adding its terms in
//      row order in fp64 and rounding once: no float atomics, bitwise
//      reproducible.  (A run is as long as the number of rows two columns
//      share, at most a column's length; a pathologically dense column makes
//      its diagonal run a serial tail, which the fixed order accepts.)
// Keys are structural: a pair whose product is 0 keeps its key, as the
// dictionary insert of the paper's program does.
//
// When every row of J has at most a few hundred terms (the common case), a
// second path builds J row by row instead, the GPU form of the per-row
// dictionary: row j gathers the rows i of A that store column j (A's CSC,
// ascending i); one wave lays their terms (beta a_ij) a_ik out in LDS in
// that order, sorts them stably by k (a bitonic sort of (k, position)
// pairs), and sums each run of equal k in fp64 in order.  These are the
// same terms, summed in the same order, as the sort path's, so both give
// the same bits; the row path reads A and writes J a few times instead of
// sorting every term twice through HBM.
#include <algorithm>
#include <cstdlib>
#include <cstring>

#include "nsd_internal.hpp"

namespace nsd {

constexpr int kBataxThreads = 256;
constexpr int64_t kBataxMaxPairs = 1LL << 30;  // positions stay in int32

static int64_t bgrid(int64_t n) { return ceil_div(n > 0 ? n : 1, kBataxThreads); }

__global__ void row_pairs_kernel(int32_t nrows, const int32_t *rowptr, int32_t *sq) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= nrows) return;
    const int32_t len = rowptr[i + 1] - rowptr[i];
    sq[i] = len * len;
}

__global__ void pairs_total_kernel(int32_t nrows, const int32_t *rowptr,
                                   unsigned long long *total) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    unsigned long long v = 0;
    if (i < nrows) {
        const unsigned long long len = (unsigned long long)(rowptr[i + 1] - rowptr[i]);
        v = len * len;
    }
    // integer sums are exact in any order: the waves' sums, then one atomic
    // per block
    __shared__ unsigned long long part[kBataxThreads / kWave];
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long b = 0;
        for (int w = 0; w < kBataxThreads / kWave; ++w) b += part[w];
        if (b) atomicAdd(total, b);
    }
}

// Term t of row i: the pair (p, q) = (u / len, u % len) of the row's
// entries, u = t - off[i]; the row is found by binary search over off.
__global__ void expand_pairs_kernel(int64_t npairs, int32_t nrows, const int32_t *off,
                                    const int32_t *rowptr, const int32_t *colind,
                                    const float *val, float beta, int32_t *key_j,
                                    int32_t *key_k, float *term) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= npairs) return;
    int32_t lo = 0, hi = nrows - 1;  // last row with off[row] <= t (rows of length 0 share off)
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo + 1) / 2;
        if (off[mid] <= t) lo = mid;
        else hi = mid - 1;
    }
    const int32_t b = rowptr[lo];
    const int32_t len = rowptr[lo + 1] - b;
    const int32_t u = (int32_t)(t - off[lo]);
    const int32_t p = b + u / len, q = b + u % len;
    key_j[t] = colind[p];
    key_k[t] = colind[q];
    term[t] = (beta * val[p]) * val[q];
}

__global__ void gather_keys_kernel(int64_t n, const int32_t *perm, const int32_t *src,
                                   int32_t *dst) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n) dst[t] = src[perm[t]];
}

__global__ void pair_heads_kernel(int64_t n, const int32_t *js, const int32_t *ks, int32_t *head) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n) return;
    head[t] = (t == 0 || js[t] != js[t - 1] || ks[t] != ks[t - 1]) ? 1 : 0;
}

// run[t] = index of the run holding sorted term t; heads name J's keys.
__global__ void runs_kernel(int64_t n, const int32_t *head, const int32_t *pos,
                            const int32_t *js, const int32_t *ks, int32_t *run, int32_t *run_j,
                            int32_t *jcolind) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n) return;
    run[t] = pos[t] + head[t] - 1;
    if (head[t]) {
        run_j[pos[t]] = js[t];
        jcolind[pos[t]] = ks[t];
    }
}

// jval[r] = sum of the terms of run r (sorted positions runptr[r] ..
// runptr[r+1], terms reached through perm), in order, in fp64.
__global__ void run_sums_kernel(int32_t nruns, const int32_t *runptr, const int32_t *perm,
                                const float *term, float *jval) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= nruns) return;
    double s = 0.0;
    for (int32_t t = runptr[r]; t < runptr[r + 1]; ++t) s += (double)term[perm[t]];
    jval[r] = (float)s;
}

// ------------------------------------------------------- row path

constexpr int kRowCap = 512;     // terms of one row of J held in LDS (a power of two)
constexpr int kRowThreads = 64;  // one wave per row of J (the compaction's block)
// Rows of J per block of the row kernel, one wave each (build-time knob
// NSD_BATAX_ROW_WAVES).  The waves share nothing but the block: each has
// its own LDS region and synchronises only itself.  Measured on MI355X on
// the uniform 1M-entry input: 207 us with one wave per block, 218 / 220 /
// 230 us with 2 / 4 / 8 (what raised the waves per CU was sizing the LDS
// regions by the largest row instead of the row cap: 344 us before).
#ifdef NSD_BATAX_ROW_WAVES
constexpr int kRowWaves = NSD_BATAX_ROW_WAVES;
#else
constexpr int kRowWaves = 1;
#endif
constexpr int kRowBlock = kRowWaves * kWave;
// The row path takes rows of J with at most this many terms: kRowCap, or
// less when the environment says so (NSD_BATAX_ROW_CAP; 0 keeps every call
// on the sort path).
static int row_cap() {
    const char *e = std::getenv("NSD_BATAX_ROW_CAP");
    if (!e) return kRowCap;
    const int v = std::atoi(e);
    return v < 0 ? 0 : std::min(v, kRowCap);
}

// row[p] = the row of A holding CSR slot p: the last r with rowptr[r] <= p
// (an empty row shares its start with the next); for a CSR given without
// its row index.
__global__ void slot_rows_kernel(int64_t n, int32_t nrows, const int32_t *rowptr,
                                 int32_t *row) {
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= n) return;
    const int32_t p = (int32_t)c;
    int32_t lo = 0, hi = nrows - 1;
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo + 1) / 2;
        if (rowptr[mid] <= p) lo = mid;
        else hi = mid - 1;
    }
    row[c] = lo;
}

// len[c] = the length of the row of A holding CSC slot c: the terms that
// entry contributes to its column's row of J.
__global__ void slot_len_kernel(int64_t n, const int32_t *crow, const int32_t *rowptr,
                                int32_t *len) {
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= n) return;
    const int32_t i = crow[c];
    len[c] = rowptr[i + 1] - rowptr[i];
}

// From the exclusive prefix sums `pre` of those lengths over the CSC slots
// (nnz of them, their total at *total): toff[j] = the first term of row j of
// J, and the largest row's term count to mx[0], the longest column of A to
// mx[1] (integer maxima: any order).
__global__ void row_terms_kernel(int32_t ncols, int32_t nnz, const int32_t *colptr,
                                 const int32_t *pre, const int32_t *total, int32_t *toff,
                                 int32_t *mx) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int32_t t = 0, nr = 0;
    if (j < ncols) {
        const int32_t c0 = colptr[j], c1 = colptr[j + 1];
        const int32_t b = c0 < nnz ? pre[c0] : *total;
        const int32_t e = c1 < nnz ? pre[c1] : *total;
        toff[j] = b;
        t = e - b;
        nr = c1 - c0;
    }
    // the waves' maxima, then the block's, then one atomic each per block
    // (atomics of every wave on the same two words serialise: 39 us for
    // 100K columns)
    __shared__ int32_t bt[kBataxThreads / kWave], bn[kBataxThreads / kWave];
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) {
        t = max(t, __shfl_xor(t, m, kWave));
        nr = max(nr, __shfl_xor(nr, m, kWave));
    }
    if ((threadIdx.x & (kWave - 1)) == 0) {
        bt[threadIdx.x / kWave] = t;
        bn[threadIdx.x / kWave] = nr;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kBataxThreads / kWave; ++w) {
            t = max(t, bt[w]);
            nr = max(nr, bn[w]);
        }
        if (t > 0) atomicMax(mx, t);
        if (nr > 0) atomicMax(mx + 1, nr);
    }
}

struct BataxRows {
    int32_t ncols;
    const int32_t *rowptr, *colind;
    const float *val;
    const int32_t *colptr, *crow;  // A's CSC: column pointers, rows
    const float *cval;             // and values
    float beta;
    const int32_t *toff;  // first temporary slot of each row of J
    int32_t *tkey;        // keys of each row, compact, at toff[j]
    float *tval;
    int32_t *cnt;         // keys of each row
    // one wave's LDS region: the sort keys at its start, then the terms, the
    // gathered rows' first positions, first CSR slots and beta * a_ij, each
    // sized for the largest row of this J (byte offsets, 16-byte aligned)
    int32_t lds_wave, off_term, off_pre, off_beg, off_a;
};

// Inclusive scan of one value per lane over the wave.
__device__ __forceinline__ int32_t wave_incl_scan(int32_t x, int lane) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int32_t y = __shfl_up(x, d, kWave);
        if (lane >= d) x += y;
    }
    return x;
}

// Sort keys (k, position) packed in one word: 32 bits while k < 2^23 (the
// position takes 9 bits), else 64.
constexpr int kPosBits = 9;
static_assert((1 << kPosBits) == kRowCap, "positions fill the low bits");

template <class Key>
struct RowKey;
template <>
struct RowKey<uint32_t> {
    static constexpr uint32_t pad = ~0u;
    __device__ static uint32_t make(int32_t k, int32_t s) {
        return ((uint32_t)k << kPosBits) | (uint32_t)s;
    }
    __device__ static uint32_t k(uint32_t x) { return x >> kPosBits; }
    __device__ static int32_t pos(uint32_t x) { return (int32_t)(x & (kRowCap - 1)); }
};
template <>
struct RowKey<unsigned long long> {
    static constexpr unsigned long long pad = ~0ull;
    __device__ static unsigned long long make(int32_t k, int32_t s) {
        return ((unsigned long long)(uint32_t)k << 32) | (uint32_t)s;
    }
    __device__ static uint32_t k(unsigned long long x) { return (uint32_t)(x >> 32); }
    __device__ static int32_t pos(unsigned long long x) { return (int32_t)(uint32_t)x; }
};

// Compare-exchange of two keys of the bitonic network, a at the lower index:
// afterwards a <= b when up, a >= b otherwise.
template <class Key>
__device__ __forceinline__ void row_ce(Key &a, Key &b, bool up) {
    const bool sw = (a > b) == up;
    const Key x = sw ? b : a, y = sw ? a : b;
    a = x;
    b = y;
}

// E consecutive keys at p (p aligned to E keys) in and out of LDS: whole
// 16-byte words where the run holds some (one instruction per 16 bytes
// instead of one per key).
template <class Key, int E>
__device__ __forceinline__ void load_run(const Key *p, Key (&v)[E]) {
    if constexpr (E * sizeof(Key) % 16 == 0) {
        constexpr int NV = E * (int)sizeof(Key) / 16;
        uint4 w[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i) w[i] = reinterpret_cast<const uint4 *>(p)[i];
        __builtin_memcpy(v, w, sizeof(w));
    } else {
#pragma unroll
        for (int m = 0; m < E; ++m) v[m] = p[m];
    }
}

template <class Key, int E>
__device__ __forceinline__ void store_run(Key *p, const Key (&v)[E]) {
    if constexpr (E * sizeof(Key) % 16 == 0) {
        constexpr int NV = E * (int)sizeof(Key) / 16;
        uint4 w[NV];
        __builtin_memcpy(w, v, sizeof(w));
#pragma unroll
        for (int i = 0; i < NV; ++i) reinterpret_cast<uint4 *>(p)[i] = w[i];
    } else {
#pragma unroll
        for (int m = 0; m < E; ++m) p[m] = v[m];
    }
}

// Substeps of bitonic stage `size` with strides 2^(lo + C - 1) down to 2^lo
// in one pass over LDS: each lane holds the 2^C keys that those substeps
// exchange among themselves (indices base + m 2^lo), so the C substeps
// cost one LDS round trip.  The direction is that of the stage for all of
// them (bit `size` of the index lies above the exchanged bits).
template <class Key, int C>
__device__ __forceinline__ void bitonic_group(Key *skey, int32_t np2, int32_t size, int lo,
                                              int l) {
    constexpr int E = 1 << C;
    for (int32_t t = l; t < (np2 >> C); t += kWave) {
        const int32_t base = ((t >> lo) << (lo + C)) | (t & ((1 << lo) - 1));
        Key v[E];
        if (lo == 0) {  // the same for the whole wave: a contiguous run
            load_run<Key, E>(skey + base, v);
        } else {
#pragma unroll
            for (int m = 0; m < E; ++m) v[m] = skey[base + (m << lo)];
        }
        const bool up = (base & size) == 0;
#pragma unroll
        for (int b = C - 1; b >= 0; --b)
#pragma unroll
            for (int m = 0; m < E; ++m)
                if (!(m & (1 << b))) row_ce(v[m], v[m | (1 << b)], up);
        if (lo == 0) {
            store_run<Key, E>(skey + base, v);
        } else {
#pragma unroll
            for (int m = 0; m < E; ++m) skey[base + (m << lo)] = v[m];
        }
    }
    __syncwarp();  // this wave only
}

// Stages 2, 4 and 8 of the bitonic network on every group of 8 consecutive
// keys in one pass (the directions of stages 2 and 4 change inside a group:
// bits 1 and 2 of the index).
template <class Key>
__device__ __forceinline__ void bitonic_first8(Key *skey, int32_t np2, int l) {
    for (int32_t t = l; t < (np2 >> 3); t += kWave) {
        const int32_t base = t << 3;
        Key v[8];
        load_run<Key, 8>(skey + base, v);
#pragma unroll
        for (int m = 0; m < 8; m += 2) row_ce(v[m], v[m + 1], (m & 2) == 0);
#pragma unroll
        for (int m = 0; m < 8; ++m)
            if (!(m & 2)) row_ce(v[m], v[m + 2], (m & 4) == 0);
#pragma unroll
        for (int m = 0; m < 8; m += 2) row_ce(v[m], v[m + 1], (m & 4) == 0);
        const bool up = (base & 8) == 0;
#pragma unroll
        for (int m = 0; m < 4; ++m) row_ce(v[m], v[m + 4], up);
#pragma unroll
        for (int m = 0; m < 8; ++m)
            if (!(m & 2)) row_ce(v[m], v[m + 2], up);
#pragma unroll
        for (int m = 0; m < 8; m += 2) row_ce(v[m], v[m + 1], up);
        store_run<Key, 8>(skey + base, v);
    }
    __syncwarp();  // this wave only
}

// Row j of J by one wave (at most kRowCap terms, checked by the caller); the
// LDS regions are sized by the caller from the largest row's term count and
// the longest column of A, so every index below stays inside its array.
template <class Key>
__global__ __launch_bounds__(kRowBlock) void batax_rows_kernel(BataxRows a) {
    using RK = RowKey<Key>;
    extern __shared__ __align__(16) unsigned char row_lds[];
    const int wid = threadIdx.x / kWave;
    const int l = threadIdx.x % kWave;
    const int32_t j = blockIdx.x * kRowWaves + wid;
    if (j >= a.ncols) return;  // the whole wave
    unsigned char *base = row_lds + (size_t)wid * a.lds_wave;
    Key *skey = reinterpret_cast<Key *>(base);                        // (k, position), sorted
    float *sterm = reinterpret_cast<float *>(base + a.off_term);      // terms by position
    int32_t *spre = reinterpret_cast<int32_t *>(base + a.off_pre);    // first position of each gathered row
    int32_t *sbeg = reinterpret_cast<int32_t *>(base + a.off_beg);    // its first CSR slot
    float *sa = reinterpret_cast<float *>(base + a.off_a);            // beta * a_ij
    const int32_t cb = a.colptr[j], nr = a.colptr[j + 1] - cb;  // nr <= terms <= kRowCap
    // 1. the rows of A storing column j, in CSC (ascending) order
    int32_t carry = 0;
    for (int32_t base = 0; base < nr; base += kWave) {
        const bool v = base + l < nr;
        int32_t len = 0, b = 0;
        float av = 0.f;
        if (v) {
            const int32_t c = cb + base + l;
            const int32_t i = a.crow[c];
            b = a.rowptr[i];
            len = a.rowptr[i + 1] - b;
            av = a.beta * a.cval[c];
        }
        const int32_t x = wave_incl_scan(len, l);
        if (v) {
            spre[base + l + 1] = carry + x;
            sbeg[base + l] = b;
            sa[base + l] = av;
        }
        carry += __shfl(x, kWave - 1, kWave);
    }
    const int32_t P = carry;
    if (P == 0) {  // uniform over the wave
        if (l == 0) a.cnt[j] = 0;
        return;
    }
    if (l == 0) spre[0] = 0;
    __syncwarp();  // this wave only
    // 2. the terms, row by row: position s of gathered row r is its entry
    //    sbeg[r] + s - spre[r]
    int32_t np2 = kWave;
    while (np2 < P) np2 <<= 1;
    for (int32_t s = l; s < np2; s += kWave) {
        if (s < P) {
            int32_t lo = 0, hi = nr - 1;  // last r with spre[r] <= s
            while (lo < hi) {
                const int32_t mid = (lo + hi + 1) >> 1;
                if (spre[mid] <= s) lo = mid;
                else hi = mid - 1;
            }
            const int32_t q = sbeg[lo] + (s - spre[lo]);
            skey[s] = RK::make(a.colind[q], s);
            sterm[s] = sa[lo] * a.val[q];
        } else {
            skey[s] = RK::pad;
        }
    }
    __syncwarp();  // this wave only
    // 3. bitonic sort of the (k, position) pairs in LDS, ascending: equal
    //    keys keep their positions' order (measured on MI355X with LDS
    //    regions sized for 512 terms, against a sort in registers with
    //    cross-lane shuffles, 634 us per call on the uniform 1M-entry
    //    workload, and ranks by binary searches in the other gathered rows,
    //    685 us: this took 407 us with 64-bit keys, 346 with 32-bit ones;
    //    with regions sized for the largest row, one substep per round trip
    //    200 us, up to three 187 us)
#ifdef NSD_BATAX_SORT_PLAIN
    for (int32_t size = 2; size <= np2; size <<= 1) {
        for (int32_t stride = size >> 1; stride > 0; stride >>= 1) {
            for (int32_t t = l; t < np2 / 2; t += kWave) {
                const int32_t i1 = 2 * t - (t & (stride - 1)), i2 = i1 + stride;
                const Key x1 = skey[i1], x2 = skey[i2];
                if ((x1 > x2) == ((i1 & size) == 0)) {
                    skey[i1] = x2;
                    skey[i2] = x1;
                }
            }
            __syncwarp();  // this wave only
        }
    }
#else
    // the same network, up to three substeps per LDS round trip: stages
    // 2-8 in one pass, then each stage's strides from the top, the first
    // pass taking log2(size) mod 3 of them and every later one three
    bitonic_first8<Key>(skey, np2, l);
    for (int32_t size = 16, n = 4; size <= np2; size <<= 1, ++n) {
        int hi = n - 1;  // log2 of the largest stride left
        const int first = n % 3;
        if (first == 1) bitonic_group<Key, 1>(skey, np2, size, hi, l);
        if (first == 2) bitonic_group<Key, 2>(skey, np2, size, hi - 1, l);
        hi -= first;
        for (; hi >= 2; hi -= 3) bitonic_group<Key, 3>(skey, np2, size, hi - 2, l);
    }
#endif
    // 4. runs of equal k: each lane takes a contiguous chunk of the sorted
    //    terms, numbers the runs that start there, and sums each of them in
    //    order in fp64 (a run may continue into the next lanes' chunks)
    const int32_t C = (P + kWave - 1) / kWave;
    const int32_t s0 = min(l * C, P), s1 = min(s0 + C, P);
    auto kof = [&](int32_t s) { return RK::k(skey[s]); };
    int32_t h = 0;
    for (int32_t s = s0; s < s1; ++s) h += (s == 0 || kof(s - 1) != kof(s)) ? 1 : 0;
    const int32_t incl = wave_incl_scan(h, l);
    int32_t r = incl - h;
    const int32_t o = a.toff[j];
    for (int32_t s = s0; s < s1; ++s) {
        const uint32_t k = kof(s);
        if (s == 0 || kof(s - 1) != k) {
            double sum = 0.0;
            for (int32_t t = s; t < P && kof(t) == k; ++t)
                sum += (double)sterm[RK::pos(skey[t])];
            a.tkey[o + r] = (int32_t)k;
            a.tval[o + r] = (float)sum;
            ++r;
        }
    }
    if (l == kWave - 1) a.cnt[j] = incl;
}

// Rows of J moved from their temporary slots to the CSR.
__global__ __launch_bounds__(kRowThreads) void batax_compact_kernel(
    const int32_t *toff, const int32_t *cnt, const int32_t *jrowptr, const int32_t *tkey,
    const float *tval, int32_t *jcolind, float *jval) {
    const int32_t j = blockIdx.x;
    const int32_t n = cnt[j], src = toff[j], dst = jrowptr[j];
    for (int32_t t = threadIdx.x; t < n; t += kRowThreads) {
        jcolind[dst + t] = tkey[src + t];
        jval[dst + t] = tval[src + t];
    }
}

struct BataxRowWs {
    int32_t *csort, *ridx, *crow, *colptr, *toff, *cnt, *tkey, *mx;
    float *cval, *tval;
    void *sort_ws, *scan_ws;
};

static void batax_row_carve(Carver &c, int32_t ncols, int32_t nnz, int64_t P, BataxRowWs *w) {
    const int64_t z = std::max<int32_t>(nnz, 1), n = std::max<int32_t>(ncols, 1);
    w->csort = c.take<int32_t>(z);
    w->ridx = c.take<int32_t>(z);
    w->cval = c.take<float>(z);
    w->crow = c.take<int32_t>(z);
    w->colptr = c.take<int32_t>(n + 1);
    w->toff = c.take<int32_t>(n);
    w->cnt = c.take<int32_t>(n);
    w->mx = c.take<int32_t>(64);
    w->tkey = c.take<int32_t>(std::max<int64_t>(P, 1));
    w->tval = c.take<float>(std::max<int64_t>(P, 1));
    const size_t sb = sort_ws_bytes(z, (int32_t)n, 2), cb = scan_ws_bytes(std::max(z, n));
    char *s = c.take<char>((int64_t)std::max(sb, cb));
    w->sort_ws = w->scan_ws = s;
}

// J by rows when every row has at most `cap` terms; *done says whether it did.
static nsd_status batax_by_rows(const nsd_csr *A, float beta, int64_t P, int cap,
                                const BataxRowWs &w, int32_t *jrowptr, int32_t *jcolind,
                                float *jval, int32_t *nnz_out, bool *done, hipStream_t st) {
    *done = false;
    const int32_t m = A->nrows, n = A->ncols, z = A->nnz;
    // A's CSC: columns sorted stably (rows ascend within a column), each
    // entry's row and value travelling with its column
    const int32_t *ridx = A->rowidx;
    if (ridx == nullptr) {
        slot_rows_kernel<<<bgrid(z), kBataxThreads, 0, st>>>(z, m, A->rowptr, w.ridx);
        NSD_TRY(check_launch("slot_rows_kernel"));
        ridx = w.ridx;
    }
    const int32_t *in[2] = {ridx, reinterpret_cast<const int32_t *>(A->val)};
    int32_t *out[2] = {w.crow, reinterpret_cast<int32_t *>(w.cval)};
    NSD_TRY(radix_sort_multi(z, n, A->colind, 2, in, w.csort, out, w.sort_ws, st));
    NSD_TRY(segptr_from_sorted(z, n, w.csort, w.colptr, st));
    // every row of J's first term: the prefix sums of the gathered row
    // lengths over the CSC slots (their total is the number of products)
    int32_t *len = w.ridx;  // free once the sort has read it
    slot_len_kernel<<<bgrid(z), kBataxThreads, 0, st>>>(z, w.crow, A->rowptr, len);
    NSD_TRY(check_launch("slot_len_kernel"));
    // w.mx: [0] the most terms of a row of J, [1] the longest column of A,
    // [2] the scan's (32-bit) total, [4..5] the products counted in 64 bits
    auto *pairs = reinterpret_cast<unsigned long long *>(w.mx + 4);
    NSD_HIP(hipMemsetAsync(w.mx, 0, 8 * sizeof(int32_t), st));
    pairs_total_kernel<<<bgrid(m), kBataxThreads, 0, st>>>(m, A->rowptr, pairs);
    NSD_TRY(check_launch("pairs_total_kernel"));
    NSD_TRY(scan_exclusive(len, len, z, w.mx + 2, w.scan_ws, st));
    row_terms_kernel<<<bgrid(n), kBataxThreads, 0, st>>>(n, z, w.colptr, len, w.mx + 2, w.toff,
                                                         w.mx);
    NSD_TRY(check_launch("row_terms_kernel"));
    int32_t mx[6] = {0, 0, 0, 0, 0, 0};
    NSD_HIP(hipMemcpyAsync(mx, w.mx, sizeof(mx), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    unsigned long long np = 0;
    std::memcpy(&np, mx + 4, sizeof(np));
    if (np != (unsigned long long)P)
        return fail(NSD_ERR_INVALID_ARG, "npairs = %lld, but A's rows give %llu pairs",
                    (long long)P, np);
    if (mx[0] > cap) return NSD_OK;  // some row of J is too long: the sort path
    BataxRows a;
    a.ncols = n;
    a.rowptr = A->rowptr;
    a.colind = A->colind;
    a.val = A->val;
    a.colptr = w.colptr;
    a.cval = w.cval;
    a.crow = w.crow;
    a.beta = beta;
    a.toff = w.toff;
    a.tkey = w.tkey;
    a.tval = w.tval;
    a.cnt = w.cnt;
    // every gathered row stores column j, so a column's rows are at most its
    // row's terms: mx[1] <= mx[0] <= kRowCap
    const bool narrow = n < (1 << (32 - kPosBits));  // every real key below the padding
    int32_t np2 = kWave;
    while (np2 < mx[0]) np2 <<= 1;
    auto r16 = [](int64_t b) { return (int32_t)((b + 15) / 16 * 16); };
    const int32_t nrm = std::max(mx[1], 1);
    a.off_term = r16((int64_t)np2 * (narrow ? 4 : 8));
    a.off_pre = a.off_term + r16(4LL * std::max(mx[0], 1));
    a.off_beg = a.off_pre + r16(4LL * (nrm + 1));
    a.off_a = a.off_beg + r16(4LL * nrm);
    a.lds_wave = a.off_a + r16(4LL * nrm);
    const size_t lds = (size_t)kRowWaves * a.lds_wave;  // at most 12.3 KB per wave
    const unsigned blocks = (unsigned)ceil_div(n, kRowWaves);
    probe_begin(NSD_KERNEL_BATAX_ROWS, st);
    if (narrow)
        batax_rows_kernel<uint32_t><<<blocks, kRowBlock, lds, st>>>(a);
    else
        batax_rows_kernel<unsigned long long><<<blocks, kRowBlock, lds, st>>>(a);
    probe_end(NSD_KERNEL_BATAX_ROWS, st);
    NSD_TRY(check_launch("batax_rows_kernel"));
    NSD_TRY(scan_exclusive(w.cnt, jrowptr, n, jrowptr + n, w.scan_ws, st));
    batax_compact_kernel<<<(unsigned)n, kRowThreads, 0, st>>>(w.toff, w.cnt, jrowptr, w.tkey,
                                                              w.tval, jcolind, jval);
    NSD_TRY(check_launch("batax_compact_kernel"));
    int32_t nk = 0;
    NSD_HIP(hipMemcpyAsync(&nk, jrowptr + n, sizeof(nk), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    (void)P;
    *nnz_out = nk;
    *done = true;
    return NSD_OK;
}

// Workspace layout shared by the size query and the call.
struct BataxWs {
    int32_t *sq, *off, *tot;
    int32_t *key_j, *key_k, *kperm, *jg, *js, *perm2, *ks, *head, *pos, *run, *runptr, *run_j;
    float *term;
    void *sort_ws, *scan_ws;
    size_t sort_bytes, scan_bytes;
};

static nsd_status batax_carve(void *ws, int32_t nrows, int32_t n, int64_t P, BataxWs *w,
                              size_t *total, int32_t nnz = 0, BataxRowWs *rw = nullptr) {
    Carver c(ws);
    // the row path's buffers first (it runs first; the sort path reuses
    // nothing of it)
    BataxRowWs rw_tmp;
    batax_row_carve(c, n, nnz, P, rw ? rw : &rw_tmp);
    w->sq = c.take<int32_t>(std::max<int64_t>(nrows, 1));
    w->off = c.take<int32_t>(std::max<int64_t>(nrows, 1));
    w->tot = c.take<int32_t>(64);
    const int64_t Q = std::max<int64_t>(P, 1);
    w->key_j = c.take<int32_t>(Q);
    w->key_k = c.take<int32_t>(Q);
    w->term = c.take<float>(Q);
    w->kperm = c.take<int32_t>(Q);
    w->jg = c.take<int32_t>(Q);
    w->js = c.take<int32_t>(Q);
    w->perm2 = c.take<int32_t>(Q);
    w->ks = c.take<int32_t>(Q);
    w->head = c.take<int32_t>(Q);
    w->pos = c.take<int32_t>(Q);
    w->run = c.take<int32_t>(Q);
    w->runptr = c.take<int32_t>(Q + 1);
    w->run_j = c.take<int32_t>(Q);
    w->sort_bytes = sort_ws_bytes(Q, std::max(n, 1));
    w->scan_bytes = scan_ws_bytes(std::max<int64_t>(Q, nrows));
    // the sort and scan scratch are used one after another
    char *s = c.take<char>((int64_t)std::max(w->sort_bytes, w->scan_bytes));
    w->sort_ws = w->scan_ws = s;
    *total = c.bytes();
    return NSD_OK;
}

static nsd_status check_batax_csr(const nsd_csr *A) {
    NSD_REQUIRE(A != nullptr, "CSR descriptor is NULL");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative CSR size");
    NSD_REQUIRE(A->rowptr != nullptr, "CSR rowptr is NULL");
    if (A->nnz > 0) {
        NSD_REQUIRE(A->nrows > 0 && A->ncols > 0, "nnz > 0 in an empty shape");
        NSD_REQUIRE(A->colind && A->val, "CSR colind/val is NULL");
    }
    return NSD_OK;
}

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_batax_pairs(const nsd_csr *A, int64_t *npairs, void *ws, size_t ws_bytes,
                           void *stream) {
    NSD_TRY(check_batax_csr(A));
    NSD_REQUIRE(npairs != nullptr, "npairs is NULL");
    NSD_REQUIRE(ws != nullptr && ws_bytes >= 256, "workspace of at least 256 bytes needed");
    hipStream_t st = as_stream(stream);
    auto *total = static_cast<unsigned long long *>(ws);
    NSD_HIP(hipMemsetAsync(total, 0, sizeof(unsigned long long), st));
    if (A->nrows > 0) {
        pairs_total_kernel<<<bgrid(A->nrows), kBataxThreads, 0, st>>>(A->nrows, A->rowptr, total);
        NSD_TRY(check_launch("pairs_total_kernel"));
    }
    unsigned long long h = 0;
    NSD_HIP(hipMemcpyAsync(&h, total, sizeof(h), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    *npairs = (int64_t)h;
    return NSD_OK;
}

nsd_status nsd_batax_workspace_size(const nsd_csr *A, int64_t npairs, size_t *bytes) {
    NSD_TRY(check_batax_csr(A));
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(npairs >= 0, "negative pair count");
    if (npairs >= kBataxMaxPairs)
        return fail(NSD_ERR_TOO_LARGE, "%lld row pairs (at most 2^30)", (long long)npairs);
    BataxWs w;
    return batax_carve(nullptr, A->nrows, A->ncols, npairs, &w, bytes, A->nnz);
}

nsd_status nsd_batax_jacobian(const nsd_csr *A, float beta, int64_t npairs, int32_t *jrowptr,
                              int32_t *jcolind, float *jval, int32_t *nnz_out, void *ws,
                              size_t ws_bytes, void *stream) {
    NSD_TRY(check_batax_csr(A));
    NSD_REQUIRE(jrowptr != nullptr && nnz_out != nullptr, "jrowptr/nnz_out is NULL");
    NSD_REQUIRE(npairs >= 0, "negative pair count");
    if (npairs >= kBataxMaxPairs)
        return fail(NSD_ERR_TOO_LARGE, "%lld row pairs (at most 2^30)", (long long)npairs);
    NSD_REQUIRE(npairs == 0 || (jcolind && jval), "jcolind/jval is NULL");
    size_t need = 0;
    BataxWs w;
    BataxRowWs rw;
    NSD_TRY(batax_carve(nullptr, A->nrows, A->ncols, npairs, &w, &need, A->nnz, &rw));
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    NSD_TRY(batax_carve(ws, A->nrows, A->ncols, npairs, &w, &need, A->nnz, &rw));
    hipStream_t st = as_stream(stream);
    const int32_t m = A->nrows, n = A->ncols;
    const int64_t P = npairs;
    if (P == 0) {
        NSD_TRY(segptr_from_sorted(0, n, nullptr, jrowptr, st));
        NSD_HIP(hipStreamSynchronize(st));
        *nnz_out = 0;
        return NSD_OK;
    }
    // 1. term offsets per row and the terms
    // the row path checks npairs against A before it writes anything but
    // workspace; the sort path checks it here when the row path is off
    const int cap = row_cap();
    if (cap > 0) {
        bool done = false;
        NSD_TRY(batax_by_rows(A, beta, P, cap, rw, jrowptr, jcolind, jval, nnz_out, &done, st));
        if (done) return NSD_OK;
    }
    if (cap == 0) {  // the products counted in 64 bits
        auto *pairs = reinterpret_cast<unsigned long long *>(w.tot + 4);
        NSD_HIP(hipMemsetAsync(pairs, 0, sizeof(*pairs), st));
        pairs_total_kernel<<<bgrid(m), kBataxThreads, 0, st>>>(m, A->rowptr, pairs);
        NSD_TRY(check_launch("pairs_total_kernel"));
        unsigned long long np = 0;
        NSD_HIP(hipMemcpyAsync(&np, pairs, sizeof(np), hipMemcpyDeviceToHost, st));
        NSD_HIP(hipStreamSynchronize(st));
        if (np != (unsigned long long)P)
            return fail(NSD_ERR_INVALID_ARG, "npairs = %lld, but A's rows give %llu pairs",
                        (long long)P, np);
    }
    // npairs is A's, below 2^30: every row's square and their sums fit int32
    row_pairs_kernel<<<bgrid(m), kBataxThreads, 0, st>>>(m, A->rowptr, w.sq);
    NSD_TRY(check_launch("row_pairs_kernel"));
    NSD_TRY(scan_exclusive(w.sq, w.off, m, w.tot, w.scan_ws, st));
    expand_pairs_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, m, w.off, A->rowptr, A->colind,
                                                            A->val, beta, w.key_j, w.key_k,
                                                            w.term);
    NSD_TRY(check_launch("expand_pairs_kernel"));
    // 2. stable sort by k, then stably by j: (j, k) order, runs in row order
    NSD_TRY(radix_sort_pairs(P, n, w.key_k, nullptr, w.ks, w.kperm, w.sort_ws, st));
    gather_keys_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.kperm, w.key_j, w.jg);
    NSD_TRY(check_launch("gather_keys_kernel"));
    NSD_TRY(radix_sort_pairs(P, n, w.jg, w.kperm, w.js, w.perm2, w.sort_ws, st));
    gather_keys_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.perm2, w.key_k, w.ks);
    NSD_TRY(check_launch("gather_keys_kernel"));
    // 3. runs -> keys of J
    pair_heads_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.js, w.ks, w.head);
    NSD_TRY(check_launch("pair_heads_kernel"));
    NSD_TRY(scan_exclusive(w.head, w.pos, P, w.tot + 1, w.scan_ws, st));
    runs_kernel<<<bgrid(P), kBataxThreads, 0, st>>>(P, w.head, w.pos, w.js, w.ks, w.run, w.run_j,
                                                    jcolind);
    NSD_TRY(check_launch("runs_kernel"));
    int32_t nk = 0;
    NSD_HIP(hipMemcpyAsync(&nk, w.tot + 1, sizeof(nk), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    NSD_TRY(segptr_from_sorted(P, nk, w.run, w.runptr, st));
    NSD_TRY(segptr_from_sorted(nk, n, w.run_j, jrowptr, st));
    // 4. run sums (terms reached through perm2)
    run_sums_kernel<<<bgrid(nk), kBataxThreads, 0, st>>>(nk, w.runptr, w.perm2, w.term, jval);
    NSD_TRY(check_launch("run_sums_kernel"));
    NSD_HIP(hipStreamSynchronize(st));
    *nnz_out = nk;
    return NSD_OK;
}

}  // extern "C"
