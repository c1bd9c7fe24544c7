// Format builders: COO -> CSR, CSR -> CSC, mode index of a COO tensor, row
// expansion, value permutation and CSR validation.
//
// Every ordering is a stable sort by key, done as least-significant-digit
// radix sort: a sequence of stable counting sorts on 8-bit digits (histogram
// per tile, one device-wide exclusive scan over [digit][tile], stable scatter
// with wave-level match masks).  Ties keep their input order, so the results
// are bit-exact and equal to a sequential stable sort.
#include <algorithm>

#include "nsd_internal.hpp"

namespace nsd {

// ------------------------------------------------------------------ scan

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

struct OpSum {
    static constexpr int kIdentity = 0;
    __device__ static int apply(int a, int b) { return a + b; }
};
struct OpMax {
    static constexpr int kIdentity = INT32_MIN;
    __device__ static int apply(int a, int b) { return a > b ? a : b; }
};

// Exclusive scan of one value per thread across the block; returns the
// block total through *total.
template <class Op>
__device__ int block_exclusive_scan(int v, int *total) {
    __shared__ int wave_tot[kScanThreads / kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    int inc = v;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        int t = __shfl_up(inc, d, kWave);
        if (lane >= d) inc = Op::apply(t, inc);
    }
    int exc = __shfl_up(inc, 1, kWave);
    if (lane == 0) exc = Op::kIdentity;
    if (lane == kWave - 1) wave_tot[wave] = inc;
    __syncthreads();
    int base = Op::kIdentity, all = Op::kIdentity;
#pragma unroll
    for (int w = 0; w < kScanThreads / kWave; ++w) {
        if (w < wave) base = Op::apply(base, wave_tot[w]);
        all = Op::apply(all, wave_tot[w]);
    }
    __syncthreads();
    *total = all;
    return Op::apply(base, exc);
}

template <class Op>
__global__ __launch_bounds__(kScanThreads) void scan_reduce_kernel(const int32_t *in, int64_t n,
                                                                   int32_t *sums) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int s = Op::kIdentity;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i)
        if (base + i < n) s = Op::apply(s, in[base + i]);
    int total;
    block_exclusive_scan<Op>(s, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

template <class Op>
__global__ __launch_bounds__(kScanThreads) void scan_tile_kernel(const int32_t *in, int32_t *out,
                                                                 int64_t n, const int32_t *offs,
                                                                 int32_t *total_dev) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int v[kScanItems];
    int s = Op::kIdentity;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        v[i] = base + i < n ? in[base + i] : Op::kIdentity;
        s = Op::apply(s, v[i]);
    }
    int total;
    const int pre = offs ? offs[blockIdx.x] : Op::kIdentity;
    int run = Op::apply(pre, block_exclusive_scan<Op>(s, &total));
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        if (base + i < n) out[base + i] = run;
        run = Op::apply(run, v[i]);
    }
    if (total_dev && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0)
        *total_dev = Op::apply(pre, total);
}

// A tile scan whose block first forms its own prefix from the tile sums of
// the blocks before it (at most kScanTile of them): one level and one launch
// fewer than scanning the sums separately.
template <class Op>
__global__ __launch_bounds__(kScanThreads) void scan_tile_prefix_kernel(const int32_t *in,
                                                                        int32_t *out, int64_t n,
                                                                        const int32_t *sums,
                                                                        int32_t *total_dev) {
    int s = Op::kIdentity;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        const int j = threadIdx.x * kScanItems + i;  // tiles before this block, in order
        if (j < (int)blockIdx.x) s = Op::apply(s, sums[j]);
    }
    int pre;
    block_exclusive_scan<Op>(s, &pre);  // pre = the sum over all of them
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int v[kScanItems];
    int t = Op::kIdentity;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        v[i] = base + i < n ? in[base + i] : Op::kIdentity;
        t = Op::apply(t, v[i]);
    }
    int total;
    int run = Op::apply(pre, block_exclusive_scan<Op>(t, &total));
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        if (base + i < n) out[base + i] = run;
        run = Op::apply(run, v[i]);
    }
    if (total_dev && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0)
        *total_dev = Op::apply(pre, total);
}

size_t scan_ws_bytes(int64_t n) {
    Carver c(nullptr);
    int64_t m = ceil_div(n, kScanTile);
    while (m > 1) {
        c.take<int32_t>(m);
        m = ceil_div(m, kScanTile);
    }
    return c.bytes();
}

template <class Op>
static nsd_status scan_level(const int32_t *in, int32_t *out, int64_t n, int32_t *total_dev,
                             Carver &c, hipStream_t st) {
    const int64_t tiles = ceil_div(n, kScanTile);
    if (tiles <= 1) {
        scan_tile_kernel<Op><<<1, kScanThreads, 0, st>>>(in, out, n, nullptr, total_dev);
        return check_launch("scan_tile_kernel");
    }
    int32_t *sums = c.take<int32_t>(tiles);
    scan_reduce_kernel<Op><<<tiles, kScanThreads, 0, st>>>(in, n, sums);
    NSD_TRY(check_launch("scan_reduce_kernel"));
    if (tiles <= kScanTile) {
        scan_tile_prefix_kernel<Op><<<tiles, kScanThreads, 0, st>>>(in, out, n, sums, total_dev);
        return check_launch("scan_tile_prefix_kernel");
    }
    NSD_TRY(scan_level<Op>(sums, sums, tiles, nullptr, c, st));
    scan_tile_kernel<Op><<<tiles, kScanThreads, 0, st>>>(in, out, n, sums, total_dev);
    return check_launch("scan_tile_kernel");
}

// n == 0 is not allowed here (the callers handle empty inputs themselves).
nsd_status scan_exclusive(const int32_t *in, int32_t *out, int64_t n, int32_t *total_dev,
                          void *ws, hipStream_t st) {
    Carver c(ws);
    return scan_level<OpSum>(in, out, n, total_dev, c, st);
}

nsd_status scan_exclusive_max(const int32_t *in, int32_t *out, int64_t n, void *ws,
                              hipStream_t st) {
    Carver c(ws);
    return scan_level<OpMax>(in, out, n, nullptr, c, st);
}

// ------------------------------------------------------------ radix sort

constexpr int kSortThreads = 256;
constexpr int kSortRounds = 16;  // 64-element rounds per wave
constexpr int kSortTile = kSortThreads * kSortRounds;
constexpr int kBins = 256;
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kMaxPayloads = 3;

// A sort's reads of its keys and payloads: non-temporal when the arrays are
// far larger than the L2s (they are streamed once per pass; the scatter's
// output runs are what should stay), ordinary otherwise (measured on
// MI355X: the 50M-entry builders 5.53 -> 5.43 ms; a 1M-entry sort a little
// slower so).
constexpr int64_t kSortStreamMin = int64_t(1) << 23;

template <bool NT>
__device__ __forceinline__ int32_t sort_load(const int32_t *p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}

// The digit of a key at bit `shift`.  A composite key (lo_bits > 0) is the
// pair (hi, lo) read as hi * 2^lo_bits + lo, with lo < 2^lo_bits: sorting by
// it orders by hi, then by lo, in one sort.
__device__ __forceinline__ int key_digit(int32_t lo, int32_t hi, int lo_bits, int shift) {
    const uint32_t l = (uint32_t)lo, h = (uint32_t)hi;
    // lo_bits and shift are the same for every thread: scalar branches
    if (lo_bits == 0 || shift + 8 <= lo_bits) return (int)((l >> shift) & (kBins - 1));
    if (shift >= lo_bits) return (int)((h >> (shift - lo_bits)) & (kBins - 1));
    return (int)(((l >> shift) | (h << (lo_bits - shift))) & (kBins - 1));  // straddles both
}

// Digit counts of one tile.  Keys drawn from a skewed distribution share
// their high digits, and same-address LDS atomics of one instruction are
// serialised, so each round first peels off up to kHistPeel digit groups:
// the digit of the lowest lane not yet counted, its lanes found by one
// ballot, added by one atomic.  The keys left (a spread of digits) take an
// atomic each.  Measured on MI355X over the nine passes of the 50M-entry
// builders: 97.8 us per pass with an atomic per key as each key arrives,
// 85.1 with the tile's keys loaded first, 61.3 / 62.5 / 88.0 peeling 1 / 2 /
// 4 groups, 131 with the full 8-ballot digit match of the scatter.
// Build-time knob NSD_HIST_PEEL.
#ifdef NSD_HIST_PEEL
constexpr int kHistPeel = NSD_HIST_PEEL;
#else
constexpr int kHistPeel = 1;
#endif

// With `bad` set (the first pass of a sort whose keys come from a caller),
// a key outside [0, max_lo) (or a high word outside [0, max_hi)) sets *bad:
// the range check of a builder rides on the read the sort makes anyway.
// Digits are masked, so such keys stay within the sort's own arrays.
template <bool PAIR, bool NT>
__global__ __launch_bounds__(kSortThreads) void radix_hist_kernel(const int32_t *keys,
                                                                  const int32_t *khi,
                                                                  int lo_bits, int64_t n,
                                                                  int shift, int64_t ntiles,
                                                                  int32_t *hist, int32_t *bad,
                                                                  int32_t max_lo,
                                                                  int32_t max_hi) {
    __shared__ int cnt[kBins];
    cnt[threadIdx.x] = 0;
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    int key[kSortRounds], hi[kSortRounds];
#pragma unroll
    for (int i = 0; i < kSortRounds; ++i) {
        const int64_t q = base + (int64_t)i * kSortThreads + threadIdx.x;
        key[i] = q < n ? sort_load<NT>(keys + q) : 0;
        if constexpr (PAIR) hi[i] = q < n ? sort_load<NT>(khi + q) : 0;  // a composite key's high words
    }
    if (bad) {
        bool out = false;
#pragma unroll
        for (int i = 0; i < kSortRounds; ++i) {
            out = out || key[i] < 0 || key[i] >= max_lo;
            if constexpr (PAIR) out = out || hi[i] < 0 || hi[i] >= max_hi;
        }
        if (__ballot(out) && lane == 0) atomicOr(bad, 1);
    }
#pragma unroll
    for (int i = 0; i < kSortRounds; ++i) {
        const int64_t q = base + (int64_t)i * kSortThreads + threadIdx.x;
        const bool valid = q < n;
        const int d = PAIR ? key_digit(key[i], hi[i], lo_bits, shift)
                           : (int)(((uint32_t)key[i] >> shift) & (kBins - 1));
        uint64_t rest = __ballot(valid);  // lanes not yet counted (wave-uniform)
#pragma unroll
        for (int it = 0; it < kHistPeel; ++it) {
            if (rest == 0) break;
            const int lead = __ffsll((unsigned long long)rest) - 1;
            const int d0 = __builtin_amdgcn_readlane(d, lead);
            const uint64_t m = __ballot(d == d0) & rest;
            if (lane == lead) atomicAdd(&cnt[d0], __popcll(m));
            rest &= ~m;
        }
        if ((rest >> lane) & 1) atomicAdd(&cnt[d], 1);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = cnt[threadIdx.x];
}

// Workgroups go to the eight XCDs round-robin (block b on XCD b mod 8), each
// XCD with its own L2.  This renumbers the blocks so that every XCD takes one
// contiguous range of the tiles: neighbouring tiles write adjacent runs of
// one output region, and with the renumbering those runs meet in one L2 and
// leave it as whole lines instead of partial ones from eight L2s.
__device__ __forceinline__ int64_t xcd_contiguous_tile() {
    const int nb = (int)gridDim.x, b = (int)blockIdx.x, x = b % 8;
    int start = 0;
    for (int y = 0; y < x; ++y) start += (nb - y + 7) / 8;  // blocks on XCDs before x
    return start + b / 8;
}

// Stable scatter of one tile.  Wave w owns the tile's elements
// [w * 1024, (w + 1) * 1024) and walks them in 16 rounds of 64 consecutive
// elements, so (wave, round, lane) order is input order.  Inside a round the
// lanes holding the same digit are found with 8 ballots; a lane's rank is the
// count of such lanes below it plus what earlier rounds of its wave placed.
// The tile is then staged in LDS in digit order (digit runs in input order)
// and written back run by run, so consecutive lanes store consecutive
// addresses of a digit's output range instead of scattering single words.
// Payloads carried with the keys: in[j] NULL is the element's own index.
// Carrying what a caller would otherwise gather through the sort's
// permutation (one random 4-byte read per element) costs 8 more bytes per
// element and pass, read and written in runs.  With a composite key
// (lo_bits > 0) payload 0 is the key's high word.
struct SortPayloads {
    const int32_t *in[kMaxPayloads];
    int32_t *out[kMaxPayloads];
};

template <int NP, bool NT>
__global__ __launch_bounds__(kSortThreads) void radix_scatter_kernel(
    const int32_t *kin, SortPayloads pl, int32_t *kout, int64_t n, int lo_bits, int shift,
    int64_t ntiles, const int32_t *offs) {
    __shared__ int wcnt[kSortWaves][kBins];
    __shared__ int tile_off[kBins];
    __shared__ int tile_start[kBins];
    __shared__ int skey[kSortTile];
    __shared__ int sval[kSortTile];  // one payload at a time
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t tile = xcd_contiguous_tile();
    for (int w = 0; w < kSortWaves; ++w) wcnt[w][threadIdx.x] = 0;
    tile_off[threadIdx.x] = offs[(int64_t)threadIdx.x * ntiles + tile];
    __syncthreads();

    const int64_t tile0 = tile * kSortTile;
    const int64_t base = tile0 + (int64_t)wave * (kSortRounds * kWave);
    int key[kSortRounds], val[NP][kSortRounds], rank[kSortRounds], dig[kSortRounds];
#pragma unroll
    for (int i = 0; i < kSortRounds; ++i) {
        const int64_t q = base + (int64_t)i * kWave + lane;
        const bool valid = q < n;
        key[i] = valid ? sort_load<NT>(kin + q) : 0;
#pragma unroll
        for (int j = 0; j < NP; ++j)
            val[j][i] = valid ? (pl.in[j] ? sort_load<NT>(pl.in[j] + q) : (int32_t)q) : 0;
        const int d = key_digit(key[i], val[0][i], lo_bits, shift);
        dig[i] = d;
        uint64_t same = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (d >> b) & 1;
            const uint64_t m = __ballot(bit);
            same &= bit ? m : ~m;
        }
        const int below = __popcll(same & __lanemask_lt());
        const int prev = valid ? wcnt[wave][d] : 0;
        rank[i] = prev + below;
        if (valid && below == 0) wcnt[wave][d] = prev + __popcll(same);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    // per digit: waves' offsets inside the digit's run, then the run starts
    // (exclusive scan of the digit totals over the tile)
    int total = 0;
    {
        const int d = threadIdx.x;
        for (int w = 0; w < kSortWaves; ++w) {
            const int c = wcnt[w][d];
            wcnt[w][d] = total;
            total += c;
        }
        tile_start[d] = total;
    }
    __syncthreads();
    for (int off = 1; off < kBins; off <<= 1) {
        const int add = (int)threadIdx.x >= off ? tile_start[threadIdx.x - off] : 0;
        __syncthreads();
        tile_start[threadIdx.x] += add;
        __syncthreads();
    }
    tile_start[threadIdx.x] -= total;  // inclusive -> exclusive
    __syncthreads();
    const int tile_n = (int)min<int64_t>(kSortTile, n - tile0);
    // the keys with the first payload, then each further payload through the
    // same buffer (the staged keys give every position its output slot): one
    // buffer keeps four blocks per CU where a buffer per payload allowed two
    // (measured on MI355X: 0.52 against 0.62 ms per pass of 50M with three
    // payloads, 0.37 against 0.53 with two).  The staged positions' digits,
    // found with the first payload (a composite key's high word), serve the
    // later payloads.
    int lpos[kSortRounds];  // each element's staging slot (its digit run, its rank)
#pragma unroll
    for (int i = 0; i < kSortRounds; ++i) {
        const int64_t q = base + (int64_t)i * kWave + lane;
        lpos[i] = q < n ? tile_start[dig[i]] + wcnt[wave][dig[i]] + rank[i] : -1;
    }
    int odig[kSortRounds];
#pragma unroll
    for (int j = 0; j < NP; ++j) {
        if (j > 0) __syncthreads();  // the previous payload is written out
#pragma unroll
        for (int i = 0; i < kSortRounds; ++i) {
            if (lpos[i] >= 0) {
                if (j == 0) skey[lpos[i]] = key[i];
                sval[lpos[i]] = val[j][i];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kSortRounds; ++r) {
            const int lp = threadIdx.x + r * kSortThreads;
            if (lp < tile_n) {
                if (j == 0) odig[r] = key_digit(skey[lp], sval[lp], lo_bits, shift);
                const int d = odig[r];
                const int64_t pos = (int64_t)tile_off[d] + (lp - tile_start[d]);
                if (j == 0) kout[pos] = skey[lp];
                pl.out[j][pos] = sval[lp];
            }
        }
    }
}

// Bits of the largest key below max_key (0 for max_key <= 1).
static int key_bits(int32_t max_key) {
    uint32_t top = max_key > 0 ? (uint32_t)(max_key - 1) : 0u;
    int bits = 0;
    while (top) {
        ++bits;
        top >>= 1;
    }
    return bits;
}

static int digit_passes(int bits) { return bits == 0 ? 1 : (bits + 7) / 8; }

size_t sort_ws_bytes(int64_t n, int32_t max_key, int np) {
    Carver c(nullptr);
    const int64_t ntiles = ceil_div(n, kSortTile);
    c.take<int32_t>(n);  // ping keys
    c.take<int32_t>(n);  // pong keys
    for (int j = 0; j < np; ++j) {
        c.take<int32_t>(n);  // ping payload j
        c.take<int32_t>(n);  // pong payload j
    }
    c.take<int32_t>(ntiles * kBins);
    const size_t scan = scan_ws_bytes(ntiles * kBins);
    (void)max_key;
    return c.bytes() + scan;
}

template <int NP>
static nsd_status launch_scatter(int64_t ntiles, const int32_t *ksrc, const SortPayloads &pl,
                                 int32_t *kdst, int64_t n, int lo_bits, int shift,
                                 const int32_t *hist, hipStream_t st) {
    if (n >= kSortStreamMin)
        radix_scatter_kernel<NP, true><<<ntiles, kSortThreads, 0, st>>>(ksrc, pl, kdst, n, lo_bits,
                                                                        shift, ntiles, hist);
    else
        radix_scatter_kernel<NP, false><<<ntiles, kSortThreads, 0, st>>>(ksrc, pl, kdst, n,
                                                                         lo_bits, shift, ntiles,
                                                                         hist);
    return check_launch("radix_scatter_kernel");
}

template <bool PAIR>
static void launch_hist(int64_t ntiles, const int32_t *keys, const int32_t *khi, int lo_bits,
                        int64_t n, int shift, int32_t *hist, int32_t *bad, int32_t max_lo,
                        int32_t max_hi, hipStream_t st) {
    if (n >= kSortStreamMin)
        radix_hist_kernel<PAIR, true><<<ntiles, kSortThreads, 0, st>>>(
            keys, khi, lo_bits, n, shift, ntiles, hist, bad, max_lo, max_hi);
    else
        radix_hist_kernel<PAIR, false><<<ntiles, kSortThreads, 0, st>>>(
            keys, khi, lo_bits, n, shift, ntiles, hist, bad, max_lo, max_hi);
}

// The passes of one sort: keys of `bits` bits, composite when lo_bits > 0
// (then payload 0 is the key's high word).
static nsd_status radix_sort_passes(int64_t n, int bits, int lo_bits, const int32_t *key_in,
                                    int np, const int32_t *const *payload_in, int32_t *key_out,
                                    int32_t *const *payload_out, void *ws, hipStream_t st,
                                    int32_t *bad = nullptr, int32_t max_lo = 0,
                                    int32_t max_hi = 0) {
    if (n <= 0) return NSD_OK;
    if (np < 1 || np > kMaxPayloads) return fail(NSD_ERR_INVALID_ARG, "%d sort payloads", np);
    Carver c(ws);
    const int64_t ntiles = ceil_div(n, kSortTile);
    int32_t *kbuf[2] = {c.take<int32_t>(n), c.take<int32_t>(n)};
    int32_t *vbuf[kMaxPayloads][2];
    for (int j = 0; j < np; ++j) {
        vbuf[j][0] = c.take<int32_t>(n);
        vbuf[j][1] = c.take<int32_t>(n);
    }
    int32_t *hist = c.take<int32_t>(ntiles * kBins);
    void *scan_ws = c.base + c.bytes();
    const int passes = digit_passes(bits);
    const int32_t *ksrc = key_in;
    SortPayloads pl{};
    for (int j = 0; j < np; ++j) pl.in[j] = payload_in[j];
    for (int p = 0; p < passes; ++p) {
        const bool last = p == passes - 1;
        int32_t *kdst = last ? key_out : kbuf[p & 1];
        for (int j = 0; j < np; ++j) pl.out[j] = last ? payload_out[j] : vbuf[j][p & 1];
        int32_t *chk = p == 0 ? bad : nullptr;  // the caller's keys: the first pass reads them
        if (lo_bits > 0)
            launch_hist<true>(ntiles, ksrc, pl.in[0], lo_bits, n, 8 * p, hist, chk, max_lo, max_hi,
                              st);
        else
            launch_hist<false>(ntiles, ksrc, nullptr, 0, n, 8 * p, hist, chk, max_lo, max_hi, st);
        NSD_TRY(check_launch("radix_hist_kernel"));
        NSD_TRY(scan_exclusive(hist, hist, ntiles * kBins, nullptr, scan_ws, st));
        probe_begin(NSD_KERNEL_SORT, st);
        const int sh = 8 * p;
        switch (np) {
            case 1: NSD_TRY(launch_scatter<1>(ntiles, ksrc, pl, kdst, n, lo_bits, sh, hist, st)); break;
            case 2: NSD_TRY(launch_scatter<2>(ntiles, ksrc, pl, kdst, n, lo_bits, sh, hist, st)); break;
            default: NSD_TRY(launch_scatter<3>(ntiles, ksrc, pl, kdst, n, lo_bits, sh, hist, st));
        }
        probe_end(NSD_KERNEL_SORT, st);
        ksrc = kdst;
        for (int j = 0; j < np; ++j) pl.in[j] = pl.out[j];
    }
    return NSD_OK;
}

nsd_status radix_sort_multi(int64_t n, int32_t max_key, const int32_t *key_in, int np,
                            const int32_t *const *payload_in, int32_t *key_out,
                            int32_t *const *payload_out, void *ws, hipStream_t st) {
    return radix_sort_passes(n, key_bits(max_key), 0, key_in, np, payload_in, key_out,
                             payload_out, ws, st);
}

// The same by the pair (hi, lo), hi in [0, max_hi) and lo in [0, max_lo):
// ordered by hi, then by lo, stable, in one sort of the combined bits.  The
// high words come in (and go out) as payload 0; lo is the key array.  The
// workspace is sort_ws_bytes(n, any, np).  *bad is set when a key is out of
// its range (the order is then unspecified).
static nsd_status radix_sort_pair_key(int64_t n, int32_t max_hi, int32_t max_lo,
                                      const int32_t *lo_in, int np,
                                      const int32_t *const *payload_in, int32_t *lo_out,
                                      int32_t *const *payload_out, void *ws, hipStream_t st,
                                      int32_t *bad) {
    if (np < 1 || payload_in[0] == nullptr)
        return fail(NSD_ERR_INVALID_ARG, "a pair key needs its high word as payload 0");
    const int lo_bits = std::max(key_bits(max_lo), 1);
    return radix_sort_passes(n, lo_bits + key_bits(max_hi), lo_bits, lo_in, np, payload_in,
                             lo_out, payload_out, ws, st, bad, max_lo, max_hi);
}

nsd_status radix_sort_pairs(int64_t n, int32_t max_key, const int32_t *key_in,
                            const int32_t *payload_in, int32_t *key_out, int32_t *payload_out,
                            void *ws, hipStream_t st) {
    return radix_sort_multi(n, max_key, key_in, 1, &payload_in, key_out, &payload_out, ws, st);
}

// ------------------------------------------------------- small kernels

constexpr int kThreads = 256;

static int64_t grid_for(int64_t n) { return ceil_div(n > 0 ? n : 1, kThreads); }

// Positions q of [0, n], kSegPer consecutive ones per thread: segment r
// starts at the first q whose key is >= r (q = n stands for key nseg).
constexpr int kSegPer = 4;

__global__ void segptr_kernel(int64_t n, int32_t nseg, const int32_t *key, int32_t *segptr) {
    const int64_t q0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kSegPer;
    if (q0 > n) return;
    // keys outside [0, nseg) (a malformed input) never write out of range
    int32_t prev = q0 == 0 ? -1 : min(key[q0 - 1], nseg);
    int32_t cur[kSegPer];
#pragma unroll
    for (int u = 0; u < kSegPer; ++u) {
        const int64_t q = q0 + u;
        cur[u] = q < n ? min(key[q], nseg) : nseg;
    }
#pragma unroll
    for (int u = 0; u < kSegPer; ++u) {
        const int64_t q = q0 + u;
        if (q > n) break;
        for (int32_t r = max(prev + 1, 0); r <= cur[u]; ++r) segptr[r] = (int32_t)q;
        prev = cur[u];
    }
}

// segptr_kernel over sorted (row, col) pairs that also adds to *ndup the
// positions whose pair equals the previous one (coordinates given more than
// once, beyond the first): one read of the sorted rows serves both.
__global__ void segptr_dups_kernel(int64_t n, int32_t nseg, const int32_t *key,
                                   const int32_t *col, int32_t *segptr, int32_t *ndup) {
    const int64_t q0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kSegPer;
    int dups = 0;
    if (q0 <= n) {
        int32_t prev = q0 == 0 ? -1 : min(key[q0 - 1], nseg);
        int32_t pcol = q0 == 0 ? -1 : col[q0 - 1];
        int32_t cur[kSegPer], cc[kSegPer];
#pragma unroll
        for (int u = 0; u < kSegPer; ++u) {
            const int64_t q = q0 + u;
            cur[u] = q < n ? min(key[q], nseg) : nseg;
            cc[u] = q < n ? col[q] : -1;
        }
#pragma unroll
        for (int u = 0; u < kSegPer; ++u) {
            const int64_t q = q0 + u;
            if (q > n) break;
            for (int32_t r = max(prev + 1, 0); r <= cur[u]; ++r) segptr[r] = (int32_t)q;
            dups += (q < n && q > 0 && cur[u] == prev && cc[u] == pcol) ? 1 : 0;
            prev = cur[u];
            pcol = cc[u];
        }
    }
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) dups += __shfl_xor(dups, m, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0 && dups) atomicAdd(ndup, dups);
}

nsd_status segptr_from_sorted(int64_t n, int32_t nseg, const int32_t *sorted_key,
                              int32_t *segptr, hipStream_t st) {
    segptr_kernel<<<grid_for(ceil_div(n + 1, kSegPer)), kThreads, 0, st>>>(n, nseg, sorted_key,
                                                                           segptr);
    return check_launch("segptr_kernel");
}

__global__ void expand_rows_kernel(int32_t nrows, int32_t nnz, const int32_t *rowptr,
                                   int32_t *rowidx) {
    const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= nnz) return;
    // last r with rowptr[r] <= p
    int32_t lo = 0, hi = nrows;
    while (hi - lo > 1) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (rowptr[mid] <= p) lo = mid;
        else hi = mid;
    }
    rowidx[p] = lo;
}

template <class T>
__global__ void gather_kernel(int64_t n, const int32_t *perm, const T *src, T *dst) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q < n) dst[q] = src[perm[q]];
}

__global__ void key_range_kernel(int64_t n, int32_t dim, const int32_t *key, int32_t *flag) {
    const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (p < n && (key[p] < 0 || key[p] >= dim)) atomicOr(flag, 1);
}

__global__ void run_heads_kernel(int64_t n, const int32_t *row_s, const int32_t *col_s,
                                 int32_t *head) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= n) return;
    head[q] = (q == 0 || row_s[q] != row_s[q - 1] || col_s[q] != col_s[q - 1]) ? 1 : 0;
}

// One thread per run of equal (row, col): the first occurrence names the
// output slot; duplicate values are added in input order.
__global__ void emit_runs_kernel(int64_t n, const int32_t *head, const int32_t *pos,
                                 const int32_t *row_s, const int32_t *col_s, const int32_t *perm,
                                 const float *val_s, int32_t *rowidx, int32_t *colind,
                                 float *val_out, int32_t *perm_out) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= n || !head[q]) return;
    const int32_t o = pos[q];
    float s = val_s[q];  // the values in sorted order; a run's in input order
    for (int64_t t = q + 1; t < n && !head[t]; ++t) s += val_s[t];
    rowidx[o] = row_s[q];
    colind[o] = col_s[q];
    perm_out[o] = perm[q];
    val_out[o] = s;
}

// One thread per row: rowptr monotone, columns in range (and strictly
// increasing when asked), rowidx consistent.  Bit 0: rowptr, bit 1: column
// range, bit 2: order, bit 3: rowidx.
__global__ void validate_csr_kernel(int32_t nrows, int32_t ncols, int32_t nnz,
                                    const int32_t *rowptr, const int32_t *rowidx,
                                    const int32_t *colind, int check_sorted, int32_t *flag) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r == 0 && (rowptr[0] != 0 || rowptr[nrows] != nnz)) atomicOr(flag, 1);
    if (r >= nrows) return;
    const int32_t b = rowptr[r], e = rowptr[r + 1];
    if (b > e || b < 0 || e > nnz) {
        atomicOr(flag, 1);
        return;
    }
    int32_t last = -1;
    for (int32_t p = b; p < e; ++p) {
        const int32_t c = colind[p];
        if (c < 0 || c >= ncols) atomicOr(flag, 2);
        if (check_sorted && c <= last) atomicOr(flag, 4);
        if (rowidx && rowidx[p] != r) atomicOr(flag, 8);
        last = c;
    }
}

// Coordinate arrays of a COO tensor, one per mode.
struct CoordArrays {
    const int32_t *p[NSD_MAX_ORDER];
};

// Flags (bit 2) an entry equal in every coordinate to the entry before it in
// lexicographic order perm.
__global__ void adjacent_equal_kernel(int64_t n, int order, CoordArrays c, const int32_t *perm,
                                      int32_t *flag) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q == 0 || q >= n) return;
    const int32_t a = perm[q], b = perm[q - 1];
    bool eq = true;
    for (int m = 0; m < order; ++m) eq = eq && c.p[m][a] == c.p[m][b];
    if (eq) atomicOr(flag, 2);
}

static size_t validate_coo_ws_bytes(int64_t n, int32_t max_dim) {
    Carver c(nullptr);
    c.take<int32_t>(64);  // flag
    for (int i = 0; i < 4; ++i) c.take<int32_t>(n > 0 ? n : 1);
    return c.bytes() + sort_ws_bytes(n, max_dim);
}

static nsd_status read_flag(int32_t *flag_dev, int32_t *flag_host, hipStream_t st) {
    NSD_HIP(hipMemcpyAsync(flag_host, flag_dev, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    return NSD_OK;
}

static bool too_large(int64_t v) { return v < 0 || v >= (int64_t(1) << 31); }

// n-element arrays a builder carves before the sort's own workspace
constexpr int kBuildArrays = 6;

}  // namespace nsd

using namespace nsd;

extern "C" {

nsd_status nsd_build_workspace_size(int32_t n, int32_t max_key, size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr, "bytes is NULL");
    NSD_REQUIRE(n >= 0 && max_key >= 1, "n must be >= 0 and max_key >= 1");
    Carver c(nullptr);
    for (int i = 0; i < kBuildArrays; ++i) c.take<int32_t>(n > 0 ? n : 1);
    c.take<int32_t>(64);
    *bytes = c.bytes() + sort_ws_bytes(n, max_key, kMaxPayloads) + scan_ws_bytes(n);
    return NSD_OK;
}

nsd_status nsd_csr_expand_rows(int32_t nrows, int32_t nnz, const int32_t *rowptr,
                               int32_t *rowidx, void *stream) {
    NSD_REQUIRE(nrows >= 0 && nnz >= 0, "negative size");
    NSD_REQUIRE(rowptr != nullptr && (nnz == 0 || rowidx != nullptr), "null pointer");
    if (nnz == 0) return NSD_OK;
    NSD_REQUIRE(nrows > 0, "nnz > 0 needs nrows > 0");
    expand_rows_kernel<<<grid_for(nnz), kThreads, 0, as_stream(stream)>>>(nrows, nnz, rowptr,
                                                                           rowidx);
    return check_launch("expand_rows_kernel");
}

nsd_status nsd_gather_f32(int32_t n, const int32_t *perm, const float *src, float *dst,
                          void *stream) {
    NSD_REQUIRE(n >= 0, "negative size");
    if (n == 0) return NSD_OK;
    NSD_REQUIRE(perm && src && dst, "null pointer");
    gather_kernel<float><<<grid_for(n), kThreads, 0, as_stream(stream)>>>(n, perm, src, dst);
    return check_launch("gather_kernel");
}

nsd_status nsd_gather_i32(int32_t n, const int32_t *perm, const int32_t *src, int32_t *dst,
                          void *stream) {
    NSD_REQUIRE(n >= 0, "negative size");
    if (n == 0) return NSD_OK;
    NSD_REQUIRE(perm && src && dst, "null pointer");
    gather_kernel<int32_t><<<grid_for(n), kThreads, 0, as_stream(stream)>>>(n, perm, src, dst);
    return check_launch("gather_kernel");
}

nsd_status nsd_coo_to_csr(int32_t nrows, int32_t ncols, int32_t nnz, const int32_t *row,
                          const int32_t *col, const float *val, int policy, int32_t *rowptr,
                          int32_t *rowidx, int32_t *colind, float *val_out, int32_t *perm,
                          int32_t *nnz_out, void *ws, size_t ws_bytes, void *stream) {
    NSD_REQUIRE(nrows >= 0 && ncols >= 0 && nnz >= 0, "negative size");
    NSD_REQUIRE(policy == NSD_DUP_SUM || policy == NSD_DUP_ERROR, "unknown duplicate policy %d",
                policy);
    NSD_REQUIRE(rowptr && nnz_out, "null pointer");
    NSD_REQUIRE(nnz == 0 || (row && col && val && rowidx && colind && val_out && perm && ws),
                "null pointer");
    const int32_t max_key = std::max(std::max(nrows, ncols), 1);
    size_t need;
    NSD_TRY(nsd_build_workspace_size(nnz, max_key, &need));
    if (nnz > 0 && ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
    hipStream_t st = as_stream(stream);
    if (nnz == 0) {
        NSD_HIP(hipMemsetAsync(rowptr, 0, sizeof(int32_t) * (nrows + 1), st));
        NSD_HIP(hipStreamSynchronize(st));
        *nnz_out = 0;
        return NSD_OK;
    }
    NSD_REQUIRE(nrows > 0 && ncols > 0, "nnz > 0 needs a non-empty shape");
    Carver c(ws);
    int32_t *row_s = c.take<int32_t>(nnz);
    int32_t *pm = c.take<int32_t>(nnz);
    int32_t *col_s = c.take<int32_t>(nnz);
    int32_t *val_s = c.take<int32_t>(nnz);
    int32_t *head = c.take<int32_t>(nnz);
    int32_t *pos = c.take<int32_t>(nnz);
    static_assert(kBuildArrays >= 6, "the arrays above");
    int32_t *flag = c.take<int32_t>(64);
    void *sort_ws = c.base + c.bytes();
    void *scan_ws = static_cast<char *>(sort_ws) + sort_ws_bytes(nnz, max_key, kMaxPayloads);

    // one stable sort by the pair (row, col), ties in input order, straight
    // into the outputs: the row (the key's high word), the input position
    // and the value's bits travel with the column; its first pass checks
    // the coordinates' ranges (flag[0]).  With coordinates in range and
    // distinct (counted next, flag[1]) the sorted arrays are the CSR.
    NSD_HIP(hipMemsetAsync(flag, 0, 2 * sizeof(int32_t), st));
    {
        const int32_t *in[3] = {row, nullptr, reinterpret_cast<const int32_t *>(val)};
        int32_t *out[3] = {rowidx, perm, reinterpret_cast<int32_t *>(val_out)};
        NSD_TRY(radix_sort_pair_key(nnz, nrows, ncols, col, 3, in, colind, out, sort_ws, st,
                                    flag));
    }
    // the row pointers as if the coordinates were distinct, and how many
    // are not
    segptr_dups_kernel<<<grid_for(ceil_div(nnz + 1, kSegPer)), kThreads, 0, st>>>(
        nnz, nrows, rowidx, colind, rowptr, flag + 1);
    NSD_TRY(check_launch("segptr_dups_kernel"));
    int32_t fl[2] = {0, 0};
    NSD_HIP(hipMemcpyAsync(fl, flag, sizeof(fl), hipMemcpyDeviceToHost, st));
    NSD_HIP(hipStreamSynchronize(st));
    if (fl[0]) return fail(NSD_ERR_BAD_FORMAT, "COO coordinate out of range");
    const int32_t ndup = fl[1];
    if (ndup > 0 && policy == NSD_DUP_ERROR)
        return fail(NSD_ERR_DUPLICATE, "%d duplicate coordinates", ndup);
    int32_t nuniq = nnz;
    if (ndup > 0) {
        // merge the runs of equal (row, col): the sorted arrays move to the
        // workspace and come back one entry per run
        const size_t b = sizeof(int32_t) * (size_t)nnz;
        NSD_HIP(hipMemcpyAsync(row_s, rowidx, b, hipMemcpyDeviceToDevice, st));
        NSD_HIP(hipMemcpyAsync(col_s, colind, b, hipMemcpyDeviceToDevice, st));
        NSD_HIP(hipMemcpyAsync(pm, perm, b, hipMemcpyDeviceToDevice, st));
        NSD_HIP(hipMemcpyAsync(val_s, val_out, b, hipMemcpyDeviceToDevice, st));
        run_heads_kernel<<<grid_for(nnz), kThreads, 0, st>>>(nnz, row_s, col_s, head);
        NSD_TRY(check_launch("run_heads_kernel"));
        NSD_TRY(scan_exclusive(head, pos, nnz, flag + 2, scan_ws, st));
        NSD_TRY(read_flag(flag + 2, &nuniq, st));
        emit_runs_kernel<<<grid_for(nnz), kThreads, 0, st>>>(
            nnz, head, pos, row_s, col_s, pm, reinterpret_cast<const float *>(val_s), rowidx,
            colind, val_out, perm);
        NSD_TRY(check_launch("emit_runs_kernel"));
        NSD_TRY(segptr_from_sorted(nuniq, nrows, rowidx, rowptr, st));
    }
    NSD_HIP(hipStreamSynchronize(st));
    *nnz_out = nuniq;
    return NSD_OK;
}

nsd_status nsd_csr_to_csc(const nsd_csr *A, int32_t *colptr, int32_t *colidx, int32_t *rowind,
                          int32_t *perm, void *ws, size_t ws_bytes, void *stream) {
    NSD_REQUIRE(A != nullptr && colptr != nullptr, "null pointer");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative size");
    hipStream_t st = as_stream(stream);
    const int32_t nnz = A->nnz;
    if (nnz > 0) {
        NSD_REQUIRE(A->rowidx && A->colind && colidx && rowind && perm && ws, "null pointer");
        size_t need;
        NSD_TRY(nsd_build_workspace_size(nnz, std::max(A->ncols, 1), &need));
        if (ws_bytes < need) return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
        Carver c(ws);
        for (int i = 0; i < kBuildArrays; ++i) c.take<int32_t>(nnz);
        int32_t *flag = c.take<int32_t>(64);
        void *sort_ws = c.base + c.bytes();
        // the CSR slot and its row travel with the column keys; the sort's
        // first pass checks the columns' range
        NSD_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
        const int32_t *in[2] = {nullptr, A->rowidx};
        int32_t *out[2] = {perm, rowind};
        NSD_TRY(radix_sort_passes(nnz, key_bits(std::max(A->ncols, 1)), 0, A->colind, 2, in,
                                  colidx, out, sort_ws, st, flag, A->ncols));
        NSD_TRY(segptr_from_sorted(nnz, A->ncols, colidx, colptr, st));
        int32_t h = 0;
        NSD_TRY(read_flag(flag, &h, st));
        if (h) return fail(NSD_ERR_BAD_FORMAT, "column index out of range [0, %d)", A->ncols);
        return NSD_OK;
    }
    NSD_TRY(segptr_from_sorted(nnz, A->ncols, colidx, colptr, st));
    NSD_HIP(hipStreamSynchronize(st));
    return NSD_OK;
}

nsd_status nsd_coo_mode_index(int32_t nnz, int32_t dim, const int32_t *key, int32_t *segptr,
                              int32_t *segidx, int32_t *perm, void *ws, size_t ws_bytes,
                              void *stream) {
    NSD_REQUIRE(nnz >= 0 && dim >= 1, "need nnz >= 0 and dim >= 1");
    NSD_REQUIRE(segptr != nullptr, "null pointer");
    hipStream_t st = as_stream(stream);
    if (nnz > 0) {
        NSD_REQUIRE(key && segidx && perm && ws, "null pointer");
        size_t need;
        NSD_TRY(nsd_build_workspace_size(nnz, dim, &need));
        if (ws_bytes < need) return fail(NSD_ERR_WORKSPACE, "workspace %zu < %zu", ws_bytes, need);
        Carver c(ws);
        for (int i = 0; i < kBuildArrays; ++i) c.take<int32_t>(nnz);
        int32_t *flag = c.take<int32_t>(64);
        void *sort_ws = c.base + c.bytes();
        // the sort's first pass checks the keys' range
        NSD_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
        const int32_t *in[1] = {nullptr};
        int32_t *out[1] = {perm};
        NSD_TRY(radix_sort_passes(nnz, key_bits(dim), 0, key, 1, in, segidx, out, sort_ws, st,
                                  flag, dim));
        NSD_TRY(segptr_from_sorted(nnz, dim, segidx, segptr, st));
        int32_t h = 0;
        NSD_TRY(read_flag(flag, &h, st));
        if (h) return fail(NSD_ERR_BAD_FORMAT, "key out of range [0, %d)", dim);
        return NSD_OK;
    }
    NSD_TRY(segptr_from_sorted(nnz, dim, segidx, segptr, st));
    NSD_HIP(hipStreamSynchronize(st));
    return NSD_OK;
}

nsd_status nsd_validate_coo_workspace_size(int32_t order, const int32_t *dims, int32_t nnz,
                                           size_t *bytes) {
    NSD_REQUIRE(bytes != nullptr && dims != nullptr, "null pointer");
    NSD_REQUIRE(order >= 2 && order <= NSD_MAX_ORDER, "order %d outside [2, %d]", order,
                NSD_MAX_ORDER);
    NSD_REQUIRE(nnz >= 0, "negative nnz");
    int32_t max_dim = 1;
    for (int m = 0; m < order; ++m) {
        NSD_REQUIRE(dims[m] >= 0, "negative dimension");
        max_dim = std::max(max_dim, dims[m]);
    }
    *bytes = validate_coo_ws_bytes(nnz, max_dim);
    return NSD_OK;
}

nsd_status nsd_validate_coo(int32_t order, const int32_t *dims, int32_t nnz,
                            const int32_t *const *coords, int check_unique, void *ws,
                            size_t ws_bytes, void *stream) {
    size_t need = 0;
    NSD_TRY(nsd_validate_coo_workspace_size(order, dims, nnz, &need));
    if (nnz == 0) return NSD_OK;
    NSD_REQUIRE(coords != nullptr, "coords is NULL");
    CoordArrays c;
    int32_t max_dim = 1;
    for (int m = 0; m < order; ++m) {
        NSD_REQUIRE(coords[m] != nullptr, "coordinate array %d is NULL", m);
        NSD_REQUIRE(dims[m] >= 1, "nnz > 0 needs non-empty dimensions");
        c.p[m] = coords[m];
        max_dim = std::max(max_dim, dims[m]);
    }
    if (ws == nullptr || ws_bytes < need)
        return fail(NSD_ERR_WORKSPACE, "workspace %zu bytes at %p, need %zu", ws_bytes, ws, need);
    hipStream_t st = as_stream(stream);
    Carver cv(ws);
    int32_t *flag = cv.take<int32_t>(64);
    int32_t *key = cv.take<int32_t>(nnz);
    int32_t *key_sorted = cv.take<int32_t>(nnz);
    int32_t *perm[2] = {cv.take<int32_t>(nnz), cv.take<int32_t>(nnz)};
    void *sort_ws = cv.base + cv.bytes();
    NSD_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
    for (int m = 0; m < order; ++m) {
        key_range_kernel<<<grid_for(nnz), kThreads, 0, st>>>(nnz, dims[m], c.p[m], flag);
        NSD_TRY(check_launch("key_range_kernel"));
    }
    int32_t h = 0;
    NSD_TRY(read_flag(flag, &h, st));
    if (h) return fail(NSD_ERR_BAD_FORMAT, "COO coordinate out of range");
    if (!check_unique || nnz < 2) return NSD_OK;
    // lexicographic order: stable sorts by the last coordinate first
    const int32_t *pm = nullptr;
    int cur = 0;
    for (int m = order - 1; m >= 0; --m) {
        const int32_t *k = c.p[m];
        if (pm) {
            gather_kernel<int32_t><<<grid_for(nnz), kThreads, 0, st>>>(nnz, pm, c.p[m], key);
            NSD_TRY(check_launch("gather_kernel"));
            k = key;
        }
        NSD_TRY(radix_sort_pairs(nnz, dims[m], k, pm, key_sorted, perm[cur], sort_ws, st));
        pm = perm[cur];
        cur ^= 1;
    }
    adjacent_equal_kernel<<<grid_for(nnz), kThreads, 0, st>>>(nnz, order, c, pm, flag);
    NSD_TRY(check_launch("adjacent_equal_kernel"));
    NSD_TRY(read_flag(flag, &h, st));
    if (h) return fail(NSD_ERR_DUPLICATE, "COO coordinates repeat a key");
    return NSD_OK;
}

nsd_status nsd_validate_csr(const nsd_csr *A, int check_sorted, void *ws, size_t ws_bytes,
                            void *stream) {
    NSD_REQUIRE(A != nullptr && A->rowptr != nullptr, "null pointer");
    NSD_REQUIRE(A->nrows >= 0 && A->ncols >= 0 && A->nnz >= 0, "negative size");
    NSD_REQUIRE(A->nnz == 0 || A->colind != nullptr, "null colind");
    NSD_REQUIRE(ws != nullptr && ws_bytes >= 256, "validation needs 256 bytes of workspace");
    hipStream_t st = as_stream(stream);
    int32_t *flag = static_cast<int32_t *>(ws);
    NSD_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t), st));
    validate_csr_kernel<<<grid_for(A->nrows + 1), kThreads, 0, st>>>(
        A->nrows, A->ncols, A->nnz, A->rowptr, A->rowidx, A->colind, check_sorted, flag);
    NSD_TRY(check_launch("validate_csr_kernel"));
    int32_t h = 0;
    NSD_TRY(read_flag(flag, &h, st));
    if (h) {
        return fail(NSD_ERR_BAD_FORMAT, "malformed CSR:%s%s%s%s", (h & 1) ? " rowptr" : "",
                    (h & 2) ? " column-range" : "", (h & 4) ? " column-order" : "",
                    (h & 8) ? " rowidx" : "");
    }
    return NSD_OK;
}

}  // extern "C"
