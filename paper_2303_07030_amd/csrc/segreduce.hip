// Segmented gather-reduce and sampled dense-dense products.
//
// Gather-reduce computes, for every segment s of a sorted sparse operand
// (a row of a CSR, or a column of its CSC),
//     out[s, :] = alpha * sum_{p in s} w_p * X[idx_p, :]
// which is SpMV / SpMM (segments = rows, idx = colind, w = val) and the
// transposed product A^T G (segments = columns, idx = rowind, w = val[perm]).
// It is the `sum(<j, a> in row) a * X(j)` of the paper's matrix product with
// the singleton insert "+=" of its code generation (Section 5.5), done so that
// every output is written once, with no atomics.
//
// Load balance: the nnz are cut into equal slots of L entries, independent of
// where rows begin (nnz-split).  A slot is G lanes holding VEC floats of a
// dense row each (VEC * G = up to 256 columns per pass).  Inside a slot the
// entries are walked in order with U gathers in flight; a row that starts and
// ends inside the slot is written directly (alpha applied), and the partial
// sums of rows that cross a slot boundary go to per-slot carries.  A second
// kernel adds, for every row that spans slots, its owner's partial and the
// following slots' partials in slot order.  Power-law rows therefore cost the
// same per nnz as short ones, and results are bitwise deterministic.
//
// Empty rows are written as zeros by the slot that holds the entry just
// before them (slot 0 for leading empty rows, the last slot for trailing ones).
#include <algorithm>

#include "nsd_internal.hpp"
#include "segreduce.hpp"

namespace nsd {

constexpr int kBlock = 256;

template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void sgr_main_kernel(SgrParams a) {
    constexpr int kSlots = kBlock / G;
    const int g = threadIdx.x % G;
    const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
    if (s >= a.nslots) return;
    const int col = blockIdx.y * (G * VEC) + g * VEC;
    const bool on = col < a.k;
    const int64_t k = a.k;
    const int64_t a0 = s * a.L;
    const int64_t b0 = min(a0 + (int64_t)a.L, (int64_t)a.nnz);

    int row = a.segidx[a0];
    bool carry = a0 > 0 && a.segidx[a0 - 1] == row;

    Vec<VEC> zero;
    zero.zero();
    auto zero_rows = [&](int r0, int r1) {
        if (on)
            for (int r = r0; r < r1; ++r) zero.store(a.out + (int64_t)r * k + col);
    };
    Vec<VEC> acc;
    acc.zero();
    auto flush = [&]() {
        if (!on) return;
        if (carry) {
            acc.store(a.pfirst + s * k + col);
        } else {
            Vec<VEC> t = acc;
            t.scale(a.alpha);
            t.store(a.out + (int64_t)row * k + col);
        }
    };
    auto weight = [&](int64_t p) -> float {
        if (!a.w) return 1.f;
        return a.wperm ? a.w[a.wperm[p]] : a.w[p];
    };

    if (s == 0) zero_rows(0, row);

    int64_t p = a0;
    for (; p + U <= b0; p += U) {
        int r[U], c[U];
        float wt[U];
        Vec<VEC> xv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            r[u] = a.segidx[p + u];
            c[u] = a.idx[p + u];
            wt[u] = weight(p + u);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (a.X && on) xv[u].load(a.X + (int64_t)c[u] * k + col);
            else xv[u].ones();
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (r[u] != row) {
                flush();
                zero_rows(row + 1, r[u]);
                row = r[u];
                carry = false;
                acc.zero();
            }
            acc.fma(wt[u], xv[u]);
        }
    }
    for (; p < b0; ++p) {
        const int r = a.segidx[p];
        const int c = a.idx[p];
        const float wt = weight(p);
        Vec<VEC> xv;
        if (a.X && on) xv.load(a.X + (int64_t)c * k + col);
        else xv.ones();
        if (r != row) {
            flush();
            zero_rows(row + 1, r);
            row = r;
            carry = false;
            acc.zero();
        }
        acc.fma(wt, xv);
    }

    const bool ends = b0 == a.nnz || a.segidx[b0] != row;
    const bool lead = g == 0 && blockIdx.y == 0;
    if (ends) {
        flush();
        zero_rows(row + 1, b0 == a.nnz ? a.nseg : a.segidx[b0]);
        if (lead) a.span[s] = -1;
    } else if (carry) {
        if (on) acc.store(a.pfirst + s * k + col);
        if (lead) a.span[s] = -1;
    } else {
        if (on) acc.store(a.plast + s * k + col);
        if (lead) a.span[s] = row;
    }
}

// One block per slot.  For a slot that owns a row continuing past its end,
// out[row] = alpha * (plast[s] + sum_{t = s+1..t_end} pfirst[t]); the four
// waves take interleaved t and are added in a fixed order.
template <int VEC>
__global__ __launch_bounds__(kBlock) void sgr_fix_kernel(SgrParams a) {
    const int64_t s = blockIdx.x;
    const int r = a.span[s];
    if (r < 0) return;
    const int64_t k = a.k;
    const int64_t t_end = ((int64_t)a.segptr[r + 1] - 1) / a.L;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    __shared__ float part[kBlock / kWave][kWave * VEC];
    for (int c0 = 0; c0 < a.k; c0 += kWave * VEC) {
        const int col = c0 + lane * VEC;
        const bool on = col < a.k;
        Vec<VEC> acc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i].zero();
        if (on) {
            int64_t t = s + 1 + wave;
            for (; t + 12 <= t_end; t += 16) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    Vec<VEC> x;
                    x.load(a.pfirst + (t + 4 * i) * k + col);
                    acc[i].add(x);
                }
            }
            for (int i = 0; t <= t_end; t += 4, ++i) {
                Vec<VEC> x;
                x.load(a.pfirst + t * k + col);
                acc[i & 3].add(x);
            }
        }
        acc[0].add(acc[1]);
        acc[2].add(acc[3]);
        acc[0].add(acc[2]);
#pragma unroll
        for (int i = 0; i < VEC; ++i) part[wave][lane * VEC + i] = acc[0].v[i];
        __syncthreads();
        if (wave == 0 && on) {
            Vec<VEC> tot;
            tot.load(a.plast + s * k + col);
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                const int e = lane * VEC + i;
                tot.v[i] += (part[0][e] + part[1][e]) + (part[2][e] + part[3][e]);
            }
            tot.scale(a.alpha);
            tot.store(a.out + (int64_t)r * k + col);
        }
        __syncthreads();
    }
}

// Zero-fill of a whole output when there is nothing to reduce.
__global__ void fill_zero_kernel(float *out, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] = 0.f;
}

int choose_slot_len(int64_t nnz, int slots_per_wave) {
    // aim for ~8192 waves (8 per SIMD on 256 CUs); 16 <= L <= 256
    const int64_t target = 8192LL * slots_per_wave;
    int L = 16;
    while (L < 256 && (int64_t)L * 2 * target <= nnz) L <<= 1;
    return L;
}

SgrShape sgr_shape(int64_t nnz, int k) {
    SgrShape sh;
    sh.wp = width_plan(k, true);
    sh.L = choose_slot_len(nnz, kWave / sh.wp.g);
    sh.nslots = nnz > 0 ? ceil_div(nnz, sh.L) : 0;
    return sh;
}

void sgr_carve(Carver &c, int64_t nnz, int k, SgrParams *p) {
    const SgrShape sh = sgr_shape(nnz, k);
    // sized for the smallest slot length either lane layout can choose
    const SgrShape sh1 = sgr_shape_vec1(nnz, k);
    const int64_t ns = std::max<int64_t>({sh.nslots, sh1.nslots, 1});
    float *pf = c.take<float>(ns * k);
    float *pl = c.take<float>(ns * k);
    int32_t *sp = c.take<int32_t>(ns);
    if (p) {
        p->pfirst = pf;
        p->plast = pl;
        p->span = sp;
    }
}

// Slot length and count for the lane layout segreduce will launch.
static void sgr_finalize_shape(SgrParams &a, const WidthPlan &wp) {
    a.L = choose_slot_len(a.nnz, kWave / wp.g);
    a.nslots = (int32_t)ceil_div(a.nnz, a.L);
}

template <int VEC, int G>
static void launch_sgr_vg(const SgrParams &a, hipStream_t st) {
    constexpr int U = G >= 16 ? 4 : 8;
    constexpr int kSlots = kBlock / G;
    dim3 grid((unsigned)ceil_div(a.nslots, kSlots), (unsigned)ceil_div(a.k, G * VEC));
    sgr_main_kernel<VEC, G, U><<<grid, kBlock, 0, st>>>(a);
    sgr_fix_kernel<VEC><<<(unsigned)a.nslots, kBlock, 0, st>>>(a);
}

SgrShape sgr_shape_vec1(int64_t nnz, int k) {
    SgrShape sh;
    sh.wp = width_plan(k, false);
    sh.L = choose_slot_len(nnz, kWave / sh.wp.g);
    sh.nslots = nnz > 0 ? ceil_div(nnz, sh.L) : 0;
    return sh;
}

static bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

nsd_status segreduce(SgrParams a, hipStream_t st) {
    const int64_t total = (int64_t)a.nseg * a.k;
    if (a.nnz == 0) {
        if (total > 0) fill_zero_kernel<<<ceil_div(total, 256), 256, 0, st>>>(a.out, total);
        return check_launch("fill_zero_kernel");
    }
    // float4 lanes need 16-byte aligned dense rows; otherwise use scalar lanes
    const WidthPlan wp = width_plan(a.k, aligned16(a.out) && (!a.X || aligned16(a.X)));
    sgr_finalize_shape(a, wp);
    if (wp.vec == 4) {
        switch (wp.g) {
            case 1: launch_sgr_vg<4, 1>(a, st); break;
            case 2: launch_sgr_vg<4, 2>(a, st); break;
            case 4: launch_sgr_vg<4, 4>(a, st); break;
            case 8: launch_sgr_vg<4, 8>(a, st); break;
            case 16: launch_sgr_vg<4, 16>(a, st); break;
            case 32: launch_sgr_vg<4, 32>(a, st); break;
            default: launch_sgr_vg<4, 64>(a, st); break;
        }
    } else {
        switch (wp.g) {
            case 1: launch_sgr_vg<1, 1>(a, st); break;
            case 2: launch_sgr_vg<1, 2>(a, st); break;
            case 4: launch_sgr_vg<1, 4>(a, st); break;
            case 8: launch_sgr_vg<1, 8>(a, st); break;
            case 16: launch_sgr_vg<1, 16>(a, st); break;
            case 32: launch_sgr_vg<1, 32>(a, st); break;
            default: launch_sgr_vg<1, 64>(a, st); break;
        }
    }
    return check_launch("segreduce");
}

// ------------------------------------------------------------------ SDDMM

// Reduces U partial dot products across the G lanes of a slot with a
// transposing butterfly: at each step a lane keeps half of its values and
// receives the partner's matching half, so U values cost U - 1 exchanges
// plus log2(G / U) for the last one.  Lane g ends with the total of value
// number g / (G / U).
template <int G, int U>
__device__ __forceinline__ float transpose_reduce(float (&v)[U], int lane) {
    int c = U;
#pragma unroll
    for (int m = G / 2; m >= 1; m >>= 1) {
        if (c > 1) {
            const bool upper = (lane & m) != 0;
#pragma unroll
            for (int i = 0; i < U / 2; ++i) {
                if (i < c / 2) {
                    const float send = upper ? v[i] : v[i + c / 2];
                    const float keep = upper ? v[i + c / 2] : v[i];
                    v[i] = keep + shfl_xor(send, m);
                }
            }
            c >>= 1;
        } else {
            v[0] += shfl_xor(v[0], m);
        }
    }
    return v[0];
}

template <int VEC, int G, int U>
__global__ __launch_bounds__(kBlock) void sddmm_kernel(SddmmParams a) {
    constexpr int kSlots = kBlock / G;
    const int lane = threadIdx.x % kWave;
    const int g = threadIdx.x % G;
    const int64_t s = (int64_t)blockIdx.x * kSlots + threadIdx.x / G;
    const int64_t k = a.k;
    double lsum = 0.0;
    if (s < a.nslots) {
        const int64_t a0 = s * a.L;
        const int64_t b0 = min(a0 + (int64_t)a.L, (int64_t)a.nnz);
        for (int64_t p = a0; p < b0; p += U) {
            int rr[U], cc[U];
            float part[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const bool valid = p + u < b0;
                rr[u] = valid ? a.rowidx[p + u] : 0;
                cc[u] = valid ? a.colind[p + u] : 0;
                part[u] = 0.f;
            }
            for (int c0 = 0; c0 < a.k; c0 += G * VEC) {
                const int col = c0 + g * VEC;
                const bool on = col < a.k;
                Vec<VEC> xv[U], yv[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (on && p + u < b0) {
                        if (a.X) xv[u].load(a.X + (int64_t)rr[u] * k + col);
                        else xv[u].ones();
                        yv[u].load(a.Y + (int64_t)cc[u] * k + col);
                    } else {
                        xv[u].zero();
                        yv[u].zero();
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u) part[u] += xv[u].dot(yv[u]);
            }
            if constexpr (G == 1) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if (p + u < b0) {
                        a.out[p + u] = a.alpha * part[u];
                        if (a.w) lsum += (double)a.w[p + u] * (double)part[u];
                    }
                }
            } else {
                const float tot = transpose_reduce<G, U>(part, lane);
                constexpr int kRep = G / U;
                const int64_t q = p + g / kRep;
                if (g % kRep == 0 && q < b0) {
                    a.out[q] = a.alpha * tot;
                    if (a.w) lsum += (double)a.w[q] * (double)tot;
                }
            }
        }
    }
    if (a.part) {
        // block total of the fused loss, fixed order
        __shared__ double wsum[kBlock / kWave];
#pragma unroll
        for (int m = kWave / 2; m >= 1; m >>= 1) lsum += __shfl_xor(lsum, m, kWave);
        if (lane == 0) wsum[threadIdx.x / kWave] = lsum;
        __syncthreads();
        if (threadIdx.x == 0)
            a.part[blockIdx.x] = a.beta * ((wsum[0] + wsum[1]) + (wsum[2] + wsum[3]));
    }
}

SddmmShape sddmm_shape(int64_t nnz, int k, bool vec_ok) {
    SddmmShape sh;
    sh.wp = width_plan(k, vec_ok);
    const int slots_per_block = kBlock / sh.wp.g;
    sh.L = choose_slot_len(nnz, kWave / sh.wp.g);
    sh.nslots = nnz > 0 ? ceil_div(nnz, sh.L) : 0;
    sh.nblocks = sh.nslots > 0 ? ceil_div(sh.nslots, slots_per_block) : 0;
    return sh;
}

bool sddmm_vec_ok(const SddmmParams &a) { return (!a.X || aligned16(a.X)) && aligned16(a.Y); }

template <int VEC, int G>
static void launch_sddmm_vg(const SddmmParams &a, int64_t nblocks, hipStream_t st) {
    constexpr int U = G >= 8 ? 8 : (G == 1 ? 4 : G);
    sddmm_kernel<VEC, G, U><<<(unsigned)nblocks, kBlock, 0, st>>>(a);
}

nsd_status sddmm(SddmmParams a, hipStream_t st) {
    const SddmmShape sh = sddmm_shape(a.nnz, a.k, sddmm_vec_ok(a));
    a.L = sh.L;
    a.nslots = (int32_t)sh.nslots;
    if (sh.nblocks == 0) return NSD_OK;
    if (sh.wp.vec == 4) {
        switch (sh.wp.g) {
            case 1: launch_sddmm_vg<4, 1>(a, sh.nblocks, st); break;
            case 2: launch_sddmm_vg<4, 2>(a, sh.nblocks, st); break;
            case 4: launch_sddmm_vg<4, 4>(a, sh.nblocks, st); break;
            case 8: launch_sddmm_vg<4, 8>(a, sh.nblocks, st); break;
            case 16: launch_sddmm_vg<4, 16>(a, sh.nblocks, st); break;
            case 32: launch_sddmm_vg<4, 32>(a, sh.nblocks, st); break;
            default: launch_sddmm_vg<4, 64>(a, sh.nblocks, st); break;
        }
    } else {
        switch (sh.wp.g) {
            case 1: launch_sddmm_vg<1, 1>(a, sh.nblocks, st); break;
            case 2: launch_sddmm_vg<1, 2>(a, sh.nblocks, st); break;
            case 4: launch_sddmm_vg<1, 4>(a, sh.nblocks, st); break;
            case 8: launch_sddmm_vg<1, 8>(a, sh.nblocks, st); break;
            case 16: launch_sddmm_vg<1, 16>(a, sh.nblocks, st); break;
            case 32: launch_sddmm_vg<1, 32>(a, sh.nblocks, st); break;
            default: launch_sddmm_vg<1, 64>(a, sh.nblocks, st); break;
        }
    }
    return check_launch("sddmm_kernel");
}

// ------------------------------------------------------------ loss total

// One block: strided partial sums per thread, then a fixed tree.
__global__ __launch_bounds__(kBlock) void loss_finalize_kernel(const double *part, int64_t n,
                                                               double *loss) {
    __shared__ double sh[kBlock];
    double s = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += kBlock) s += part[i];
    sh[threadIdx.x] = s;
    __syncthreads();
    for (int w = kBlock / 2; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w) sh[threadIdx.x] += sh[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = sh[0];
}

nsd_status loss_finalize(const double *part, int64_t n, double *loss, hipStream_t st) {
    loss_finalize_kernel<<<1, kBlock, 0, st>>>(part, n, loss);
    return check_launch("loss_finalize_kernel");
}

}  // namespace nsd
