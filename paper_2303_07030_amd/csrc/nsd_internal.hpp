// Internal helpers of libnsd: error state, workspace carving, wave-level
// device utilities.  gfx950 only: 64-lane wavefronts throughout.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstddef>
#include <cstdint>

#include "nsd.h"

namespace nsd {

constexpr int kWave = 64;

// ------------------------------------------------------------ error state

void set_error(const char *fmt, ...);
void clear_error();
nsd_status fail(nsd_status s, const char *fmt, ...);
// Maps a pending launch / runtime error to NSD_ERR_HIP with its message.
nsd_status check_hip(hipError_t e, const char *what);
nsd_status check_launch(const char *what);

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Timing probe hooks around a kernel launch (no-ops unless a probe is set
// on this thread for that kernel id).
void probe_begin(int kernel_id, hipStream_t st);
void probe_end(int kernel_id, hipStream_t st);

#define NSD_REQUIRE(cond, ...)                                   \
    do {                                                         \
        if (!(cond)) return ::nsd::fail(NSD_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)

#define NSD_TRY(expr)                                            \
    do {                                                         \
        nsd_status _s = (expr);                                  \
        if (_s != NSD_OK) return _s;                             \
    } while (0)

#define NSD_HIP(expr) NSD_TRY(::nsd::check_hip((expr), #expr))

// ---------------------------------------------------------- workspace

// Hands out 256-byte aligned pieces of a caller workspace.  With base == NULL
// it only measures, which is how the size queries are computed, so the
// queries and the carving can never disagree.
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base(static_cast<char *>(b)) {}
    template <class T>
    T *take(size_t count) {
        off = (off + 255) & ~size_t(255);
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
    size_t bytes() const { return (off + 255) & ~size_t(255); }
};

// ------------------------------------------------------------ sizes

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// --------------------------------------------------- device utilities

__device__ __forceinline__ float shfl_xor(float v, int m) { return __shfl_xor(v, m, kWave); }

// v of this lane's partner in a butterfly step of span M: a lane of the
// other half of its aligned 2M-lane group.  Spans 1 and 2 pair lane i with
// i ^ M (DPP quad permutation), spans 4 and 8 mirror the group (i with
// 2M - 1 - i: DPP row half-mirror and row mirror), span 16 pairs i ^ 16
// (swizzle within 32 lanes), span 32 goes through the LDS crossbar.  A
// butterfly sum over all lanes is the same with either pairing; the DPP
// forms are plain VALU moves instead of LDS round trips.
template <int M>
__device__ __forceinline__ float lane_xor(float v) {
    const int x = __float_as_int(v);
    if constexpr (M == 1) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false));
    } else if constexpr (M == 2) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false));
    } else if constexpr (M == 4) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x141, 0xF, 0xF, false));
    } else if constexpr (M == 8) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(x, 0x140, 0xF, 0xF, false));
    } else if constexpr (M == 16) {
        return __int_as_float(__builtin_amdgcn_ds_swizzle(x, (16 << 10) | 0x1F));
    } else {
        return __shfl_xor(v, M, kWave);
    }
}

template <int VEC>
struct Vec;

template <>
struct Vec<4> {
    float v[4];
    __device__ __forceinline__ void zero() { v[0] = v[1] = v[2] = v[3] = 0.f; }
    __device__ __forceinline__ void ones() { v[0] = v[1] = v[2] = v[3] = 1.f; }
    __device__ __forceinline__ void load(const float *p) {
        const float4 t = *reinterpret_cast<const float4 *>(p);
        v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
    }
    __device__ __forceinline__ void store(float *p) const {
        *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
    }
    // Streamed data, read or written once (a segment's own row, its output
    // row): non-temporal, so that it displaces less of what the L2 holds
    // for reuse (the gathered rows).
    __device__ __forceinline__ void load_nt(const float *p) {
        typedef float f4 __attribute__((ext_vector_type(4)));
        const f4 t = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p));
        v[0] = t.x;
        v[1] = t.y;
        v[2] = t.z;
        v[3] = t.w;
    }
    __device__ __forceinline__ void store_nt(float *p) const {
        typedef float f4 __attribute__((ext_vector_type(4)));
        const f4 t = {v[0], v[1], v[2], v[3]};
        __builtin_nontemporal_store(t, reinterpret_cast<f4 *>(p));
    }
    __device__ __forceinline__ void fma(float w, const Vec &x) {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = __builtin_fmaf(w, x.v[i], v[i]);
    }
    __device__ __forceinline__ void add(const Vec &x) {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] += x.v[i];
    }
    __device__ __forceinline__ void scale(float a) {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] *= a;
    }
    __device__ __forceinline__ float dot(const Vec &x) const {
        float s = v[0] * x.v[0];
        s = __builtin_fmaf(v[1], x.v[1], s);
        s = __builtin_fmaf(v[2], x.v[2], s);
        s = __builtin_fmaf(v[3], x.v[3], s);
        return s;
    }
};

template <>
struct Vec<1> {
    float v[1];
    __device__ __forceinline__ void zero() { v[0] = 0.f; }
    __device__ __forceinline__ void ones() { v[0] = 1.f; }
    __device__ __forceinline__ void load(const float *p) { v[0] = *p; }
    __device__ __forceinline__ void store(float *p) const { *p = v[0]; }
    __device__ __forceinline__ void load_nt(const float *p) { v[0] = __builtin_nontemporal_load(p); }
    __device__ __forceinline__ void store_nt(float *p) const { __builtin_nontemporal_store(v[0], p); }
    __device__ __forceinline__ void fma(float w, const Vec &x) { v[0] = __builtin_fmaf(w, x.v[0], v[0]); }
    __device__ __forceinline__ void add(const Vec &x) { v[0] += x.v[0]; }
    __device__ __forceinline__ void scale(float a) { v[0] *= a; }
    __device__ __forceinline__ float dot(const Vec &x) const { return v[0] * x.v[0]; }
};

// ----------------------------------------------------- kernel launchers

// Dense width k -> (VEC, G): VEC fp32 per lane, G lanes per dense row chunk.
struct WidthPlan {
    int vec;   // 4 or 1
    int g;     // lanes per row chunk, power of two, <= 64
    int chunk; // columns covered by one chunk = vec * g
};

inline WidthPlan width_plan(int k, bool vec_ok) {
    WidthPlan p;
    if (k % 4 == 0 && vec_ok) {
        p.vec = 4;
        int lanes = k / 4;
        p.g = 1;
        while (p.g < lanes && p.g < 64) p.g <<= 1;
    } else {
        p.vec = 1;
        p.g = 1;
        while (p.g < k && p.g < 64) p.g <<= 1;
    }
    p.chunk = p.vec * p.g;
    return p;
}

// ------------------------------------------- shared internal operations

// Device-wide exclusive prefix sum of n int32 (in and out may alias).
// The total goes to *total_dev when it is not NULL.
size_t scan_ws_bytes(int64_t n);
nsd_status scan_exclusive(const int32_t *in, int32_t *out, int64_t n, int32_t *total_dev,
                          void *ws, hipStream_t st);
// Exclusive max-scan (identity INT32_MIN), same workspace as scan_exclusive.
nsd_status scan_exclusive_max(const int32_t *in, int32_t *out, int64_t n, void *ws,
                              hipStream_t st);

// Stable LSD radix sort of (key, payload) by key in [0, max_key); payload_in
// NULL means the identity 0..n-1.  Results land in key_out / payload_out.
// radix_sort_multi carries np (1 to 3) payloads, the first of which may be
// the identity; its workspace is sort_ws_bytes(n, max_key, np).
size_t sort_ws_bytes(int64_t n, int32_t max_key, int np = 1);
nsd_status radix_sort_pairs(int64_t n, int32_t max_key, const int32_t *key_in,
                            const int32_t *payload_in, int32_t *key_out, int32_t *payload_out,
                            void *ws, hipStream_t st);
nsd_status radix_sort_multi(int64_t n, int32_t max_key, const int32_t *key_in, int np,
                            const int32_t *const *payload_in, int32_t *key_out,
                            int32_t *const *payload_out, void *ws, hipStream_t st);

// segptr[r] = first position q with sorted_key[q] >= r, for r in [0, nseg].
nsd_status segptr_from_sorted(int64_t n, int32_t nseg, const int32_t *sorted_key,
                              int32_t *segptr, hipStream_t st);

}  // namespace nsd
