// Shared device helpers for the gfx950 SpGEMM kernels: wave64 scans and
// ballots, block scans, bounded binary searches and small launch utilities.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define GM_DEV __device__ __forceinline__
#define GM_WAVE 64

namespace gm {

// Read-only view of a device CSR matrix with its column-index and value
// types chosen at run time (int32 / int64 columns, fp64 / fp32 values).
struct Csr {
    int64_t n_rows, n_cols, nnz;
    const int64_t *rp;
    const void *ci;
    const void *v;
    bool ci64 = false;  // column indices are int64
    bool v32 = false;   // values are fp32
};

// The same view with its types fixed, as kernels take it.
template <typename CI, typename V>
struct CsrV {
    int64_t n_rows, n_cols, nnz;
    const int64_t *rp;
    const CI *ci;
    const V *v;
};

template <typename CI, typename V>
inline CsrV<CI, V> typed(const Csr &m) {
    return CsrV<CI, V>{m.n_rows, m.n_cols, m.nnz, m.rp, static_cast<const CI *>(m.ci), static_cast<const V *>(m.v)};
}

// Value type of views whose kernels never read values.
using NoV = unsigned char;

// Calls f(CI{}, V{}) with the column-index and value types of a view.
template <class F>
inline void with_types(bool ci64, bool v32, F &&f) {
    if (ci64) {
        if (v32)
            f(int64_t{}, float{});
        else
            f(int64_t{}, double{});
    } else {
        if (v32)
            f(int32_t{}, float{});
        else
            f(int32_t{}, double{});
    }
}
template <class F>
inline void with_types(const Csr &m, F &&f) {
    with_types(m.ci64, m.v32, static_cast<F &&>(f));
}
// Calls f(CI{}) with the column-index type.
template <class F>
inline void with_index_type(bool ci64, F &&f) {
    if (ci64)
        f(int64_t{});
    else
        f(int32_t{});
}
// Calls f(V{}) with the value type.
template <class F>
inline void with_value_type(bool v32, F &&f) {
    if (v32)
        f(float{});
    else
        f(double{});
}

GM_DEV int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0)); }

GM_DEV uint64_t lanemask_lt() { return (uint64_t(1) << lane_id()) - 1; }

GM_DEV uint64_t ballot(bool p) { return __ballot(p); }

GM_DEV int ilog2_dev(int x) { return 31 - __clz(x); }

// Orders this lane's earlier LDS accesses before its later ones as seen by
// the other lanes of the wave (lanes of a wave run in lockstep).
GM_DEV void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

template <typename T>
GM_DEV T wave_incl_scan(T x) {
    const int lane = threadIdx.x & (GM_WAVE - 1);
#pragma unroll
    for (int d = 1; d < GM_WAVE; d <<= 1) {
        T y = __shfl_up(x, d, GM_WAVE);
        if (lane >= d) x += y;
    }
    return x;
}

// 32-bit values: the same scan with DPP moves (VALU only, no LDS permute).
// row_shr:1,2,4,8 scan each row of 16 lanes (lanes whose source lies before
// the row read 0); row_bcast:15 then adds lane 15's sum to row 1 and lane 47's
// to row 3, and row_bcast:31 adds lane 31's sum to rows 2 and 3.
template <>
GM_DEV int32_t wave_incl_scan<int32_t>(int32_t x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15, rows 1 and 3
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31, rows 2 and 3
    return x;
}

// Value held by the previous lane of the wave (lane 0 gets `first`): one DPP
// move with wave_shr:1.
GM_DEV int32_t prev_lane(int32_t x, int32_t first) { return __builtin_amdgcn_update_dpp(first, x, 0x138, 0xf, 0xf, false); }

template <typename T>
GM_DEV T wave_reduce_sum(T x) {
#pragma unroll
    for (int d = GM_WAVE / 2; d >= 1; d >>= 1) x += __shfl_xor(x, d, GM_WAVE);
    return x;
}

// 32-bit values: the DPP scan's last lane holds the sum.
template <>
GM_DEV int32_t wave_reduce_sum<int32_t>(int32_t x) {
    return __builtin_amdgcn_readlane(wave_incl_scan<int32_t>(x), GM_WAVE - 1);
}

// Exclusive scan over the block in thread order. `smem` holds BLOCK/64
// entries; the block total is returned through *total when not null.
// Contains __syncthreads: every thread of the block must call it.
template <int BLOCK, typename T>
GM_DEV T block_excl_scan(T x, T *smem, T *total = nullptr) {
    constexpr int NW = BLOCK / GM_WAVE;
    const int lane = threadIdx.x & (GM_WAVE - 1), w = threadIdx.x / GM_WAVE;
    T inc = wave_incl_scan(x);
    if (lane == GM_WAVE - 1) smem[w] = inc;
    __syncthreads();
    if (w == 0) {
        T s = lane < NW ? smem[lane] : T(0);
        s = wave_incl_scan(s);
        if (lane < NW) smem[lane] = s;
    }
    __syncthreads();
    T off = w > 0 ? smem[w - 1] : T(0);
    if (total) *total = smem[NW - 1];
    __syncthreads();
    return off + inc - x;
}

template <int BLOCK, typename T>
GM_DEV T block_reduce_sum(T x, T *smem) {
    T t;
    block_excl_scan<BLOCK, T>(x, smem, &t);
    return t;
}

// Largest index i in [lo, hi) with a[i] <= key, assuming a[lo] <= key and a
// non-decreasing (the row containing flattened position `key`, skipping
// empty rows to the last one that starts at or before key).
template <typename T, typename K>
GM_DEV int64_t find_row(const T *a, int64_t lo, int64_t hi, K key) {
    while (hi - lo > 1) {
        int64_t mid = lo + ((hi - lo) >> 1);
        if (a[mid] <= (T)key)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// XCD-aware remap of a linear block id: the hardware deals consecutive
// workgroups round-robin to the 8 XCDs; this gives each XCD a contiguous run
// of tiles so neighbouring tiles share that XCD's L2.
GM_DEV int64_t xcd_tile(int64_t bid, int64_t nblocks) {
    constexpr int64_t NX = 8;
    const int64_t per = nblocks / NX, rem = nblocks % NX;
    const int64_t x = bid % NX, q = bid / NX;
    // XCD x owns tiles [x*per + min(x, rem), ...) of length per + (x < rem)
    const int64_t base = x * per + (x < rem ? x : rem);
    const int64_t len = per + (x < rem ? 1 : 0);
    return q < len ? base + q : bid;  // q < len always holds for a full grid
}

template <typename T>
__global__ void k_fill(T *p, T v, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

template <typename T>
__global__ void k_iota(T *p, T start, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = start + (T)i;
}

inline unsigned grid_for(int64_t n, int block, int64_t cap = 1 << 20) {
    int64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (unsigned)g;
}

inline int ilog2(int64_t x) {
    int r = 0;
    while ((int64_t(1) << (r + 1)) <= x) ++r;
    return r;
}
inline int64_t floor_pow2(int64_t x) { return x < 1 ? 0 : int64_t(1) << ilog2(x); }
inline int64_t ceil_pow2(int64_t x) {
    int64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

}  // namespace gm
