// Setup-phase kernels (Algorithm 3): per-row product counts (InterOffsets),
// CSR validation, and the masked CSR->CSC conversion of the heavy rows with
// its slice offsets (Section III-B).
#include "host.hpp"

namespace gm {

namespace {

constexpr int FLAT_BLOCK = 256;
constexpr int FLAT_ITEMS = 8;  // consecutive entries per thread

// InterOffsets for rows [r0, r1): every thread walks FLAT_ITEMS consecutive
// nonzeros of A, adding nnz(B[k,:]) to its current row and tracking the
// smallest first column and largest last column of the B rows it touches
// (the row's column span, used to pick a dense window for light rows).
// A row split across threads is merged with atomics. Without SPAN only the
// counts are taken (one B.rp pair per entry, no reads of B's columns).
// The rows of the work group's entries are found once (two searches of
// A.rp), their row pointers staged in LDS when they are few, and each thread
// issues all its loads of one kind together (entries, then B.rp pairs, then
// the first and last columns) instead of one dependent chain per entry.
constexpr int RP_ROWS = 1024;  // row pointers a work group stages in LDS

// Per-B-row summary (length, first and last column) in one 16-byte record
// (int32 columns), so that an A entry's B-row facts come from one random read
// instead of the row pointer pair plus two column reads; built when the
// panel has many more A entries than B has rows.
template <typename CI>
struct BRowInfo {
    int64_t len;
    CI first, last;
};

template <typename CI>
__global__ void k_brow_info(CsrV<CI, NoV> B, BRowInfo<CI> *info) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < B.n_rows;
         k += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b0 = B.rp[k], b1 = B.rp[k + 1];
        BRowInfo<CI> r;
        r.len = b1 - b0;
        r.first = b1 > b0 ? B.ci[b0] : (CI)0;
        r.last = b1 > b0 ? B.ci[b1 - 1] : (CI)0;
        info[k] = r;
    }
}

template <bool SPAN, bool INFO, typename CI>
__global__ __launch_bounds__(FLAT_BLOCK) void k_row_products(CsrV<CI, NoV> A, CsrV<CI, NoV> B,
                                                             const BRowInfo<CI> *binfo, int64_t r0, int64_t r1,
                                                             int64_t *ip, CI *minc, CI *maxc) {
    constexpr CI CI_MAX = sizeof(CI) == 8 ? (CI)INT64_MAX : (CI)INT32_MAX;
    __shared__ int64_t rp_s[RP_ROWS + 1];
    __shared__ int64_t rows[2];
    const int64_t e_begin = A.rp[r0], e_end = A.rp[r1];
    const int64_t blk0 = e_begin + blockIdx.x * (int64_t)FLAT_BLOCK * FLAT_ITEMS;
    const int64_t blk1 = blk0 + (int64_t)FLAT_BLOCK * FLAT_ITEMS < e_end ? blk0 + (int64_t)FLAT_BLOCK * FLAT_ITEMS : e_end;
    if (threadIdx.x == 0) rows[0] = find_row(A.rp, r0, r1 + 1, blk0);
    if (threadIdx.x == GM_WAVE) rows[1] = find_row(A.rp, r0, r1 + 1, blk1 - 1);
    __syncthreads();
    const int64_t ra = rows[0], rb = rows[1];  // rows of the group's first and last entry
    const int64_t nr = rb - ra + 1;
    const bool staged = nr <= RP_ROWS;
    if (staged)
        for (int64_t q = threadIdx.x; q <= nr; q += FLAT_BLOCK) rp_s[q] = A.rp[ra + q];
    __syncthreads();
    const int64_t e0 = blk0 + (int64_t)threadIdx.x * FLAT_ITEMS;
    if (e0 >= blk1) return;
    const int64_t e1 = e0 + FLAT_ITEMS < blk1 ? e0 + FLAT_ITEMS : blk1;
    const int ne = (int)(e1 - e0);
    int64_t kk[FLAT_ITEMS], b0[FLAT_ITEMS], b1[FLAT_ITEMS];
    CI f[FLAT_ITEMS], l[FLAT_ITEMS];
#pragma unroll
    for (int i = 0; i < FLAT_ITEMS; ++i) kk[i] = (int64_t)A.ci[i < ne ? e0 + i : e0];
    if (INFO) {
#pragma unroll
        for (int i = 0; i < FLAT_ITEMS; ++i) {
            const BRowInfo<CI> r = binfo[kk[i]];
            b0[i] = 0;
            b1[i] = r.len;
            f[i] = r.first;
            l[i] = r.last;
        }
    } else {
#pragma unroll
        for (int i = 0; i < FLAT_ITEMS; ++i) {
            b0[i] = B.rp[kk[i]];
            b1[i] = B.rp[kk[i] + 1];
        }
        if (SPAN) {
#pragma unroll
            for (int i = 0; i < FLAT_ITEMS; ++i) {
                const bool nonempty = b1[i] > b0[i];  // (an empty B may have no column array)
                f[i] = nonempty ? B.ci[b0[i]] : (CI)0;
                l[i] = nonempty ? B.ci[b1[i] - 1] : (CI)0;
            }
        }
    }
    int64_t row = staged ? ra + find_row(rp_s, 0, nr + 1, e0) : find_row(A.rp, ra, rb + 1, e0);
    int64_t row_end = staged ? rp_s[row - ra + 1] : A.rp[row + 1];
    int64_t acc = 0;
    CI lo = CI_MAX, hi = -1;
#pragma unroll
    for (int i = 0; i < FLAT_ITEMS; ++i) {
        if (i >= ne) break;
        while (e0 + i >= row_end) {  // flush and move to the next nonempty row
            if (acc) atomicAdd((unsigned long long *)&ip[row - r0], (unsigned long long)acc);
            if (SPAN && hi >= 0) {
                __hip_atomic_fetch_min(&minc[row - r0], lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_fetch_max(&maxc[row - r0], hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            acc = 0;
            lo = CI_MAX;
            hi = -1;
            ++row;
            row_end = staged ? rp_s[row - ra + 1] : A.rp[row + 1];
        }
        if (b1[i] > b0[i]) {
            acc += b1[i] - b0[i];
            if (SPAN) {
                lo = f[i] < lo ? f[i] : lo;
                hi = l[i] > hi ? l[i] : hi;
            }
        }
    }
    if (acc) atomicAdd((unsigned long long *)&ip[row - r0], (unsigned long long)acc);
    if (SPAN && hi >= 0) {
        __hip_atomic_fetch_min(&minc[row - r0], lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_max(&maxc[row - r0], hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <typename CI>
__global__ void k_validate_rows(CsrV<CI, NoV> M, int32_t *flag) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < M.n_rows;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t s = M.rp[i], e = M.rp[i + 1];
        if (i == 0 && s != 0) atomicOr(flag, 1);
        if (i == M.n_rows - 1 && e != M.nnz) atomicOr(flag, 2);
        if (e < s) {
            atomicOr(flag, 4);
            continue;
        }
        int64_t prev = -1;
        for (int64_t p = s; p < e && p < M.nnz; ++p) {
            const int64_t c = (int64_t)M.ci[p];
            if (c < 0 || c >= M.n_cols) atomicOr(flag, 8);
            if (c <= prev) atomicOr(flag, 16);
            prev = c;
        }
    }
}

// Visits the nonzeros of the heavy rows of A in the flattened order given
// by a_heavy_ptr (exclusive scan of the heavy rows' lengths); calls
// f(h, j) with the heavy index h and the position j in A.
template <class M, class F>
GM_DEV void for_heavy_entries(const M &A, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
                              const int64_t *a_heavy_ptr, int64_t total, F f) {
    const int64_t e0 = (blockIdx.x * (int64_t)FLAT_BLOCK + threadIdx.x) * FLAT_ITEMS;
    if (e0 >= total) return;
    const int64_t e1 = e0 + FLAT_ITEMS < total ? e0 + FLAT_ITEMS : total;
    int64_t h = find_row(a_heavy_ptr, 0, n_heavy + 1, e0);
    int64_t h_end = a_heavy_ptr[h + 1];
    int64_t a_base = A.rp[r0 + heavy_rows[h]] - a_heavy_ptr[h];
    for (int64_t e = e0; e < e1; ++e) {
        while (e >= h_end) {
            ++h;
            h_end = a_heavy_ptr[h + 1];
            a_base = A.rp[r0 + heavy_rows[h]] - a_heavy_ptr[h];
        }
        f(h, a_base + e, e);
    }
}

template <typename CI>
__global__ __launch_bounds__(FLAT_BLOCK) void k_csc_count(CsrV<CI, NoV> A, Csr B, const int64_t *heavy_rows,
                                                          int64_t n_heavy, int64_t r0, const int64_t *a_heavy_ptr,
                                                          int64_t total, int64_t *colcnt) {
    for_heavy_entries(A, heavy_rows, n_heavy, r0, a_heavy_ptr, total, [&](int64_t, int64_t j, int64_t) {
        const int64_t k = (int64_t)A.ci[j];
        if (B.rp[k + 1] > B.rp[k]) atomicAdd((unsigned long long *)&colcnt[k], 1ull);
    });
}

__global__ void k_slice_flags(Csr B, const int64_t *colcnt, int64_t n_k, uint8_t *cls) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n_k; k += (int64_t)gridDim.x * blockDim.x)
        cls[k] = (colcnt[k] > 0 && B.rp[k + 1] > B.rp[k]) ? 0 : 1;
}

__global__ void k_slice_build(Csr B, const int64_t *colcnt, const int64_t *perm, int64_t n_slices, int32_t *slice_k,
                              int64_t *cnt_out, int64_t *ip_out, int32_t *k_to_slice) {
    for (int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; s < n_slices;
         s += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = perm[s];
        slice_k[s] = (int32_t)k;
        cnt_out[s] = colcnt[k];
        ip_out[s] = colcnt[k] * (B.rp[k + 1] - B.rp[k]);
        k_to_slice[k] = (int32_t)s;
    }
}

template <typename CI, typename V>
__global__ __launch_bounds__(FLAT_BLOCK) void k_csc_fill(CsrV<CI, V> A, const int64_t *heavy_rows, int64_t n_heavy,
                                                         int64_t r0, const int64_t *a_heavy_ptr, int64_t total,
                                                         const int32_t *k_to_slice, const int64_t *col_ptr,
                                                         int64_t *fill_cursor, int32_t *row_h, V *a_val) {
    for_heavy_entries(A, heavy_rows, n_heavy, r0, a_heavy_ptr, total, [&](int64_t h, int64_t j, int64_t) {
        const int32_t s = k_to_slice[(int64_t)A.ci[j]];
        if (s < 0) return;
        const int64_t pos =
            col_ptr[s] + (int64_t)atomicAdd((unsigned long long *)&fill_cursor[s], 1ull);
        row_h[pos] = (int32_t)h;
        a_val[pos] = A.v[j];
    });
}

__global__ void k_slice_lengths(Csr B, const int32_t *slice_k, int64_t n, int64_t *len) {
    for (int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; s < n; s += (int64_t)gridDim.x * blockDim.x)
        len[s] = B.rp[slice_k[s] + 1] - B.rp[slice_k[s]];
}

// Level-0 chunk boundaries of every slice's B row: bnd[s * (nc + 1) + c] =
// offset in B[k,:] of the row's first column >= c << shift (c = 0..nc). The
// row is sorted, so lane c of a wave finds it by binary search; chunk c of
// the row is [bnd[c], bnd[c + 1]). A row of at most 64 elements (most of
// them) is loaded once, one element per lane, and searched across the lanes
// with shuffles instead of a chain of dependent global loads.
template <typename CI>
__global__ __launch_bounds__(256) void k_slice_chunk_bounds(CsrV<CI, NoV> B, const int32_t *slice_k, int64_t n_slices,
                                                            int nc, int shift, int32_t *bnd) {
    const int lane = threadIdx.x & (GM_WAVE - 1);
    const int64_t nwaves = (int64_t)gridDim.x * (blockDim.x / GM_WAVE);
    for (int64_t s = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / GM_WAVE; s < n_slices; s += nwaves) {
        const int32_t k = slice_k[s];
        const int64_t b0 = B.rp[k], b1 = B.rp[k + 1];
        if (b1 - b0 <= GM_WAVE) {  // uniform over the wave
            const int len = (int)(b1 - b0);
            // chunk of each element (lanes past the row: past every chunk)
            const int ch = lane < len ? (int)((int64_t)B.ci[b0 + lane] >> shift) : INT32_MAX;
            int lo = 0, hi = len;  // lane c: first element whose chunk is >= c
#pragma unroll
            for (int st = 0; st < 7; ++st) {  // 2^7 > 64: every search closes
                const int mid = (lo + hi) >> 1;
                const int v = __shfl(ch, mid < GM_WAVE ? mid : GM_WAVE - 1, GM_WAVE);
                if (lo < hi) {
                    if (v < lane)
                        lo = mid + 1;
                    else
                        hi = mid;
                }
            }
            if (lane <= nc) bnd[s * (nc + 1) + lane] = lo;
            continue;
        }
        int64_t lo = b0, hi = b1;
        if (lane <= nc) {
            const int64_t bound = (int64_t)lane << shift;
            while (lo < hi) {
                const int64_t mid = lo + ((hi - lo) >> 1);
                if ((int64_t)B.ci[mid] < bound)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            bnd[s * (nc + 1) + lane] = (int32_t)(lo - b0);
        }
    }
}

// Level-0 histogram from the structure (Algorithm 3, Histogram at the first
// level): the C-hat row of heavy row h is the union of the B rows of its
// A~ entries, so counts[h * nc + c] = sum over those entries of the slices'
// chunk sizes (differences of the boundaries above). Each wave walks
// SH_ENTRIES consecutive A~ entries in row-major order, lane c accumulating
// chunk c, and flushes at row ends.
constexpr int SH_ENTRIES = 256, SH_U = 8;

template <typename CI>
__global__ __launch_bounds__(256) void k_struct_hist(CsrV<CI, NoV> A, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
                                                     const int64_t *a_heavy_ptr, int64_t total,
                                                     const int32_t *k_to_slice, const int32_t *bnd, int nc,
                                                     int64_t cmajor_rows, int64_t *counts) {
    const int lane = threadIdx.x & (GM_WAVE - 1);
    const int64_t wid = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / GM_WAVE;
    const int64_t e0 = wid * SH_ENTRIES;
    if (e0 >= total) return;  // uniform across the wave
    const int64_t e1 = e0 + SH_ENTRIES < total ? e0 + SH_ENTRIES : total;
    int64_t cur = find_row(a_heavy_ptr, 0, n_heavy + 1, e0);  // row of the wave's first entry
    int64_t acc = 0;
    int64_t h = cur, h_end = a_heavy_ptr[h + 1];
    int64_t a_base = A.rp[r0 + heavy_rows[h]] - a_heavy_ptr[h];
    for (int64_t eb = e0; eb < e1; eb += GM_WAVE) {
        // lane l resolves entry eb + l: its heavy row and slice
        const int64_t e = eb + lane;
        int32_t s = -1;
        if (e < e1) {
            while (e >= h_end) {
                ++h;
                h_end = a_heavy_ptr[h + 1];
                a_base = A.rp[r0 + heavy_rows[h]] - a_heavy_ptr[h];
            }
            s = k_to_slice[(int64_t)A.ci[a_base + e]];
        }
        const int cnt = (int)(e1 - eb < GM_WAVE ? e1 - eb : GM_WAVE);
        for (int q0 = 0; q0 < cnt; q0 += SH_U) {
            // the chunk bounds of SH_U entries, loaded with no branch between
            // the loads so that they are in flight together (a slot with
            // nothing to read loads bnd[0] and is dropped)
            int32_t lo[SH_U], hi[SH_U];
            int64_t hq[SH_U];
            bool ok[SH_U];
#pragma unroll
            for (int u = 0; u < SH_U; ++u) {
                const int q = q0 + u < cnt ? q0 + u : cnt - 1;
                hq[u] = __shfl(h, q, GM_WAVE);
                const int32_t sq = __shfl(s, q, GM_WAVE);
                ok[u] = q0 + u < cnt && sq >= 0 && lane < nc;
                const int32_t *bq = bnd + (int64_t)(sq >= 0 ? sq : 0) * (nc + 1);
                lo[u] = *(ok[u] ? bq + lane : bnd);
                hi[u] = *(ok[u] ? bq + lane + 1 : bnd);
            }
#pragma unroll
            for (int u = 0; u < SH_U; ++u) {
                if (q0 + u >= cnt) break;  // uniform
                if (hq[u] != cur) {
                    if (lane < nc && acc) {
                        const int64_t ix = cmajor_rows ? lane * cmajor_rows + cur : cur * nc + lane;
                        atomicAdd((unsigned long long *)&counts[ix], (unsigned long long)acc);
                    }
                    acc = 0;
                    cur = hq[u];
                }
                if (ok[u]) acc += hi[u] - lo[u];
            }
        }
        // lanes past the last entry may have stopped walking; realign for the next group
        h = __shfl(h, cnt - 1, GM_WAVE);
        h_end = a_heavy_ptr[h + 1];
        a_base = A.rp[r0 + heavy_rows[h]] - a_heavy_ptr[h];
    }
    if (lane < nc && acc) {
        const int64_t ix = cmajor_rows ? lane * cmajor_rows + cur : cur * nc + lane;
        atomicAdd((unsigned long long *)&counts[ix], (unsigned long long)acc);
    }
}

__global__ void k_gather_row_len(const int64_t *row_ptr, const int64_t *rows, int64_t n, int64_t r0, int64_t *out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = r0 + rows[i];
        out[i] = row_ptr[r + 1] - row_ptr[r];
    }
}

__global__ void k_gather_i64(const int64_t *src, const int64_t *idx, int64_t n, int64_t *out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        out[i] = src[idx[i]];
}

unsigned flat_grid(int64_t total) {
    const int64_t per = (int64_t)FLAT_BLOCK * FLAT_ITEMS;
    int64_t g = (total + per - 1) / per;
    return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

int64_t brow_info_bytes(const Csr &B) { return B.n_rows * (B.ci64 ? 24 : 16); }

void row_products(const Csr &A, const Csr &B, int64_t r0, int64_t r1, int64_t panel_nnz, int64_t *ip, void *minc,
                  void *maxc, hipStream_t s, void *binfo) {
    const int64_t n = r1 - r0;
    if (n <= 0) return;
    fill<int64_t>(ip, 0, n, s);
    with_index_type(B.ci64, [&](auto ci) {
        using CI = decltype(ci);
        CI *mn = static_cast<CI *>(minc), *mx = static_cast<CI *>(maxc);
        if (mn) {
            fill<CI>(mn, sizeof(CI) == 8 ? (CI)INT64_MAX : (CI)INT32_MAX, n, s);
            fill<CI>(mx, (CI)-1, n, s);
        }
        if (panel_nnz <= 0) return;
        BRowInfo<CI> *bi = static_cast<BRowInfo<CI> *>(binfo);
        if (mn && bi) {
            hipLaunchKernelGGL(k_brow_info<CI>, dim3(grid_for(B.n_rows, 256, 65536)), dim3(256), 0, s,
                               typed<CI, NoV>(B), bi);
            GM_CHECK_LAUNCH();
            hipLaunchKernelGGL((k_row_products<true, true, CI>), dim3(flat_grid(panel_nnz)), dim3(FLAT_BLOCK), 0, s,
                               typed<CI, NoV>(A), typed<CI, NoV>(B), bi, r0, r1, ip, mn, mx);
        } else if (mn) {
            hipLaunchKernelGGL((k_row_products<true, false, CI>), dim3(flat_grid(panel_nnz)), dim3(FLAT_BLOCK), 0, s,
                               typed<CI, NoV>(A), typed<CI, NoV>(B), bi, r0, r1, ip, mn, mx);
        } else {
            hipLaunchKernelGGL((k_row_products<false, false, CI>), dim3(flat_grid(panel_nnz)), dim3(FLAT_BLOCK), 0, s,
                               typed<CI, NoV>(A), typed<CI, NoV>(B), bi, r0, r1, ip, mn, mx);
        }
        GM_CHECK_LAUNCH();
    });
}

void validate_csr(const Csr &M, int32_t *flag, hipStream_t s) {
    fill<int32_t>(flag, 0, 1, s);
    if (M.n_rows <= 0) return;
    with_index_type(M.ci64, [&](auto ci) {
        using CI = decltype(ci);
        hipLaunchKernelGGL(k_validate_rows<CI>, dim3(grid_for(M.n_rows, 256, 8192)), dim3(256), 0, s,
                           typed<CI, NoV>(M), flag);
        GM_CHECK_LAUNCH();
    });
}

void csc_count(const Csr &A, const Csr &B, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
               const int64_t *a_heavy_ptr, int64_t nnz_heavy_all, int64_t *colcnt, hipStream_t s) {
    fill<int64_t>(colcnt, 0, A.n_cols, s);
    if (n_heavy <= 0 || nnz_heavy_all <= 0) return;
    with_index_type(A.ci64, [&](auto ci) {
        using CI = decltype(ci);
        hipLaunchKernelGGL(k_csc_count<CI>, dim3(flat_grid(nnz_heavy_all)), dim3(FLAT_BLOCK), 0, s, typed<CI, NoV>(A),
                           B, heavy_rows, n_heavy, r0, a_heavy_ptr, nnz_heavy_all, colcnt);
        GM_CHECK_LAUNCH();
    });
}

void slice_flags(const Csr &B, const int64_t *colcnt, int64_t n_k, uint8_t *cls, hipStream_t s) {
    if (n_k <= 0) return;
    hipLaunchKernelGGL(k_slice_flags, dim3(grid_for(n_k, 256, 16384)), dim3(256), 0, s, B, colcnt, n_k, cls);
    GM_CHECK_LAUNCH();
}

void slice_build(const Csr &B, const int64_t *colcnt, const int64_t *slice_perm, int64_t n_slices, int32_t *slice_k,
                 int64_t *cnt_out, int64_t *ip_out, int32_t *k_to_slice, hipStream_t s) {
    fill<int32_t>(k_to_slice, -1, B.n_rows, s);
    if (n_slices <= 0) return;
    hipLaunchKernelGGL(k_slice_build, dim3(grid_for(n_slices, 256, 16384)), dim3(256), 0, s, B, colcnt, slice_perm,
                       n_slices, slice_k, cnt_out, ip_out, k_to_slice);
    GM_CHECK_LAUNCH();
}

void csc_fill(const Csr &A, const Csr &B, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
              const int64_t *a_heavy_ptr, int64_t nnz_heavy_all, const int32_t *k_to_slice,
              const int64_t *col_ptr, int64_t *fill_cursor, int32_t *row_h, void *a_val, hipStream_t s) {
    (void)B;
    if (n_heavy <= 0 || nnz_heavy_all <= 0) return;
    with_types(A, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        hipLaunchKernelGGL((k_csc_fill<CI, V>), dim3(flat_grid(nnz_heavy_all)), dim3(FLAT_BLOCK), 0, s,
                           typed<CI, V>(A), heavy_rows, n_heavy, r0, a_heavy_ptr, nnz_heavy_all, k_to_slice, col_ptr,
                           fill_cursor, row_h, static_cast<V *>(a_val));
        GM_CHECK_LAUNCH();
    });
}

void slice_lengths(const Csr &B, const int32_t *slice_k, int64_t n, int64_t *len, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_slice_lengths, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, B, slice_k, n, len);
    GM_CHECK_LAUNCH();
}

void slice_chunk_bounds(const Csr &B, const SliceArrays &sl, int nc, int shift, int32_t *bnd, hipStream_t s) {
    if (sl.n_slices <= 0) return;
    GM_REQUIRE(nc >= 1 && nc < GM_WAVE, GMAGNUS_ERROR_UNSUPPORTED, "level-0 chunk count must be below 64");
    with_index_type(B.ci64, [&](auto ci) {
        using CI = decltype(ci);
        hipLaunchKernelGGL(k_slice_chunk_bounds<CI>, dim3(grid_for(sl.n_slices, 4, 65536)), dim3(256), 0, s,
                           typed<CI, NoV>(B), sl.slice_k, sl.n_slices, nc, shift, bnd);
        GM_CHECK_LAUNCH();
    });
}

void struct_hist(const Csr &A, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0, const int64_t *a_heavy_ptr,
                 int64_t nnz_heavy_all, const int32_t *k_to_slice, const int32_t *bnd, int nc, bool cmajor,
                 int64_t *counts, hipStream_t s) {
    fill<int64_t>(counts, 0, n_heavy * nc, s);
    if (n_heavy <= 0 || nnz_heavy_all <= 0) return;
    const int64_t waves = (nnz_heavy_all + SH_ENTRIES - 1) / SH_ENTRIES;
    with_index_type(A.ci64, [&](auto ci) {
        using CI = decltype(ci);
        hipLaunchKernelGGL(k_struct_hist<CI>, dim3(grid_for(waves, 4, (int64_t)1 << 30)), dim3(256), 0, s,
                           typed<CI, NoV>(A), heavy_rows, n_heavy, r0, a_heavy_ptr, nnz_heavy_all, k_to_slice, bnd, nc,
                           cmajor ? n_heavy : (int64_t)0, counts);
        GM_CHECK_LAUNCH();
    });
}

void gather_row_len(const int64_t *row_ptr, const int64_t *rows, int64_t n, int64_t r0, int64_t *out,
                    hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_gather_row_len, dim3(grid_for(n, 256, 16384)), dim3(256), 0, s, row_ptr, rows, n, r0, out);
    GM_CHECK_LAUNCH();
}

void gather_i64(const int64_t *src, const int64_t *idx, int64_t n, int64_t *out, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_gather_i64, dim3(grid_for(n, 256, 16384)), dim3(256), 0, s, src, idx, n, out);
    GM_CHECK_LAUNCH();
}

}  // namespace gm
