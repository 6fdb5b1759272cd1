// Accumulation (Section III-E): symbolic (distinct-column counts) and
// numeric (sorted rows of C) for
//   * light rows of C -- Gustavson (Section II-B, Algorithm 1) with an LDS
//     hash map (modulo hashing, linear probing, load factor <= 1/2) or, when
//     the row's column span is small, an LDS dense window;
//   * final chunks of the heavy rows ("leaves" of the multisplit) -- the
//     chunk's (column, value) pairs are accumulated with the hash map when the
//     chunk is light and with an LDS dense accumulator plus bitmap when it is
//     heavy (its column range is at most W wide, Section III-D).
// Hash output is sorted with an LDS bitonic sort; dense output comes out in
// column order from a wave64 ballot over the bitmap. Columns of chunks are
// shifted back by the chunk's column base on the final write.
//
// Work is binned by size (OpSparse-style, Section III-E): one work group per
// row or chunk, with the work-group size and LDS table chosen per bin.
#include "host.hpp"

namespace gm {

namespace {

// Column of element t of a leaf set: chunk-local, stored in 32 bits, or in
// 16 bits for the final chunks the fused expansion writes (a wave-uniform
// branch on a kernel argument).
GM_DEV int32_t leaf_col(const LeafSet &L, int64_t t) { return L.col16 ? (int32_t)L.col16[t] : L.col[t]; }
GM_DEV int32_t leaf_col_nt(const LeafSet &L, int64_t t) {
    return L.col16 ? (int32_t)__builtin_nontemporal_load(&L.col16[t]) : __builtin_nontemporal_load(&L.col[t]);
}

// --------------------------------------------------------------- sources
template <int BLOCK, typename V>
struct GusLds {
    int32_t off[BLOCK];  // product offsets of the batch's entries; INT32_MAX past the last one
    int64_t bst[BLOCK];
    V av[BLOCK];
    int32_t scan[BLOCK / GM_WAVE];
};

constexpr int GUS_ILP = 4;

// Entry of product t in a batch: the largest q < BLOCK with off[q] <= t
// (off[0] = 0, off non-decreasing, INT32_MAX past the batch's entries), by a
// branch-free power-of-two search (every step one LDS read, no loop exit to
// wait for, so the searches of several products overlap).
template <int BLOCK>
GM_DEV int entry_of(const int32_t *off, int32_t t) {
    int q = 0;
#pragma unroll
    for (int step = BLOCK / 2; step >= 1; step >>= 1) q = off[q + step] <= t ? q + step : q;
    return q;
}

// Calls f(col - base, product) for every intermediate product of the A
// entries [j0, j1) (one row of A), A entries taken in batches of BLOCK.
// (base: 0, or the row's smallest column when columns are 64-bit; the row's
// columns then span less than 2^31, so the offsets fit 32 bits)
template <int BLOCK, bool NUM, typename CI, typename V, class F>
GM_DEV void gustavson_row(const CsrV<CI, V> &A, const CsrV<CI, V> &B, int64_t j0, int64_t j1, CI base,
                          GusLds<BLOCK, V> &L, F &&f) {
    const int tid = threadIdx.x;
    for (int64_t jb = j0; jb < j1; jb += BLOCK) {
        const int nb = (int)(j1 - jb < BLOCK ? j1 - jb : BLOCK);
        int32_t len = 0;
        if (tid < nb) {
            const int64_t k = (int64_t)A.ci[jb + tid];
            const int64_t bs = B.rp[k];
            len = (int32_t)(B.rp[k + 1] - bs);
            L.bst[tid] = bs;
            if (NUM) L.av[tid] = A.v[jb + tid];
        }
        int32_t tot;
        const int32_t ex = block_excl_scan<BLOCK>(len, L.scan, &tot);
        L.off[tid] = tid < nb ? ex : INT32_MAX;
        __syncthreads();
        // GUS_ILP products per thread: the searches, then every load, then the
        // accumulation, with no branch between the loads (past the end a thread
        // re-reads the batch's last product and drops it), so one thread's loads
        // are in flight together
        for (int32_t tb = tid; tb < tot; tb += BLOCK * GUS_ILP) {
            int32_t q[GUS_ILP];
            int64_t src[GUS_ILP];
#pragma unroll
            for (int u = 0; u < GUS_ILP; ++u) {
                const int32_t t = tb + u * BLOCK < tot ? tb + u * BLOCK : tot - 1;
                q[u] = entry_of<BLOCK>(L.off, t);
                src[u] = L.bst[q[u]] + (t - L.off[q[u]]);
            }
            CI c[GUS_ILP];
            V v[GUS_ILP];
#pragma unroll
            for (int u = 0; u < GUS_ILP; ++u) {
                c[u] = B.ci[src[u]];
                if (NUM) v[u] = B.v[src[u]];
            }
#pragma unroll
            for (int u = 0; u < GUS_ILP; ++u)
                if (tb + u * BLOCK < tot) f((int32_t)(c[u] - base), NUM ? (V)(L.av[q[u]] * v[u]) : (V)0);
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------ hash map
// Multiplicative (Fibonacci) hashing into a power-of-two table. The paper's
// plain modulo keeps the column's low bits, which R-MAT skews heavily (each
// bit is 0 with probability a + c), so linear probing would cluster.
template <int TS>
GM_DEV uint32_t hash_slot(int32_t c) {
    static_assert((TS & (TS - 1)) == 0 && TS >= 2, "table size must be a power of two");
    return ((uint32_t)c * 0x9E3779B1u) >> (32 - __builtin_ctz(TS));
}

// Probing stops after TS slots, so a table that were ever full could not
// hang the work group (the count check of the numeric phase reports it).
template <int TS>
GM_DEV void hash_insert_key(int32_t *keys, int32_t c, int32_t *counter) {
    uint32_t h = hash_slot<TS>(c);
    for (int probe = 0; probe < TS; ++probe) {
        int32_t old = ((volatile int32_t *)keys)[h];
        if (old == -1) {
            old = atomicCAS(&keys[h], -1, c);
            if (old == -1) {
                atomicAdd(counter, 1);
                return;
            }
        }
        if (old == c) return;
        h = (h + 1) & (TS - 1);
    }
}

template <int TS, typename V>
GM_DEV void hash_insert_add(int32_t *keys, V *vals, int32_t c, V v) {
    uint32_t h = hash_slot<TS>(c);
    for (int probe = 0; probe < TS; ++probe) {
        int32_t old = ((volatile int32_t *)keys)[h];
        if (old == -1) {
            old = atomicCAS(&keys[h], -1, c);
            if (old == -1) old = c;
        }
        if (old == c) {
            __hip_atomic_fetch_add(&vals[h], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            return;
        }
        h = (h + 1) & (TS - 1);
    }
}

template <int BLOCK, int TS, typename V = double>
GM_DEV void hash_clear(int32_t *keys, V *vals) {
    for (int i = threadIdx.x; i < TS; i += BLOCK) {
        keys[i] = -1;
        if (vals) vals[i] = (V)0;
    }
}

// Compacts the occupied slots to the front, sorts them by column (bitonic)
// and writes at most `nnz` entries (the symbolic count) with the column base
// added. Returns nothing; a count mismatch is flagged in *err.
template <int BLOCK, int TS, typename V, typename CI>
GM_DEV void hash_emit_sorted(int32_t *keys, V *vals, int64_t nnz, CI col_base, CI *out_col, V *out_val,
                             int32_t *scan_sm, int32_t *err) {
    constexpr int PER = TS / BLOCK;
    static_assert(PER * BLOCK == TS, "table size must be a multiple of the block");
    const int tid = threadIdx.x;
    int32_t k[PER];
    V v[PER];
    int cnt = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
        k[q] = keys[tid + q * BLOCK];  // strided: no LDS bank conflicts
        v[q] = vals[tid + q * BLOCK];
        cnt += k[q] != -1;
    }
    int32_t total;
    int pos = block_excl_scan<BLOCK>(cnt, scan_sm, &total);
#pragma unroll
    for (int q = 0; q < PER; ++q)
        if (k[q] != -1) {
            keys[pos] = k[q];
            vals[pos] = v[q];
            ++pos;
        }
    int P = 1;
    while (P < total) P <<= 1;
    for (int i = total + tid; i < P; i += BLOCK) keys[i] = INT32_MAX;
    __syncthreads();
    for (int kk = 2; kk <= P; kk <<= 1)
        for (int j = kk >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < P; i += BLOCK) {
                const int ixj = i ^ j;
                if (ixj > i) {
                    const int32_t a = keys[i], b = keys[ixj];
                    const bool up = (i & kk) == 0;
                    if ((a > b) == up) {
                        keys[i] = b;
                        keys[ixj] = a;
                        const V t = vals[i];
                        vals[i] = vals[ixj];
                        vals[ixj] = t;
                    }
                }
            }
            __syncthreads();
        }
    if (tid == 0 && total != nnz) atomicOr(err, 1);
    const int n_out = (int64_t)total < nnz ? total : (int)nnz;
    for (int i = tid; i < n_out; i += BLOCK) {
        out_col[i] = (CI)keys[i] + col_base;
        out_val[i] = vals[i];
    }
}

// ------------------------------------------------------ dense accumulator
// VALS = false keeps only the bitmap (symbolic passes), so more work groups
// fit a CU.
template <int BLOCK, int WMAX, bool VALS, typename V = double>
struct DenseLdsT {
    V vals[VALS ? WMAX : 1];
    uint32_t bits[(WMAX + 31) / 32];
    int32_t scan[BLOCK / GM_WAVE];
};
template <int BLOCK, int WMAX, typename V>
using DenseLds = DenseLdsT<BLOCK, WMAX, true, V>;
template <int BLOCK, int WMAX>
using DenseBits = DenseLdsT<BLOCK, WMAX, false>;

template <int BLOCK, int WMAX, bool VALS, typename V>
GM_DEV void dense_clear(DenseLdsT<BLOCK, WMAX, VALS, V> &L, int width, bool num) {
    for (int i = threadIdx.x; i < (width + 31) / 32; i += BLOCK) L.bits[i] = 0;
    if (VALS && num)
        for (int i = threadIdx.x; i < width; i += BLOCK) L.vals[i] = (V)0;
}

template <int BLOCK, int WMAX, bool VALS, typename V>
GM_DEV void dense_set(DenseLdsT<BLOCK, WMAX, VALS, V> &L, int c) {
    const uint32_t bit = 1u << (c & 31);
    if (!(((volatile uint32_t *)L.bits)[c >> 5] & bit)) atomicOr(&L.bits[c >> 5], bit);
}

template <int BLOCK, int WMAX, typename V>
GM_DEV void dense_add(DenseLds<BLOCK, WMAX, V> &L, int c, V v) {
    dense_set(L, c);
    __hip_atomic_fetch_add(&L.vals[c], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int BLOCK, int WMAX, bool VALS, typename V>
GM_DEV int32_t dense_count(DenseLdsT<BLOCK, WMAX, VALS, V> &L, int width) {
    int32_t c = 0;
    for (int i = threadIdx.x; i < (width + 31) / 32; i += BLOCK) c += __popc(L.bits[i]);
    return block_reduce_sum<BLOCK>(c, L.scan);
}

// Writes the present columns in increasing order: wave w owns a contiguous
// range of columns and walks it 64 columns at a time, one per lane.
template <int BLOCK, int WMAX, typename V, typename CI>
GM_DEV void dense_emit(DenseLds<BLOCK, WMAX, V> &L, int width, int64_t nnz, CI col_base, CI *out_col, V *out_val,
                       int32_t *err) {
    constexpr int NW = BLOCK / GM_WAVE;
    const int lane = threadIdx.x & (GM_WAVE - 1), w = threadIdx.x / GM_WAVE;
    const int span = ((width + NW - 1) / NW + GM_WAVE - 1) / GM_WAVE * GM_WAVE;
    const int c0 = w * span, c1 = c0 + span < width ? c0 + span : width;
    int32_t cnt = 0;
    for (int c = c0 + lane; c < c1; c += GM_WAVE) cnt += (L.bits[c >> 5] >> (c & 31)) & 1;
    cnt = wave_reduce_sum(cnt);
    int32_t total;
    int32_t base = block_excl_scan<BLOCK>(lane == 0 ? cnt : 0, L.scan, &total);
    base = __shfl(base, 0, GM_WAVE);
    if (threadIdx.x == 0 && total != nnz) atomicOr(err, 2);
    for (int g = c0; g < c1; g += GM_WAVE) {
        const int c = g + lane;
        const bool p = c < c1 && ((L.bits[c >> 5] >> (c & 31)) & 1);
        const uint64_t m = ballot(p);
        const int pos = base + __popcll(m & lanemask_lt());
        if (p && pos < nnz) {
            out_col[pos] = (CI)c + col_base;
            out_val[pos] = L.vals[c];
        }
        base += __popcll(m);
    }
}

// dense_emit that also leaves the accumulator zeroed (values of the present
// columns and this wave's bitmap words), so the next chunk needs no clear.
template <int BLOCK, int WMAX, typename V, typename CI>
GM_DEV void dense_emit_clear(DenseLds<BLOCK, WMAX, V> &L, int width, int64_t nnz, CI col_base, CI *out_col,
                             V *out_val, int32_t *err) {
    constexpr int NW = BLOCK / GM_WAVE;
    const int lane = threadIdx.x & (GM_WAVE - 1), w = threadIdx.x / GM_WAVE;
    const int span = ((width + NW - 1) / NW + GM_WAVE - 1) / GM_WAVE * GM_WAVE;  // multiple of 64 columns
    const int c0 = w * span, c1 = c0 + span < width ? c0 + span : width;
    int32_t cnt = 0;
    for (int c = c0 + lane; c < c1; c += GM_WAVE) cnt += (L.bits[c >> 5] >> (c & 31)) & 1;
    cnt = wave_reduce_sum(cnt);
    int32_t total;
    int32_t base = block_excl_scan<BLOCK>(lane == 0 ? cnt : 0, L.scan, &total);
    base = __shfl(base, 0, GM_WAVE);
    if (threadIdx.x == 0 && total != nnz) atomicOr(err, 2);
    for (int g = c0; g < c1; g += GM_WAVE) {
        const int c = g + lane;
        const bool p = c < c1 && ((L.bits[c >> 5] >> (c & 31)) & 1);
        const uint64_t m = ballot(p);
        const int pos = base + __popcll(m & lanemask_lt());
        if (p) {
            if (pos < nnz) {
                out_col[pos] = (CI)c + col_base;
                out_val[pos] = L.vals[c];
            }
            L.vals[c] = (V)0;
        }
        base += __popcll(m);
    }
    for (int wd = (c0 >> 5) + lane; wd < ((c1 + 31) >> 5); wd += GM_WAVE) L.bits[wd] = 0;
}

// ----------------------------------------------------------- bin tables
// Hash bins: (max elements or nnz, table slots, block).
constexpr int HS_CAP[4] = {128, 512, 2048, 8192};   // symbolic: elements (load <= 1/2)
constexpr int HN_CAP[4] = {128, 512, 2048, 7168};   // numeric: distinct columns
constexpr int WIN0 = 64, WIN1 = 2048, WIN2 = 8192;  // window bins: columns spanned

GM_DEV int hash_bin_sym(int64_t n) {
    return n <= HS_CAP[0] ? 0 : n <= HS_CAP[1] ? 1 : n <= HS_CAP[2] ? 2 : 3;
}
GM_DEV int hash_bin_num(int64_t nnz) {
    return nnz <= HN_CAP[0] ? 0 : nnz <= HN_CAP[1] ? 1 : nnz <= HN_CAP[2] ? 2 : 3;
}
// Numeric light rows: few distinct columns hash (table of HN_CAP[0]); rows of
// at most SORT_SMALL[1] products sort them in one wave (with LDS sized for
// SORT_SMALL[0] or SORT_SMALL[1] products, so the smaller rows fit more work
// groups per CU); then hashing for rows with at most HN_CAP[1] distinct
// columns; larger rows sort all products (by product count, SORT_CAP).
// Sorting a few hundred products in LDS (one or three 8-bit passes) costs far
// less LDS traffic than the bitonic sort of the hash table's occupied slots.
constexpr int SORT_SMALL[2] = {256, 512};
// (the middle cap keeps two 256-thread work groups per CU; the largest
// needs almost all of a CU's LDS)
constexpr int SORT_CAP[3] = {2048, 3456, 6912};
GM_DEV int light_bin_num(int64_t nnz, int64_t ip) {
    return nnz <= HN_CAP[0]        ? 0
           : ip <= SORT_SMALL[0]   ? 1
           : ip <= SORT_SMALL[1]   ? 2
           : nnz <= HN_CAP[1]      ? 3
           : ip <= SORT_CAP[0]     ? 4
           : ip <= SORT_CAP[1]     ? 5
                                   : 6;
}

// Window choice for a light row: span = max column - min column + 1.
GM_DEV int window_bin(int64_t ip, int64_t span, bool window) {
    if (!window || span <= 0) return -1;
    if (span <= WIN0) return 0;
    int64_t p2 = 1;
    while (p2 < ip) p2 <<= 1;
    if (span <= WIN1 && span <= 4 * p2) return 1;
    if (span <= WIN2 && span <= 4 * p2) return 2;  // (a 64 KB value window: rows of at least 2048 products)
    return -1;
}

// A row whose columns span 2^31 or more (possible with 64-bit columns only)
// cannot be keyed by 32-bit column offsets: it goes to the heavy path,
// whose chunks are at most 2^31 columns wide.
template <typename CI>
__global__ void k_light_classes(const int64_t *ip, const int64_t *row_nnz, const CI *minc, const CI *maxc, int64_t n,
                                int64_t tau, int window, uint8_t *cls) {
    for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p = ip[r];
        uint8_t c;
        if (p == 0)
            c = LIGHT_EMPTY;
        else if (p > tau || (int64_t)maxc[r] - (int64_t)minc[r] >= (int64_t)INT32_MAX)
            c = LIGHT_HEAVY;
        else {
            const int wb = window_bin(p, (int64_t)maxc[r] - minc[r] + 1, window != 0);
            if (wb >= 0)
                c = (uint8_t)(LIGHT_W0 + wb);
            else
                c = (uint8_t)(LIGHT_H0 + (row_nnz ? light_bin_num(row_nnz[r], p) : hash_bin_sym(p)));
        }
        cls[r] = c;
    }
}

constexpr int DENSE_MAX = 8192;          // columns of the LDS dense accumulator
constexpr int RANK_MAX_LOG2 = 18;        // columns of the bitmap-rank accumulator
constexpr int RANK_NNZ_MAX = 6912;       // distinct columns it holds (>= tau; two work groups per CU at 2^17 columns)
constexpr int RANK_MIN_LEN = 256;        // smaller chunks go to the hash map
constexpr int RANK_MID = 3584;           // distinct columns of the middle wide variant (three per CU)
constexpr int RANK_SMALL = 1792;         // distinct columns of the small wide rank variant (its LDS
                                         // stays under 32 KB: five work groups per CU)
constexpr int RANK_NARROW_CAP = 4096;    // chunks of at most DENSE_MAX columns and at most this many elements use
                                         // a rank accumulator (one work group per chunk, LDS sized by the chunk)
constexpr int RANK_NARROW_SMALL = 512;   // ... its small shape up to this many
constexpr int RANK_NARROW_MID = 2048;    // ... its middle shape up to this many
constexpr int RANK_WIDE_SMALL = 1024;    // wider chunks of at most this many elements count their columns with
                                         // the small wide shape

// Accumulator of a final chunk of `len` elements over `width` columns.
// Chunks of at most W columns: above RANK_NARROW_CAP elements the dense
// accumulator (a persistent kernel with the W-column value array in LDS);
// up to RANK_NARROW_CAP the bitmap-rank accumulator, one work group per
// chunk with LDS sized by the chunk, so many chunks run on a CU at once (the
// dense kernel pays a chain of memory latencies per chunk, and holds two work
// groups per CU); chunks below RANK_MIN_LEN take a one-wave shape whose word
// ranks come from a single wave scan (no hash table to sort). Wider
// chunks: the bitmap-rank accumulator while the bitmap fits LDS, else the
// hash map.
__global__ void k_leaf_classes(LeafSet L, const int64_t *leaf_nnz, int64_t tau, int64_t width, uint8_t *cls) {
    const int64_t n = L.hi - L.lo;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t j = L.lo + i;
        const int64_t len = L.ptr[j + 1] - L.ptr[j];
        uint8_t c;
        if (len == 0)
            c = LEAF_EMPTY;
        else if (width <= DENSE_MAX && width >= 32 && len < RANK_MIN_LEN)
            c = LEAF_RANK_T;
        else if (width <= DENSE_MAX && width >= 32 && len <= RANK_NARROW_CAP)
            c = len > RANK_NARROW_MID ? LEAF_RANK_XL : len > RANK_NARROW_SMALL ? LEAF_RANK_L : LEAF_RANK;
        else if (width <= DENSE_MAX && width >= 32 && len > RANK_NARROW_CAP)
            c = len >= DENSE_BIG_LEN ? LEAF_DENSE_BIG : LEAF_DENSE;
        else if (width < 32 && (len > tau || len >= width / 16))
            c = len >= DENSE_BIG_LEN ? LEAF_DENSE_BIG : LEAF_DENSE;
        else if (width <= (1 << RANK_MAX_LOG2) && width >= 32 && len >= RANK_MIN_LEN)
            // symbolic: the small wide shape for small chunks; numeric: by distinct columns
            // (for wide numeric chunks LEAF_RANK is the middle size, up to RANK_MID columns)
            c = !leaf_nnz ? (len <= RANK_WIDE_SMALL ? LEAF_RANK : LEAF_RANK_L)
                          : (leaf_nnz[i] <= RANK_SMALL ? LEAF_RANK_L
                             : leaf_nnz[i] <= RANK_MID ? LEAF_RANK
                                                       : LEAF_RANK_XL);
        else
            c = (uint8_t)(LEAF_H0 + (leaf_nnz ? hash_bin_num(leaf_nnz[i]) : hash_bin_sym(len)));
        cls[i] = c;
    }
}

// ------------------------------------------------------------- light rows
// Key base of a light row: 0 for 32-bit columns (keys are the columns), the
// row's smallest column for 64-bit ones (keys are offsets from it).
template <typename CI>
GM_DEV CI light_base(const CI *minc, int64_t r) {
    return sizeof(CI) == 8 ? minc[r] : (CI)0;
}

template <int BLOCK, int TS, typename CI>
__global__ __launch_bounds__(BLOCK) void k_light_hash_sym(CsrV<CI, NoV> A, CsrV<CI, NoV> B, int64_t r0,
                                                          const int64_t *items, const CI *minc, int64_t *row_nnz) {
    __shared__ int32_t keys[TS];
    __shared__ GusLds<BLOCK, NoV> G;
    __shared__ int32_t counter;
    const int64_t r = items[blockIdx.x];
    hash_clear<BLOCK, TS, double>(keys, nullptr);
    if (threadIdx.x == 0) counter = 0;
    __syncthreads();
    gustavson_row<BLOCK, false>(A, B, A.rp[r0 + r], A.rp[r0 + r + 1], light_base(minc, r), G,
                                [&](int32_t c, NoV) { hash_insert_key<TS>(keys, c, &counter); });
    if (threadIdx.x == 0) row_nnz[r] = counter;
}

template <int BLOCK, int TS, typename CI, typename V>
__global__ __launch_bounds__(BLOCK) void k_light_hash_num(CsrV<CI, V> A, CsrV<CI, V> B, int64_t r0,
                                                          const int64_t *items, const CI *minc,
                                                          const int64_t *c_row_ptr, CI *c_col, V *c_val,
                                                          int32_t *err) {
    __shared__ int32_t keys[TS];
    __shared__ V vals[TS];
    __shared__ GusLds<BLOCK, V> G;
    const int64_t r = items[blockIdx.x];
    const CI base = light_base(minc, r);
    hash_clear<BLOCK, TS>(keys, vals);
    __syncthreads();
    gustavson_row<BLOCK, true>(A, B, A.rp[r0 + r], A.rp[r0 + r + 1], base, G,
                               [&](int32_t c, V v) { hash_insert_add<TS>(keys, vals, c, v); });
    const int64_t dst = c_row_ptr[r];
    hash_emit_sorted<BLOCK, TS>(keys, vals, c_row_ptr[r + 1] - dst, base, c_col + dst, c_val + dst, G.scan, err);
}

// ------------------------------------------------ sort-based light rows
// Light rows with many distinct columns (their products barely repeat a
// column): every product is placed in LDS as (column - row minimum, value),
// the columns are sorted with a stable LSD radix sort carrying the product
// index, and runs of equal columns are summed into the row. This replaces a
// hash table plus a bitonic sort of the whole table, whose many
// barrier-separated stages dominated these rows.

// Stable LSD radix sort of n <= CAP keys in LDS, 8-bit digits over the low
// `bits` bits, with a 16-bit payload. Wave w ranks the contiguous range
// [w*S, w*S + S) in 64-element batches: lanes with equal digits are found
// with eight ballots, and per-(digit, wave) counters scanned digit-major give
// every element its place, so equal digits keep their order. On return
// (keys, idx) point at the sorted arrays (the two buffers are swapped).
template <int BLOCK, int CAP>
GM_DEV void radix_sort_lds(uint32_t *&keys, uint16_t *&idx, uint32_t *&keys_alt, uint16_t *&idx_alt, int n,
                           int bits, int32_t *hist, int32_t *scan_sm) {
    constexpr int NW = BLOCK / GM_WAVE;
    constexpr int NB = (CAP + BLOCK - 1) / BLOCK;  // 64-element batches per wave
    constexpr int S = NB * GM_WAVE;
    constexpr int NH = NW * 256;
    constexpr int HPT = NH / BLOCK;
    static_assert(HPT * BLOCK == NH, "counters per thread");
    const int tid = threadIdx.x, lane = tid & (GM_WAVE - 1), w = tid / GM_WAVE;
    const uint64_t lt = lanemask_lt();
    for (int shift = 0; shift < bits; shift += 8) {
        for (int i = tid; i < NH; i += BLOCK) hist[i] = 0;
        __syncthreads();
        int rk[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (w * S + b * GM_WAVE >= n) break;  // the wave's remaining batches are empty
            const int i = w * S + b * GM_WAVE + lane;
            const bool valid = i < n;
            const uint32_t d = valid ? (keys[i] >> shift) & 255u : 0u;
            uint64_t peers = ballot(valid);
#pragma unroll
            for (int bit = 0; bit < 8; ++bit) {
                const uint64_t m = ballot((d >> bit) & 1u);
                peers &= ((d >> bit) & 1u) ? m : ~m;
            }
            const int leader = peers ? __ffsll((long long)peers) - 1 : lane;
            int base = 0;
            if (valid && lane == leader) {
                base = hist[d * NW + w];
                hist[d * NW + w] = base + __popcll(peers);
            }
            base = __shfl(base, leader, GM_WAVE);
            rk[b] = base + __popcll(peers & lt);
        }
        __syncthreads();
        // exclusive scan of the counters in (digit, wave) order
        {
            int32_t v[HPT], sum = 0;
#pragma unroll
            for (int j = 0; j < HPT; ++j) {
                v[j] = hist[tid * HPT + j];
                sum += v[j];
            }
            int32_t run = block_excl_scan<BLOCK>(sum, scan_sm);
#pragma unroll
            for (int j = 0; j < HPT; ++j) {
                hist[tid * HPT + j] = run;
                run += v[j];
            }
        }
        __syncthreads();
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (w * S + b * GM_WAVE >= n) break;
            const int i = w * S + b * GM_WAVE + lane;
            if (i < n) {
                const uint32_t k = keys[i];
                const int pos = hist[((k >> shift) & 255u) * NW + w] + rk[b];
                keys_alt[pos] = k;
                idx_alt[pos] = idx[i];
            }
        }
        __syncthreads();
        uint32_t *tk = keys;
        keys = keys_alt;
        keys_alt = tk;
        uint16_t *ti = idx;
        idx = idx_alt;
        idx_alt = ti;
    }
}

// Rows of at most a few hundred products whose columns spread evenly (ER-like)
// need one pass, not three: a stable scatter by the top 8 bits of the key
// leaves buckets of a few elements, and each element's final place is its
// bucket's start plus the number of smaller keys (or equal keys placed
// earlier) in its bucket. Returns false, with keys and idx untouched, when a
// bucket holds more than MSD_MAXB elements (the caller then radix-sorts).
constexpr int MSD_MAXB = 16;

GM_DEV int32_t wave_reduce_max(int32_t x) {
#pragma unroll
    for (int d = GM_WAVE / 2; d >= 1; d >>= 1) {
        const int32_t y = __shfl_xor(x, d, GM_WAVE);
        x = x > y ? x : y;
    }
    return x;
}

template <int BLOCK, int CAP>
GM_DEV bool msd_sort_lds(uint32_t *keys, uint16_t *idx, uint32_t *keys_alt, uint16_t *idx_alt, int n, int bits,
                         int32_t *hist, int32_t *scan_sm) {
    constexpr int NW = BLOCK / GM_WAVE;
    constexpr int NB = (CAP + BLOCK - 1) / BLOCK;
    constexpr int S = NB * GM_WAVE;
    constexpr int NH = NW * 256;
    constexpr int HPT = NH / BLOCK;
    const int tid = threadIdx.x, lane = tid & (GM_WAVE - 1), w = tid / GM_WAVE;
    const uint64_t lt = lanemask_lt();
    const int shift = bits > 8 ? bits - 8 : 0;
    for (int i = tid; i < NH; i += BLOCK) hist[i] = 0;
    __syncthreads();
    int rk[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (w * S + b * GM_WAVE >= n) break;
        const int i = w * S + b * GM_WAVE + lane;
        const bool valid = i < n;
        const uint32_t d = valid ? (keys[i] >> shift) & 255u : 0u;
        uint64_t peers = ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
            const uint64_t m = ballot((d >> bit) & 1u);
            peers &= ((d >> bit) & 1u) ? m : ~m;
        }
        const int leader = peers ? __ffsll((long long)peers) - 1 : lane;
        int base = 0;
        if (valid && lane == leader) {
            base = hist[d * NW + w];
            hist[d * NW + w] = base + __popcll(peers);
        }
        base = __shfl(base, leader, GM_WAVE);
        rk[b] = base + __popcll(peers & lt);
    }
    __syncthreads();
    // largest bucket
    int big = 0;
    for (int d = tid; d < 256; d += BLOCK) {
        int sz = 0;
#pragma unroll
        for (int q = 0; q < NW; ++q) sz += hist[d * NW + q];
        big = big > sz ? big : sz;
    }
    big = (int)wave_reduce_max(big);
    if (lane == 0) scan_sm[w] = big;
    __syncthreads();
    big = 0;
#pragma unroll
    for (int q = 0; q < NW; ++q) big = big > scan_sm[q] ? big : scan_sm[q];
    __syncthreads();
    if (big > MSD_MAXB) return false;  // uniform across the work group
    // stable scatter by bucket into the alternate buffers
    {
        int32_t v[HPT], sum = 0;
#pragma unroll
        for (int j = 0; j < HPT; ++j) {
            v[j] = hist[tid * HPT + j];
            sum += v[j];
        }
        int32_t run = block_excl_scan<BLOCK>(sum, scan_sm);
#pragma unroll
        for (int j = 0; j < HPT; ++j) {
            hist[tid * HPT + j] = run;
            run += v[j];
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (w * S + b * GM_WAVE >= n) break;
        const int i = w * S + b * GM_WAVE + lane;
        if (i < n) {
            const uint32_t k = keys[i];
            const int pos = hist[((k >> shift) & 255u) * NW + w] + rk[b];
            keys_alt[pos] = k;
            idx_alt[pos] = idx[i];
        }
    }
    __syncthreads();
    // place inside the bucket, back into keys/idx
    for (int p = tid; p < n; p += BLOCK) {
        const uint32_t k = keys_alt[p];
        const uint32_t d = (k >> shift) & 255u;
        const int b0 = hist[d * NW], b1 = d < 255 ? hist[(d + 1) * NW] : n;
        int r = b0;
        for (int q = b0; q < b1; ++q) {
            const uint32_t kq = keys_alt[q];
            r += (kq < k || (kq == k && q < p)) ? 1 : 0;
        }
        keys[r] = k;
        idx[r] = idx_alt[p];
    }
    __syncthreads();
    return true;
}

template <int BLOCK, int CAP, typename V>
struct SortLds {
    uint32_t keys[2][CAP];
    V vals[CAP];
    uint16_t idx[2][CAP];
    int32_t hist[(BLOCK / GM_WAVE) * 256];
    int32_t off[BLOCK + 1];
    int64_t bst[BLOCK];
    V av[BLOCK];
    int32_t scan[BLOCK / GM_WAVE];
};

constexpr int SORT_ILP = 4;

// Writes the sums of the runs of equal keys of a sorted (keys, idx) array in
// key order: heads counted per thread over a contiguous range, their output
// positions kept in idx_free, then each head sums its run into out_val at its
// position (consecutive lanes on consecutive positions) and writes
// key + base_col to out_col. Sets err_bit in *err when the run count differs
// from nnz (the symbolic count).
template <int BLOCK, int CAP, typename V, typename CI>
GM_DEV void sorted_runs_emit(const uint32_t *keys, const uint16_t *idx, uint16_t *idx_free, const V *vals, int n,
                             int64_t nnz, CI base_col, CI *out_col, V *out_val, int32_t *err, int err_bit,
                             int32_t *scan_sm) {
    const int tid = threadIdx.x;
    constexpr int PT = (CAP + BLOCK - 1) / BLOCK;
    const int p0 = tid * PT;
    int32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < PT; ++j) {
        const int p = p0 + j;
        if (p < n && (p == 0 || keys[p] != keys[p - 1])) ++cnt;
    }
    int32_t total;
    int32_t pos = block_excl_scan<BLOCK>(cnt, scan_sm, &total);
#pragma unroll
    for (int j = 0; j < PT; ++j) {
        const int p = p0 + j;
        if (p < n && (p == 0 || keys[p] != keys[p - 1])) idx_free[p] = (uint16_t)pos++;
    }
    __syncthreads();
    if (tid == 0 && total != nnz) atomicOr(err, err_bit);
    for (int p = tid; p < n; p += BLOCK) {
        const uint32_t k = keys[p];
        if (p == 0 || k != keys[p - 1]) {
            const int o = idx_free[p];
            V sum = vals[idx[p]];
            for (int q = p + 1; q < n && keys[q] == k; ++q) sum += vals[idx[q]];
            if (o < nnz) {
                out_col[o] = (CI)k + base_col;
                out_val[o] = sum;
            }
        }
    }
}

template <int BLOCK, int CAP, typename CI, typename V>
__global__ __launch_bounds__(BLOCK) void k_light_sort_num(CsrV<CI, V> A, CsrV<CI, V> B, int64_t r0,
                                                          const int64_t *items, const CI *minc, const CI *maxc,
                                                          const int64_t *c_row_ptr, CI *c_col, V *c_val,
                                                          int32_t *err) {
    static_assert(CAP < 65536, "16-bit product indices");
    __shared__ SortLds<BLOCK, CAP, V> L;
    const int tid = threadIdx.x;
    const int64_t r = items[blockIdx.x];
    const CI base_col = minc[r];
    const uint32_t span = (uint32_t)(maxc[r] - base_col);
    const int64_t j0 = A.rp[r0 + r], j1 = A.rp[r0 + r + 1];
    const int64_t dst = c_row_ptr[r], nnz = c_row_ptr[r + 1] - dst;
    // gather every product of the row: A entries in batches of BLOCK
    int n = 0;
    for (int64_t jb = j0; jb < j1; jb += BLOCK) {
        const int nb = (int)(j1 - jb < BLOCK ? j1 - jb : BLOCK);
        int32_t len = 0;
        if (tid < nb) {
            const int64_t k = (int64_t)A.ci[jb + tid];
            const int64_t bs = B.rp[k];
            len = (int32_t)(B.rp[k + 1] - bs);
            L.bst[tid] = bs;
            L.av[tid] = A.v[jb + tid];
        }
        int32_t tot;
        const int32_t ex = block_excl_scan<BLOCK>(len, L.scan, &tot);
        L.off[tid] = tid < nb ? ex : INT32_MAX;
        __syncthreads();
        if (n + tot > CAP) {  // cannot happen for a light row of this bin (ip <= CAP)
            if (tid == 0) atomicOr(err, 8);
            return;
        }
        // as in gustavson_row: searches, then every load, with no branch between them
        for (int tb = tid; tb < tot; tb += BLOCK * SORT_ILP) {
            int q[SORT_ILP];
            int64_t src[SORT_ILP];
#pragma unroll
            for (int u = 0; u < SORT_ILP; ++u) {
                const int t = tb + u * BLOCK < tot ? tb + u * BLOCK : tot - 1;
                q[u] = entry_of<BLOCK>(L.off, t);
                src[u] = L.bst[q[u]] + (t - L.off[q[u]]);
            }
            CI c[SORT_ILP];
            V v[SORT_ILP];
#pragma unroll
            for (int u = 0; u < SORT_ILP; ++u) {
                c[u] = B.ci[src[u]];
                v[u] = B.v[src[u]];
            }
#pragma unroll
            for (int u = 0; u < SORT_ILP; ++u) v[u] *= L.av[q[u]];
#pragma unroll
            for (int u = 0; u < SORT_ILP; ++u) {
                const int t = tb + u * BLOCK;
                if (t < tot) {
                    L.keys[0][n + t] = (uint32_t)(c[u] - base_col);
                    L.vals[n + t] = v[u];
                    L.idx[0][n + t] = (uint16_t)(n + t);
                }
            }
        }
        n += tot;
        __syncthreads();
    }
    const int bits = span == 0 ? 0 : 32 - __clz((int)span);
    uint32_t *keys = L.keys[0], *keys_alt = L.keys[1];
    uint16_t *idx = L.idx[0], *idx_alt = L.idx[1];
    if (CAP > 512 || !msd_sort_lds<BLOCK, CAP>(keys, idx, keys_alt, idx_alt, n, bits, L.hist, L.scan))
        radix_sort_lds<BLOCK, CAP>(keys, idx, keys_alt, idx_alt, n, bits, L.hist, L.scan);
    sorted_runs_emit<BLOCK, CAP>(keys, idx, idx_alt, (const V *)L.vals, n, nnz, base_col, c_col + dst, c_val + dst,
                                 err, 1, L.scan);
}

// Dense window of a light row: one presence byte per column, set with a
// plain LDS store (every product of a column stores the same 1, so no atomic
// and no read are needed; the columns of a banded row repeat many times), and
// for the numeric phase a value per column added with an LDS atomic.
template <int BLOCK, int WMAX, bool VALS, typename V = double>
struct WinLds {
    V vals[VALS ? WMAX : 1];
    uint8_t flag[WMAX];
    int32_t scan[BLOCK / GM_WAVE];
};

template <int BLOCK, int WMAX, bool VALS, typename V>
GM_DEV void win_clear(WinLds<BLOCK, WMAX, VALS, V> &L, int width) {
    uint32_t *f = (uint32_t *)L.flag;
    for (int i = threadIdx.x; i < (width + 3) / 4; i += BLOCK) f[i] = 0u;
    if (VALS)
        for (int i = threadIdx.x; i < width; i += BLOCK) L.vals[i] = (V)0;
}

// number of present columns (flag words read 4 bytes at a time)
template <int BLOCK, int WMAX, bool VALS, typename V>
GM_DEV int32_t win_count(WinLds<BLOCK, WMAX, VALS, V> &L, int width) {
    const uint32_t *f = (const uint32_t *)L.flag;
    int32_t c = 0;
    for (int i = threadIdx.x; i < (width + 3) / 4; i += BLOCK) c += __popc(f[i]);  // each present byte is 0x01
    return block_reduce_sum<BLOCK>(c, L.scan);
}

// Writes the present columns in increasing order (as dense_emit, with the
// presence bytes in place of the bitmap).
template <int BLOCK, int WMAX, typename V, typename CI>
GM_DEV void win_emit(WinLds<BLOCK, WMAX, true, V> &L, int width, int64_t nnz, CI col_base, CI *out_col, V *out_val,
                     int32_t *err) {
    constexpr int NW = BLOCK / GM_WAVE;
    const int lane = threadIdx.x & (GM_WAVE - 1), w = threadIdx.x / GM_WAVE;
    const int span = ((width + NW - 1) / NW + GM_WAVE - 1) / GM_WAVE * GM_WAVE;
    const int c0 = w * span, c1 = c0 + span < width ? c0 + span : width;
    int32_t cnt = 0;
    for (int c = c0 + lane; c < c1; c += GM_WAVE) cnt += L.flag[c];
    cnt = wave_reduce_sum(cnt);
    int32_t total;
    int32_t base = block_excl_scan<BLOCK>(lane == 0 ? cnt : 0, L.scan, &total);
    base = __shfl(base, 0, GM_WAVE);
    if (threadIdx.x == 0 && total != nnz) atomicOr(err, 2);
    for (int g = c0; g < c1; g += GM_WAVE) {
        const int c = g + lane;
        const bool p = c < c1 && L.flag[c];
        const uint64_t m = ballot(p);
        const int pos = base + __popcll(m & lanemask_lt());
        if (p && pos < nnz) {
            out_col[pos] = (CI)c + col_base;
            out_val[pos] = L.vals[c];
        }
        base += __popcll(m);
    }
}

template <int BLOCK, int WMAX, typename CI>
__global__ __launch_bounds__(BLOCK) void k_light_win_sym(CsrV<CI, NoV> A, CsrV<CI, NoV> B, int64_t r0,
                                                         const int64_t *items, const CI *minc, const CI *maxc,
                                                         int64_t *row_nnz) {
    __shared__ WinLds<BLOCK, WMAX, false> D;
    __shared__ GusLds<BLOCK, NoV> G;
    const int64_t r = items[blockIdx.x];
    const CI base = minc[r];
    const int width = (int)(maxc[r] - base + 1);
    win_clear(D, width);
    __syncthreads();
    gustavson_row<BLOCK, false>(A, B, A.rp[r0 + r], A.rp[r0 + r + 1], base, G,
                                [&](int32_t c, NoV) { D.flag[c] = 1; });
    __syncthreads();
    const int32_t cnt = win_count(D, width);
    if (threadIdx.x == 0) row_nnz[r] = cnt;
}

template <int BLOCK, int WMAX, typename CI, typename V>
__global__ __launch_bounds__(BLOCK) void k_light_win_num(CsrV<CI, V> A, CsrV<CI, V> B, int64_t r0,
                                                         const int64_t *items, const CI *minc, const CI *maxc,
                                                         const int64_t *c_row_ptr, CI *c_col, V *c_val,
                                                         int32_t *err) {
    __shared__ WinLds<BLOCK, WMAX, true, V> D;
    __shared__ GusLds<BLOCK, V> G;
    const int64_t r = items[blockIdx.x];
    const CI base = minc[r];
    const int width = (int)(maxc[r] - base + 1);
    win_clear(D, width);
    __syncthreads();
    gustavson_row<BLOCK, true>(A, B, A.rp[r0 + r], A.rp[r0 + r + 1], base, G, [&](int32_t c, V v) {
        D.flag[c] = 1;
        __hip_atomic_fetch_add(&D.vals[c], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    });
    __syncthreads();
    const int64_t dst = c_row_ptr[r];
    win_emit(D, width, c_row_ptr[r + 1] - dst, base, c_col + dst, c_val + dst, err);
}

// Narrow-window symbolic from B-row column masks. A light row whose columns
// span at most WIN0 = 64 uses only B rows that span at most 64 columns, so
// each such B row k is summarized once by (its first column, a 64-bit mask of
// its columns relative to that one); the row's distinct columns are then the
// popcount of the OR of its entries' masks shifted to the row's smallest
// column: one mask read per A entry instead of one column read per product.
// Rows of B that are empty or span more than 64 columns get mask 0 (such a
// row never reaches a narrow-window row of A, except empty ones, which add nothing).
template <typename CI>
__global__ void k_brow_masks(CsrV<CI, NoV> B, uint64_t *mask, CI *first) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < B.n_rows;
         k += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b0 = B.rp[k], b1 = B.rp[k + 1];
        uint64_t m = 0;
        CI f = 0;
        if (b1 > b0) {
            f = B.ci[b0];
            if ((int64_t)B.ci[b1 - 1] - (int64_t)f < WIN0)
                for (int64_t j = b0; j < b1; ++j) m |= uint64_t(1) << (int)(B.ci[j] - f);
        }
        mask[k] = m;
        first[k] = f;
    }
}

template <typename CI>
__global__ void k_light_win0_sym_masks(CsrV<CI, NoV> A, int64_t r0, const int64_t *items, int64_t n, const CI *minc,
                                       const uint64_t *mask, const CI *first, int64_t *row_nnz) {
    constexpr int U = 8;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = items[i];
        const CI base = minc[r];
        const int64_t j0 = A.rp[r0 + r], j1 = A.rp[r0 + r + 1];
        uint64_t acc = 0;
        for (int64_t jb = j0; jb < j1; jb += U) {
            int64_t k[U];
#pragma unroll
            for (int u = 0; u < U; ++u) k[u] = (int64_t)A.ci[jb + u < j1 ? jb + u : j0];
            uint64_t m[U];
            CI f[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                m[u] = mask[k[u]];
                f[u] = first[k[u]];
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (jb + u < j1 && m[u]) acc |= m[u] << (int)(f[u] - base);
        }
        row_nnz[r] = __popcll(acc);
    }
}

// ------------------------------------------------------------------ leaves
template <int BLOCK, int TS>
__global__ __launch_bounds__(BLOCK) void k_leaf_hash_sym(LeafSet L, const LeafTask *tasks, int64_t *leaf_nnz,
                                                         int64_t *slot_cnt) {
    __shared__ int32_t keys[TS];
    __shared__ int32_t counter;
    const LeafTask tk = tasks[blockIdx.x];
    const int64_t s = tk.s, e = tk.e;
    hash_clear<BLOCK, TS, double>(keys, nullptr);
    if (threadIdx.x == 0) counter = 0;
    __syncthreads();
    for (int64_t t = s + threadIdx.x; t < e; t += BLOCK) hash_insert_key<TS>(keys, leaf_col(L, t), &counter);
    __syncthreads();
    if (threadIdx.x == 0) {
        leaf_nnz[tk.a] = counter;
        slot_cnt[tk.t] = counter;
    }
}

// Where a leaf's output goes: the slot grid of the heavy rows.
struct LeafOut {
    int64_t n_slots_log2;
    const int64_t *heavy_rows;
    const int64_t *c_row_ptr;
    const int64_t *slot_off;
};

// C's arrays for the numeric leaf kernels; a leaf's first column is its
// slot << slot_width_log2.
template <typename CI, typename V>
struct LeafDst {
    CI *c_col;
    V *c_val;
    int32_t *err;
    int slot_width_log2;
    GM_DEV CI base(const LeafTask &tk) const { return (CI)tk.b << slot_width_log2; }
};

GM_DEV void leaf_target(const LeafOut &o, int64_t origin, int64_t &dst, int64_t &nnz_cap, int32_t &slot) {
    const int64_t h = origin >> o.n_slots_log2;
    slot = (int32_t)(origin & ((int64_t(1) << o.n_slots_log2) - 1));
    const int64_t row = o.heavy_rows[h];
    dst = o.c_row_ptr[row] + o.slot_off[origin];
    nnz_cap = o.c_row_ptr[row + 1] - dst;
}

// Per-leaf launch records, in the order of a bin partition, so every leaf
// work group starts from one load instead of a chain of dependent ones.
__global__ void k_leaf_tasks_sym(LeafSet L, const int64_t *items, int64_t n, LeafTask *tasks) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n; k += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = items[k];
        const int64_t j = L.lo + i;
        tasks[k] = LeafTask{L.ptr[j], L.ptr[j + 1], L.origin[j], (int32_t)i, 0};
    }
}

__global__ void k_leaf_tasks_num(LeafSet L, const int64_t *items, int64_t n, const int64_t *leaf_nnz, LeafOut o,
                                 LeafTask *tasks) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n; k += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = items[k];
        const int64_t j = L.lo + i;
        int64_t dst, cap;
        int32_t slot;
        leaf_target(o, L.origin[j], dst, cap, slot);
        const int64_t nnz = leaf_nnz[i] < cap ? leaf_nnz[i] : cap;
        tasks[k] = LeafTask{L.ptr[j], L.ptr[j + 1], dst, (int32_t)nnz, slot};
    }
}

template <int BLOCK, int TS, typename CI, typename V>
__global__ __launch_bounds__(BLOCK) void k_leaf_hash_num(LeafSet L, const LeafTask *tasks, LeafDst<CI, V> o) {
    __shared__ int32_t keys[TS];
    __shared__ V vals[TS];
    __shared__ int32_t scan_sm[BLOCK / GM_WAVE];
    const LeafTask tk = tasks[blockIdx.x];
    const int64_t s = tk.s, e = tk.e;
    const V *lv = static_cast<const V *>(L.val);
    hash_clear<BLOCK, TS>(keys, vals);
    __syncthreads();
    for (int64_t t = s + threadIdx.x; t < e; t += BLOCK) hash_insert_add<TS>(keys, vals, leaf_col(L, t), lv[t]);
    __syncthreads();
    const int64_t dst = tk.t, nnz = tk.a;
    hash_emit_sorted<BLOCK, TS>(keys, vals, nnz, o.base(tk), o.c_col + dst, o.c_val + dst, scan_sm, o.err);
}


// Calls f(column) for the elements [s, e) of a column array, reading it in
// aligned 16-byte blocks (elements outside [s, e) skipped); a block that
// would reach past e_end, the end of the array's valid elements, is read
// element by element.
template <int BLOCK, int U, typename ColT, typename F>
GM_DEV void for_each_col_vec(const ColT *col, int64_t s, int64_t e, int64_t e_end, F f) {
    constexpr int PER = 16 / (int)sizeof(ColT);
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    for (int64_t b = (s & ~(int64_t)(PER - 1)) + (int64_t)threadIdx.x * PER; b < e; b += (int64_t)BLOCK * PER * U) {
        ColT v[U][PER];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t blk = b + (int64_t)u * BLOCK * PER;
            if (blk + PER <= e_end) {
                const u32x4 q = __builtin_nontemporal_load((const u32x4 *)(col + blk));
                __builtin_memcpy(v[u], &q, 16);
            } else {
#pragma unroll
                for (int j = 0; j < PER; ++j) v[u][j] = blk + j < e ? col[blk + j] : (ColT)0;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < PER; ++j) {
                const int64_t t = b + (int64_t)u * BLOCK * PER + j;
                if (t >= s && t < e) f((int32_t)v[u][j]);
            }
    }
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_leaf_dense_sym(LeafSet L, const LeafTask *tasks, int width, int64_t e_end,
                                                          int64_t *leaf_nnz, int64_t *slot_cnt) {
    __shared__ DenseBits<BLOCK, DENSE_MAX> D;
    const LeafTask tk = tasks[blockIdx.x];
    const int64_t s = tk.s, e = tk.e;
    dense_clear(D, width, false);
    __syncthreads();
    // 16-byte column loads (the caller checked the column array's alignment)
    if (L.col16)
        for_each_col_vec<BLOCK, 2>(L.col16, s, e, e_end, [&](int32_t c) { dense_set(D, c); });
    else
        for_each_col_vec<BLOCK, 2>(L.col, s, e, e_end, [&](int32_t c) { dense_set(D, c); });
    __syncthreads();
    const int32_t cnt = dense_count(D, width);
    if (threadIdx.x == 0) {
        leaf_nnz[tk.a] = cnt;
        slot_cnt[tk.t] = cnt;
    }
}

// Numeric dense accumulation, 1024 threads (16 waves) per work group, two
// work groups per CU (64 KB of values each). The work groups are persistent:
// each takes chunks from an atomic counter, in the bin order (the big dense
// chunks first). While a chunk is written out, the next chunk's record and
// first batch of elements are already being loaded, and the write-out leaves
// the accumulator zeroed, so the loads of one chunk overlap the LDS work of
// the previous one. Within a chunk the next batch's loads are issued before
// the current batch's LDS atomics.
constexpr int DENSE_BLOCK = 1024, DENSE_EPT = 2, DENSE_GROUPS_PER_CU = 2;

template <int BLOCK, int EPT, typename V>
GM_DEV void dense_load(const LeafSet &L, int64_t b, int64_t e, int32_t (&c)[EPT], V (&v)[EPT]) {
    const V *lv = static_cast<const V *>(L.val);
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
        const int64_t t = b + q * BLOCK + threadIdx.x;
        c[q] = t < e ? leaf_col_nt(L, t) : -1;
        v[q] = t < e ? __builtin_nontemporal_load(&lv[t]) : (V)0;
    }
}

// (at most 64 VGPRs: two 16-wave work groups per CU need 8 waves per SIMD)
template <int BLOCK, int EPT, typename CI, typename V>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(8))) void k_leaf_dense_num(
    LeafSet L, const LeafTask *tasks, int64_t n_tasks, int width, LeafDst<CI, V> o, int32_t *counter) {
    __shared__ DenseLds<BLOCK, DENSE_MAX, V> D;
    __shared__ int32_t grabbed;
    constexpr int STEP = BLOCK * EPT;
    if (threadIdx.x == 0) grabbed = atomicAdd(counter, 1);
    dense_clear(D, width, true);
    __syncthreads();
    int64_t cur = grabbed;
    if (cur >= n_tasks) return;  // uniform across the work group
    LeafTask tk = tasks[cur];
    int32_t c[EPT];
    V v[EPT];
    dense_load<BLOCK, EPT>(L, tk.s, tk.e, c, v);
    while (true) {
        __syncthreads();  // the accumulator is clear and everyone has read `grabbed`
        if (threadIdx.x == 0) grabbed = atomicAdd(counter, 1);
        for (int64_t b = tk.s; b < tk.e; b += STEP) {
            int32_t cn[EPT];
            V vn[EPT];
            dense_load<BLOCK, EPT>(L, b + STEP, tk.e, cn, vn);
#pragma unroll
            for (int q = 0; q < EPT; ++q)
                if (c[q] >= 0) dense_add(D, c[q], v[q]);
#pragma unroll
            for (int q = 0; q < EPT; ++q) {
                c[q] = cn[q];
                v[q] = vn[q];
            }
        }
        __syncthreads();
        const int64_t nxt = grabbed;
        LeafTask tn{};
        if (nxt < n_tasks) {
            tn = tasks[nxt];
            dense_load<BLOCK, EPT>(L, tn.s, tn.e, c, v);  // in flight during the write-out
        }
        dense_emit_clear(D, width, tk.a, o.base(tk), o.c_col + tk.t, o.c_val + tk.t, o.err);
        if (nxt >= n_tasks) break;
        tk = tn;
    }
}

// Bitmap-rank accumulator for light chunks whose column range is too wide
// for a dense value array: a one-bit-per-column bitmap marks the present
// columns, an exclusive scan of the bitmap words' popcounts gives every
// present column its rank, i.e. its position in the sorted output, and the
// values are summed straight into a rank-indexed array. No hashing and no
// sort; the output comes out in column order. A chunk is light (at most tau
// elements), so its elements stay in registers between the two passes.
//
// The element that first sets a column's bit writes that column to C at the
// column's rank; chunks are made of sorted B-row runs over consecutive lanes,
// so these stores are mostly consecutive. Two shapes: 256 threads with a
// 256-word bitmap and 512 value slots for chunks of at most 8192 columns
// (those hold fewer than 512 elements, so many work groups fit a CU), and
// 512 threads with up to 2^18 columns for the wide light chunks.
constexpr int RANK_BLOCK = 512;
constexpr int RANK_EPT = 16;  // RANK_BLOCK * RANK_EPT >= tau_limit()
constexpr int RANK_WBLOCK = 256, RANK_WEPT = 4;  // the small wide shape
constexpr int RANK_L2BLOCK = 512, RANK_L2EPT = 14;  // the same in 8 waves: twice the waves per CU when the
                                                   // LDS caps the work groups (R-MAT 23's 2^18 columns:
                                                   // 193 -> 150 ms per step for these kernels)
constexpr int RANK_X2BLOCK = 1024, RANK_X2EPT = 8;  // 16 waves for the shapes whose LDS allows two groups per CU
constexpr int RANK_LBLOCK = 256, RANK_LWEPT = 27;  // wide symbolic at 2^17 columns: 4 waves and 16 KB of
                                                   // LDS, so eight work groups share a CU
static_assert(RANK_LBLOCK * RANK_LWEPT >= SORT_CAP[2] && RANK_BLOCK * RANK_EPT >= SORT_CAP[2] &&
                  RANK_L2BLOCK * RANK_L2EPT >= SORT_CAP[2] && RANK_X2BLOCK * RANK_X2EPT >= SORT_CAP[2],
              "the wide shapes hold a light chunk of up to the largest tau");
static_assert(RANK_WBLOCK * RANK_WEPT >= RANK_WIDE_SMALL, "the small wide shape holds its chunks");
constexpr int RANK_SBLOCK = 256, RANK_SWORDS = 256, RANK_SCAP = 512, RANK_SEPT = 2, RANK_LEPT = 8;
static_assert(RANK_SBLOCK * RANK_SEPT >= RANK_NARROW_SMALL && RANK_SCAP >= RANK_NARROW_SMALL,
              "the small narrow shape holds its chunks");
static_assert(RANK_SBLOCK * RANK_LEPT >= RANK_NARROW_MID, "the middle narrow shape holds its chunks");
constexpr int RANK_XBLOCK = 512;
static_assert(RANK_XBLOCK * RANK_LEPT >= RANK_NARROW_CAP, "the large narrow shape holds its chunks");
static_assert(RANK_SWORDS * 32 == DENSE_MAX, "narrow bitmap covers the dense width");
constexpr int RANK_TBLOCK = 64, RANK_TEPT = 4;  // one wave for narrow chunks below RANK_MIN_LEN elements
static_assert(RANK_TBLOCK * RANK_TEPT >= RANK_MIN_LEN, "the one-wave shape holds its chunks");

template <int BLOCK, int EPT, typename V>
GM_DEV void rank_load(const LeafSet &L, int64_t s, int64_t e, int32_t (&c)[EPT], V (&v)[EPT], bool vals) {
    const V *lv = static_cast<const V *>(L.val);
#pragma unroll
    for (int q = 0; q < EPT; ++q) {
        const int64_t t = s + q * BLOCK + threadIdx.x;
        c[q] = t < e ? leaf_col_nt(L, t) : -1;
        if (vals) v[q] = t < e ? __builtin_nontemporal_load(&lv[t]) : (V)0;
    }
}

// Marks the chunk's columns in the bitmap; returns, one bit per element
// slot, the elements that found their column's bit clear (each column's
// first element), and through *count the number of distinct columns.
// (only the columns in [lo, lo + cols) are marked, at c - lo)
template <int BLOCK, int EPT>
GM_DEV uint32_t rank_mark(uint32_t *bits, int nwords, const int32_t (&c)[EPT], int32_t *count, int lo = 0,
                          int cols = INT32_MAX) {
    static_assert(EPT <= 32, "one fresh bit per element slot");
    for (int w = threadIdx.x; w < nwords; w += BLOCK) bits[w] = 0;
    if (threadIdx.x == 0) *count = 0;
    __syncthreads();
    uint32_t fresh = 0;
    int n_fresh = 0;
#pragma unroll
    for (int q = 0; q < EPT; ++q)
        if (c[q] >= 0 && (cols == INT32_MAX || (c[q] >= lo && c[q] - lo < cols))) {
            const int cq = c[q] - lo;
            const int w = cq >> 5;
            const uint32_t bit = 1u << (cq & 31);
            if (!(((volatile uint32_t *)bits)[w] & bit)) {
                const uint32_t old = atomicOr(&bits[w], bit);
                if (!(old & bit)) {
                    fresh |= 1u << q;
                    ++n_fresh;
                }
            }
        }
    n_fresh = wave_reduce_sum(n_fresh);
    if ((threadIdx.x & (GM_WAVE - 1)) == 0 && n_fresh) atomicAdd(count, n_fresh);
    __syncthreads();
    return fresh;
}

// A chunk's column range of (at most) NWORDS * 32 columns is covered in
// PASSES consecutive parts with a bitmap of NWORDS / PASSES words, so a
// 2^18-column range needs 16 KB of LDS instead of 32 KB.

template <int BLOCK, int NWORDS, int EPT, int PASSES = 1>
__global__ __launch_bounds__(BLOCK) void k_leaf_rank_sym(LeafSet L, const LeafTask *tasks, int width,
                                                         int64_t *leaf_nnz, int64_t *slot_cnt) {
    __shared__ uint32_t bits[NWORDS / PASSES];
    __shared__ int32_t count;
    const LeafTask tk = tasks[blockIdx.x];
    int32_t c[EPT];
    float v[EPT];  // not loaded: symbolic
    rank_load<BLOCK, EPT>(L, tk.s, tk.e, c, v, false);
    const int cols = width / PASSES;
    int32_t total = 0;
    if constexpr (PASSES == 1) {
        rank_mark<BLOCK, EPT>(bits, cols >> 5, c, &count);
        total = count;
    } else {
#pragma unroll 1
        for (int p = 0; p < PASSES; ++p) {
            rank_mark<BLOCK, EPT>(bits, cols >> 5, c, &count, p * cols, cols);
            total += count;
            __syncthreads();  // count and bits are reused by the next part
        }
    }
    if (threadIdx.x == 0) {
        leaf_nnz[tk.a] = total;
        slot_cnt[tk.t] = total;
    }
}

// Wide bitmaps keep one rank per group of 8 words instead of one per word
// (a sixteenth of the LDS; an element reads its group's 8 words), so more
// work groups fit a CU.
template <int BLOCK, int NWORDS, int CAP, int EPT, int PASSES, typename CI, typename V>
__global__ __launch_bounds__(BLOCK) void k_leaf_rank_num(LeafSet L, const LeafTask *tasks, int width,
                                                         LeafDst<CI, V> o) {
    constexpr int NWP = NWORDS / PASSES;  // bitmap words of one part
    constexpr bool GROUPED = NWP >= 1024;
    constexpr int NPRE = GROUPED ? NWP / 8 : NWP;
    constexpr int WPT = (NPRE + BLOCK - 1) / BLOCK;  // rank entries per thread in the scan
    __shared__ __align__(16) uint32_t bits[NWP];
    __shared__ uint16_t wpre[NPRE];  // rank of each word's (group's) first set bit (ranks < CAP <= 65535)
    __shared__ V vals[CAP];
    __shared__ int32_t scan_sm[BLOCK / GM_WAVE];
    __shared__ int32_t count;
    const LeafTask tk = tasks[blockIdx.x];
    const int64_t dst = tk.t, nnz = tk.a;
    const CI base = o.base(tk);
    const int cols = width / PASSES;
    const int nwords = cols >> 5;
    const int m = nnz < CAP ? (int)nnz : CAP;  // ranks at or above m are never written (count checked below)
    int32_t c[EPT];
    V v[EPT];
    rank_load<BLOCK, EPT>(L, tk.s, tk.e, c, v, true);
    int32_t done = 0;  // distinct columns of the parts before this one
    auto part = [&](int pass) {
        const int lo = pass * cols;
        const uint32_t fresh = PASSES == 1 ? rank_mark<BLOCK, EPT>(bits, nwords, c, &count)
                                           : rank_mark<BLOCK, EPT>(bits, nwords, c, &count, lo, cols);
        // word (group) ranks: thread t owns entries [t*WPT, t*WPT + WPT)
        {
            const int npre = GROUPED ? nwords / 8 : nwords;
            const int w0 = threadIdx.x * WPT;
            int32_t cnt[WPT], sum = 0;
#pragma unroll
            for (int j = 0; j < WPT; ++j) {
                cnt[j] = 0;
                if (w0 + j < npre) {
                    if (GROUPED) {
                        const uint4 a = *(const uint4 *)&bits[(w0 + j) * 8];
                        const uint4 b = *(const uint4 *)&bits[(w0 + j) * 8 + 4];
                        cnt[j] = __popc(a.x) + __popc(a.y) + __popc(a.z) + __popc(a.w) + __popc(b.x) + __popc(b.y) +
                                 __popc(b.z) + __popc(b.w);
                    } else {
                        cnt[j] = __popc(bits[w0 + j]);
                    }
                }
                sum += cnt[j];
            }
            int32_t r = block_excl_scan<BLOCK>(sum, scan_sm);
#pragma unroll
            for (int j = 0; j < WPT; ++j)
                if (w0 + j < npre) {
                    wpre[w0 + j] = (uint16_t)(r < 65535 ? r : 65535);
                    r += cnt[j];
                }
        }
        if (pass == 0)
            for (int q = threadIdx.x; q < m; q += BLOCK) vals[q] = (V)0;
        __syncthreads();
#pragma unroll
        for (int q = 0; q < EPT; ++q)
            if (c[q] >= 0 && (PASSES == 1 || (c[q] >= lo && c[q] - lo < cols))) {
                const int cq = c[q] - lo;
                const int w = cq >> 5;
                int rk;
                if (GROUPED) {
                    const int g = w >> 3, j0 = w & 7;
                    const uint4 a = *(const uint4 *)&bits[g * 8];
                    const uint4 b = *(const uint4 *)&bits[g * 8 + 4];
                    const uint32_t ws[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
                    rk = wpre[g];
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        rk += __popc(ws[j] & (j < j0 ? ~0u : j == j0 ? (1u << (cq & 31)) - 1u : 0u));
                } else {
                    rk = wpre[w] + __popc(bits[w] & ((1u << (cq & 31)) - 1u));
                }
                rk += done;
                if (rk < m) {
                    __hip_atomic_fetch_add(&vals[rk], v[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                    if ((fresh >> q) & 1u) o.c_col[dst + rk] = base + (CI)c[q];
                }
            }
        done += count;
    };
    if constexpr (PASSES == 1) {
        part(0);
        __syncthreads();  // every value summed before the write-out
    } else {
#pragma unroll
        for (int pass = 0; pass < PASSES; ++pass) {
            part(pass);
            __syncthreads();  // every value of the part summed; bits, wpre and count reused by the next
        }
    }
    if (threadIdx.x == 0 && (done != nnz || done > CAP)) atomicOr(o.err, 4);
    for (int q = threadIdx.x; q < m; q += BLOCK) o.c_val[dst + q] = vals[q];
}

// Small wide chunks (fewer than RANK_MIN_LEN elements, columns too wide for
// a cheap bitmap): the chunk's elements are sorted in LDS by column (one
// bucket pass when they spread evenly, else an LSD radix sort) and the runs
// summed, instead of a hash table followed by a bitonic sort of all its slots.
template <int BLOCK, int CAP, typename CI, typename V>
__global__ __launch_bounds__(BLOCK) void k_leaf_sort_num(LeafSet L, const LeafTask *tasks, int width,
                                                         LeafDst<CI, V> o) {
    static_assert(CAP < 65536, "16-bit element indices");
    __shared__ SortLds<BLOCK, CAP, V> S;
    const int tid = threadIdx.x;
    const LeafTask tk = tasks[blockIdx.x];
    const int64_t len = tk.e - tk.s;
    if (len > CAP) {  // cannot happen for the chunks of this bin (fewer than RANK_MIN_LEN elements)
        if (tid == 0) atomicOr(o.err, 4);
        return;
    }
    const int n = (int)len;
    for (int i = tid; i < n; i += BLOCK) {
        S.keys[0][i] = (uint32_t)leaf_col_nt(L, tk.s + i);
        S.vals[i] = __builtin_nontemporal_load(&static_cast<const V *>(L.val)[tk.s + i]);
        S.idx[0][i] = (uint16_t)i;
    }
    __syncthreads();
    const int bits = width <= 1 ? 0 : 32 - __clz(width - 1);
    uint32_t *keys = S.keys[0], *keys_alt = S.keys[1];
    uint16_t *idx = S.idx[0], *idx_alt = S.idx[1];
    if (!msd_sort_lds<BLOCK, CAP>(keys, idx, keys_alt, idx_alt, n, bits, S.hist, S.scan))
        radix_sort_lds<BLOCK, CAP>(keys, idx, keys_alt, idx_alt, n, bits, S.hist, S.scan);
    sorted_runs_emit<BLOCK, CAP>(keys, idx, idx_alt, (const V *)S.vals, n, tk.a, o.base(tk), o.c_col + tk.t,
                                 o.c_val + tk.t, o.err, 4, S.scan);
}

// Symbolic of the bitmap-rank bins, one wave per chunk: the wave clears its
// own bitmap, reads the chunk's columns with 16-byte loads (aligned blocks,
// elements outside the chunk masked), and counts the columns whose bit it
// set first. Waves do not wait for each other, so a CU keeps up to 32
// chunks' loads in flight (8 with work-group-wide kernels), which is what
// bounds these small, latency-bound chunks.
constexpr int WSYM_U = 2;  // 16-byte blocks per lane per pass

template <int NWORDS, int WAVES, typename ColT>
__global__ __launch_bounds__(WAVES * GM_WAVE) void k_leaf_wave_sym(const ColT *col, const LeafTask *tasks,
                                                                   int64_t n_tasks, int64_t e_end, int64_t *leaf_nnz,
                                                                   int64_t *slot_cnt) {
    static_assert(NWORDS % (4 * GM_WAVE) == 0, "bitmap cleared with 16-byte stores");
    constexpr int PER = 16 / (int)sizeof(ColT);  // elements per 16-byte block
    __shared__ __align__(16) uint32_t bits_all[WAVES][NWORDS];
    const int lane = threadIdx.x & (GM_WAVE - 1), w = threadIdx.x / GM_WAVE;
    const int64_t k = (int64_t)blockIdx.x * WAVES + w;
    if (k >= n_tasks) return;  // the whole wave; no work-group barrier below
    uint32_t *bits = bits_all[w];
    for (int i = lane * 4; i < NWORDS; i += GM_WAVE * 4) *(uint4 *)&bits[i] = make_uint4(0u, 0u, 0u, 0u);
    const LeafTask tk = tasks[k];
    wave_lds_fence();
    int fresh = 0;
    for (int64_t b = (tk.s & ~(int64_t)(PER - 1)) + (int64_t)lane * PER; b < tk.e; b += (int64_t)GM_WAVE * PER * WSYM_U) {
        ColT v[WSYM_U][PER];
#pragma unroll
        for (int u = 0; u < WSYM_U; ++u) {
            const int64_t blk = b + (int64_t)u * GM_WAVE * PER;
            if (blk + PER <= e_end) {
                typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
                const u32x4 q = __builtin_nontemporal_load((const u32x4 *)(col + blk));
                __builtin_memcpy(v[u], &q, 16);
            } else {
#pragma unroll
                for (int j = 0; j < PER; ++j) v[u][j] = blk + j < tk.e ? col[blk + j] : (ColT)0;
            }
        }
#pragma unroll
        for (int u = 0; u < WSYM_U; ++u)
#pragma unroll
            for (int j = 0; j < PER; ++j) {
                const int64_t t = b + (int64_t)u * GM_WAVE * PER + j;
                if (t >= tk.s && t < tk.e) {
                    const int32_t c = (int32_t)v[u][j];
                    const uint32_t bit = 1u << (c & 31);
                    // no return value needed: the distinct count comes from the bitmap
                    __hip_atomic_fetch_or(&bits[c >> 5], bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
                }
            }
    }
    wave_lds_fence();
    for (int i = lane * 4; i < NWORDS; i += GM_WAVE * 4) {
        const uint4 q = *(const uint4 *)&bits[i];
        fresh += __popc(q.x) + __popc(q.y) + __popc(q.z) + __popc(q.w);
    }
    const int32_t n = wave_reduce_sum<int32_t>(fresh);
    if (lane == 0) {
        leaf_nnz[tk.a] = n;
        slot_cnt[tk.t] = n;
    }
}

template <int NWORDS, int WAVES, typename ColT>
void launch_wave_sym(const ColT *col, const LeafTask *tasks, int64_t n, int64_t e_end, int64_t *leaf_nnz,
                     int64_t *slot_cnt, hipStream_t s) {
    if (n <= 0) return;
    const int64_t blocks = (n + WAVES - 1) / WAVES;
    GM_REQUIRE(blocks < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "too many work items for one launch");
    hipLaunchKernelGGL((k_leaf_wave_sym<NWORDS, WAVES, ColT>), dim3((unsigned)blocks), dim3(WAVES * GM_WAVE), 0, s,
                       col, tasks, n, e_end, leaf_nnz, slot_cnt);
    GM_CHECK_LAUNCH();
}

// -------------------------------------------------------------- slot scan
constexpr int SLOT_BLOCK = 256;

__global__ __launch_bounds__(SLOT_BLOCK) void k_slot_scan(int64_t *slot, int64_t n_slots, const int64_t *heavy_rows,
                                                          int64_t *row_nnz) {
    __shared__ int64_t sm[SLOT_BLOCK / GM_WAVE];
    int64_t *p = slot + blockIdx.x * n_slots;
    int64_t carry = 0;
    for (int64_t b = 0; b < n_slots; b += SLOT_BLOCK) {
        const int64_t i = b + threadIdx.x;
        const int64_t x = i < n_slots ? p[i] : 0;
        int64_t tot;
        const int64_t ex = block_excl_scan<SLOT_BLOCK>(x, sm, &tot);
        if (i < n_slots) p[i] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) row_nnz[heavy_rows[blockIdx.x]] = carry;
}

template <class K, class... Args>
void launch_items(K kernel, int block, int64_t n, hipStream_t s, Args... args) {
    if (n <= 0) return;
    GM_REQUIRE(n < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "too many work items for one launch");
    hipLaunchKernelGGL(kernel, dim3((unsigned)n), dim3(block), 0, s, args...);
    GM_CHECK_LAUNCH();
}

}  // namespace

void light_classes_sym(const int64_t *ip, const void *minc, const void *maxc, bool ci64, int64_t n, int64_t tau,
                       bool window, uint8_t *cls, hipStream_t s) {
    light_classes_num(ip, nullptr, minc, maxc, ci64, n, tau, window, cls, s);
}

void light_classes_num(const int64_t *ip, const int64_t *row_nnz, const void *minc, const void *maxc, bool ci64,
                       int64_t n, int64_t tau, bool window, uint8_t *cls, hipStream_t s) {
    if (n <= 0) return;
    with_index_type(ci64, [&](auto ci) {
        using CI = decltype(ci);
        hipLaunchKernelGGL(k_light_classes<CI>, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, ip, row_nnz,
                           static_cast<const CI *>(minc), static_cast<const CI *>(maxc), n, tau, (int)window, cls);
        GM_CHECK_LAUNCH();
    });
}

void leaf_classes_sym(const LeafSet &L, int64_t tau, int64_t width, uint8_t *cls, hipStream_t s) {
    const int64_t n = L.hi - L.lo;
    if (n <= 0) return;
    hipLaunchKernelGGL(k_leaf_classes, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, L, nullptr, tau, width, cls);
    GM_CHECK_LAUNCH();
}

void leaf_classes_num(const LeafSet &L, const int64_t *leaf_nnz, int64_t tau, int64_t width, uint8_t *cls,
                      hipStream_t s) {
    const int64_t n = L.hi - L.lo;
    if (n <= 0) return;
    hipLaunchKernelGGL(k_leaf_classes, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, L, leaf_nnz, tau, width, cls);
    GM_CHECK_LAUNCH();
}

int64_t brow_mask_bytes(const Csr &B) { return B.n_rows * (8 + (B.ci64 ? 8 : 4)); }

void light_symbolic_narrow(const Csr &A, const Csr &B, int64_t r0, const int64_t *items, int64_t n,
                           const void *minc_v, void *masks, int64_t *row_nnz, hipStream_t s) {
    if (n <= 0) return;
    with_index_type(B.ci64, [&](auto ci) {
        using CI = decltype(ci);
        uint64_t *mask = static_cast<uint64_t *>(masks);
        CI *first = reinterpret_cast<CI *>(mask + B.n_rows);
        if (B.n_rows > 0) {
            hipLaunchKernelGGL(k_brow_masks<CI>, dim3(grid_for(B.n_rows, 256, 65536)), dim3(256), 0, s,
                               typed<CI, NoV>(B), mask, first);
            GM_CHECK_LAUNCH();
        }
        hipLaunchKernelGGL(k_light_win0_sym_masks<CI>, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s,
                           typed<CI, NoV>(A), r0, items, n, static_cast<const CI *>(minc_v), mask, first, row_nnz);
        GM_CHECK_LAUNCH();
    });
}

void light_symbolic(const Csr &A, const Csr &B, int64_t r0, int bin, const int64_t *items, int64_t n,
                    const void *minc_v, const void *maxc_v, int64_t *row_nnz, hipStream_t s) {
    with_index_type(B.ci64, [&](auto ci) {
        using CI = decltype(ci);
        const auto a = typed<CI, NoV>(A);
        const auto b = typed<CI, NoV>(B);
        const CI *minc = static_cast<const CI *>(minc_v), *maxc = static_cast<const CI *>(maxc_v);
        switch (bin) {
        case LIGHT_W0:
            launch_items(k_light_win_sym<64, WIN0, CI>, 64, n, s, a, b, r0, items, minc, maxc, row_nnz);
            break;
        case LIGHT_W1:
            launch_items(k_light_win_sym<256, WIN1, CI>, 256, n, s, a, b, r0, items, minc, maxc, row_nnz);
            break;
        case LIGHT_W2:
            launch_items(k_light_win_sym<512, WIN2, CI>, 512, n, s, a, b, r0, items, minc, maxc, row_nnz);
            break;
        case LIGHT_H0:
            launch_items(k_light_hash_sym<64, 2 * HS_CAP[0], CI>, 64, n, s, a, b, r0, items, minc, row_nnz);
            break;
        case LIGHT_H1:
            launch_items(k_light_hash_sym<64, 2 * HS_CAP[1], CI>, 64, n, s, a, b, r0, items, minc, row_nnz);
            break;
        case LIGHT_H2:
            launch_items(k_light_hash_sym<256, 2 * HS_CAP[2], CI>, 256, n, s, a, b, r0, items, minc, row_nnz);
            break;
        case LIGHT_H3:
            launch_items(k_light_hash_sym<512, 2 * HS_CAP[3], CI>, 512, n, s, a, b, r0, items, minc, row_nnz);
            break;
        default: break;
        }
    });
}

void light_numeric(const Csr &A, const Csr &B, int64_t r0, int bin, const int64_t *items, int64_t n,
                   const void *minc_v, const void *maxc_v, const int64_t *c_row_ptr, void *c_col_v, void *c_val_v,
                   int32_t *err, hipStream_t s) {
    with_types(B, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        const auto a = typed<CI, V>(A);
        const auto b = typed<CI, V>(B);
        const CI *minc = static_cast<const CI *>(minc_v), *maxc = static_cast<const CI *>(maxc_v);
        CI *c_col = static_cast<CI *>(c_col_v);
        V *c_val = static_cast<V *>(c_val_v);
        switch (bin) {
        case LIGHT_W0:
            launch_items(k_light_win_num<64, WIN0, CI, V>, 64, n, s, a, b, r0, items, minc, maxc, c_row_ptr, c_col,
                         c_val, err);
            break;
        case LIGHT_W1:
            launch_items(k_light_win_num<256, WIN1, CI, V>, 256, n, s, a, b, r0, items, minc, maxc, c_row_ptr, c_col,
                         c_val, err);
            break;
        case LIGHT_W2:
            launch_items(k_light_win_num<512, WIN2, CI, V>, 512, n, s, a, b, r0, items, minc, maxc, c_row_ptr, c_col,
                         c_val, err);
            break;
        case LIGHT_H0:
            launch_items(k_light_hash_num<64, 256, CI, V>, 64, n, s, a, b, r0, items, minc, c_row_ptr, c_col, c_val,
                         err);
            break;
        case LIGHT_H1:
            launch_items(k_light_sort_num<64, SORT_SMALL[0], CI, V>, 64, n, s, a, b, r0, items, minc, maxc, c_row_ptr,
                         c_col, c_val, err);
            break;
        case LIGHT_H2:
            launch_items(k_light_sort_num<64, SORT_SMALL[1], CI, V>, 64, n, s, a, b, r0, items, minc, maxc, c_row_ptr,
                         c_col, c_val, err);
            break;
        case LIGHT_H3:
            launch_items(k_light_hash_num<64, 1024, CI, V>, 64, n, s, a, b, r0, items, minc, c_row_ptr, c_col, c_val,
                         err);
            break;
        case LIGHT_H4:
            launch_items(k_light_sort_num<256, SORT_CAP[0], CI, V>, 256, n, s, a, b, r0, items, minc, maxc, c_row_ptr,
                         c_col, c_val, err);
            break;
        case LIGHT_H5:
            launch_items(k_light_sort_num<256, SORT_CAP[1], CI, V>, 256, n, s, a, b, r0, items, minc, maxc, c_row_ptr,
                         c_col, c_val, err);
            break;
        case LIGHT_H6:
            launch_items(k_light_sort_num<512, SORT_CAP[2], CI, V>, 512, n, s, a, b, r0, items, minc, maxc, c_row_ptr,
                         c_col, c_val, err);
            break;
        default: break;
        }
    });
}

void leaf_tasks_sym(const LeafSet &L, const int64_t *items, int64_t n, LeafTask *tasks, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_leaf_tasks_sym, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, L, items, n, tasks);
    GM_CHECK_LAUNCH();
}

void leaf_tasks_num(const LeafSet &L, const int64_t *items, int64_t n, const int64_t *leaf_nnz, int n_slots_log2,
                    const int64_t *heavy_rows, const int64_t *c_row_ptr, const int64_t *slot_off,
                    int slot_width_log2, LeafTask *tasks, hipStream_t s) {
    if (n <= 0) return;
    (void)slot_width_log2;
    LeafOut o{n_slots_log2, heavy_rows, c_row_ptr, slot_off};
    hipLaunchKernelGGL(k_leaf_tasks_num, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, L, items, n, leaf_nnz, o,
                       tasks);
    GM_CHECK_LAUNCH();
}

void leaf_symbolic(const LeafSet &L, int bin, const LeafTask *items, int64_t n, int64_t width64, int64_t e_end,
                   int64_t *leaf_nnz, int64_t *slot_cnt, hipStream_t s) {
    // the kernels that read the width (dense and rank shapes) take chunks of at most 2^18 columns
    const int width = (int)(width64 < ((int64_t)1 << 30) ? width64 : ((int64_t)1 << 30));
    const bool rank_bin = bin == LEAF_RANK || bin == LEAF_RANK_L || bin == LEAF_RANK_XL || bin == LEAF_RANK_T;
    const void *colp = L.col16 ? (const void *)L.col16 : (const void *)L.col;
    if (rank_bin && width >= 32 && width <= DENSE_MAX && ((uintptr_t)colp & 15) == 0) {
        // narrow chunks: one wave per chunk, 16-byte column loads (for the
        // wide light chunks of a first level, whose 16 KB bitmaps leave room
        // for 10 waves per CU, the work-group kernels below were faster)
        if (L.col16)
            launch_wave_sym<DENSE_MAX / 32, 4>(L.col16, items, n, e_end, leaf_nnz, slot_cnt, s);
        else
            launch_wave_sym<DENSE_MAX / 32, 4>(L.col, items, n, e_end, leaf_nnz, slot_cnt, s);
        return;
    }
    switch (bin) {
    case LEAF_H0: launch_items(k_leaf_hash_sym<64, 2 * HS_CAP[0]>, 64, n, s, L, items, leaf_nnz, slot_cnt); break;
    case LEAF_H1: launch_items(k_leaf_hash_sym<64, 2 * HS_CAP[1]>, 64, n, s, L, items, leaf_nnz, slot_cnt); break;
    case LEAF_H2: launch_items(k_leaf_hash_sym<256, 2 * HS_CAP[2]>, 256, n, s, L, items, leaf_nnz, slot_cnt); break;
    case LEAF_H3: launch_items(k_leaf_hash_sym<512, 2 * HS_CAP[3]>, 512, n, s, L, items, leaf_nnz, slot_cnt); break;
    case LEAF_DENSE:
        GM_REQUIRE(n <= 0 || width <= DENSE_MAX, GMAGNUS_ERROR_UNSUPPORTED, "dense accumulator wider than LDS allows");
        GM_REQUIRE(((uintptr_t)colp & 15) == 0, GMAGNUS_ERROR_INVALID_VALUE, "column array not 16-byte aligned");
        launch_items(k_leaf_dense_sym<512>, 512, n, s, L, items, width, e_end, leaf_nnz, slot_cnt);
        break;
    case LEAF_RANK_T:
        GM_REQUIRE(n <= 0 || width <= DENSE_MAX, GMAGNUS_ERROR_UNSUPPORTED, "one-wave rank shape is for narrow chunks");
        launch_items(k_leaf_rank_sym<RANK_TBLOCK, RANK_SWORDS, RANK_TEPT>, RANK_TBLOCK, n, s, L, items, width, leaf_nnz,
                     slot_cnt);
        break;
    case LEAF_RANK:
    case LEAF_RANK_L:
    case LEAF_RANK_XL: {
        GM_REQUIRE(n <= 0 || width <= (1 << RANK_MAX_LOG2), GMAGNUS_ERROR_UNSUPPORTED, "rank bitmap too wide");
        constexpr int W17 = (1 << 17) / 32, W18 = (1 << 18) / 32;
        if (width <= DENSE_MAX && bin == LEAF_RANK)
            launch_items(k_leaf_rank_sym<RANK_SBLOCK, RANK_SWORDS, RANK_SEPT>, RANK_SBLOCK, n, s, L, items, width,
                         leaf_nnz, slot_cnt);
        else if (width <= DENSE_MAX && bin == LEAF_RANK_L)
            launch_items(k_leaf_rank_sym<RANK_SBLOCK, RANK_SWORDS, RANK_LEPT>, RANK_SBLOCK, n, s, L, items, width,
                         leaf_nnz, slot_cnt);
        else if (width <= DENSE_MAX)
            launch_items(k_leaf_rank_sym<RANK_XBLOCK, RANK_SWORDS, RANK_LEPT>, RANK_XBLOCK, n, s, L, items, width,
                         leaf_nnz, slot_cnt);
        else if (width <= (1 << 17) && bin == LEAF_RANK)
            launch_items(k_leaf_rank_sym<RANK_WBLOCK, W17, RANK_WEPT>, RANK_WBLOCK, n, s, L, items, width, leaf_nnz,
                         slot_cnt);
        else if (bin == LEAF_RANK)  // 32 KB bitmap: four groups per CU, 8 waves each
            launch_items(k_leaf_rank_sym<2 * RANK_WBLOCK, W18, RANK_WEPT / 2, 1>, 2 * RANK_WBLOCK, n, s, L, items, width,
                         leaf_nnz, slot_cnt);
        else if (width <= (1 << 17))  // 4 waves per work group: 8 of them (chunks) per CU
            launch_items(k_leaf_rank_sym<RANK_LBLOCK, W17, RANK_LWEPT>, RANK_LBLOCK, n, s, L, items, width, leaf_nnz,
                         slot_cnt);
        else  // the 32 KB bitmap leaves four work groups per CU: 8 waves each
            launch_items(k_leaf_rank_sym<RANK_L2BLOCK, W18, RANK_L2EPT, 1>, RANK_L2BLOCK, n, s, L, items, width,
                         leaf_nnz, slot_cnt);
        break;
    }
    default: break;
    }
}

template <typename CI, typename V>
void leaf_numeric_typed(const LeafSet &L, int bin, const LeafTask *items, int64_t n, int width, LeafDst<CI, V> o,
                        int32_t *counter, hipStream_t s) {
    switch (bin) {
    case LEAF_H0:
    case LEAF_H1:
        // bitmap-rank-wide levels send only chunks of fewer than RANK_MIN_LEN elements here
        if (width <= (1 << RANK_MAX_LOG2))
            launch_items(k_leaf_sort_num<64, RANK_MIN_LEN, CI, V>, 64, n, s, L, items, width, o);
        else if (bin == LEAF_H0)
            launch_items(k_leaf_hash_num<64, 256, CI, V>, 64, n, s, L, items, o);
        else
            launch_items(k_leaf_hash_num<64, 1024, CI, V>, 64, n, s, L, items, o);
        break;
    case LEAF_H2: launch_items(k_leaf_hash_num<256, 4096, CI, V>, 256, n, s, L, items, o); break;
    case LEAF_H3: launch_items(k_leaf_hash_num<512, 8192, CI, V>, 512, n, s, L, items, o); break;
    case LEAF_DENSE:
        GM_REQUIRE(n <= 0 || width <= DENSE_MAX, GMAGNUS_ERROR_UNSUPPORTED, "dense accumulator wider than LDS allows");
        if (n > 0) {
            int dev = 0, n_cu = 0;
            GM_HIP(hipGetDevice(&dev));
            GM_HIP(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev));
            fill<int32_t>(counter, 0, 1, s);
            const int64_t groups = std::min<int64_t>(n, (int64_t)n_cu * DENSE_GROUPS_PER_CU);
            hipLaunchKernelGGL((k_leaf_dense_num<DENSE_BLOCK, DENSE_EPT, CI, V>), dim3((unsigned)groups),
                               dim3(DENSE_BLOCK), 0, s, L, items, n, width, o, counter);
            GM_CHECK_LAUNCH();
        }
        break;
    case LEAF_RANK_T:
        GM_REQUIRE(n <= 0 || width <= DENSE_MAX, GMAGNUS_ERROR_UNSUPPORTED, "one-wave rank shape is for narrow chunks");
        launch_items(k_leaf_rank_num<RANK_TBLOCK, RANK_SWORDS, RANK_MIN_LEN, RANK_TEPT, 1, CI, V>, RANK_TBLOCK, n, s, L,
                     items, width, o);
        break;
    case LEAF_RANK:
    case LEAF_RANK_L:
    case LEAF_RANK_XL: {
        GM_REQUIRE(n <= 0 || width <= (1 << RANK_MAX_LOG2), GMAGNUS_ERROR_UNSUPPORTED, "rank bitmap too wide");
        constexpr int W17 = (1 << 17) / 32, W18 = (1 << 18) / 32;
        const bool narrow = width <= (1 << 17);
        if (width <= DENSE_MAX && bin == LEAF_RANK)  // at most RANK_NARROW_SMALL elements
            launch_items(k_leaf_rank_num<RANK_SBLOCK, RANK_SWORDS, RANK_SCAP, RANK_SEPT, 1, CI, V>, RANK_SBLOCK, n, s, L,
                         items, width, o);
        else if (width <= DENSE_MAX && bin == LEAF_RANK_L)  // at most RANK_NARROW_MID elements
            launch_items(k_leaf_rank_num<RANK_SBLOCK, RANK_SWORDS, RANK_NARROW_MID, RANK_LEPT, 1, CI, V>, RANK_SBLOCK,
                         n, s, L, items, width, o);
        else if (width <= DENSE_MAX)  // at most RANK_NARROW_CAP elements
            launch_items(k_leaf_rank_num<RANK_XBLOCK, RANK_SWORDS, RANK_NARROW_CAP, RANK_LEPT, 1, CI, V>, RANK_XBLOCK,
                         n, s, L, items, width, o);
        else if (bin == LEAF_RANK && narrow)  // wide, at most RANK_MID distinct columns
            launch_items(k_leaf_rank_num<RANK_BLOCK, W17, RANK_MID, RANK_EPT, 1, CI, V>, RANK_BLOCK, n, s, L, items,
                         width, o);
        else if (bin == LEAF_RANK)  // 64 KB of LDS: two groups per CU, so 16 waves each
            launch_items(k_leaf_rank_num<RANK_X2BLOCK, W18, RANK_MID, RANK_X2EPT, 1, CI, V>, RANK_X2BLOCK, n, s, L,
                         items, width, o);
        else if (bin != LEAF_RANK_XL && narrow)  // at most RANK_SMALL distinct columns
            launch_items(k_leaf_rank_num<RANK_L2BLOCK, W17, RANK_SMALL, RANK_L2EPT, 1, CI, V>, RANK_L2BLOCK, n, s, L,
                         items, width, o);
        else if (bin != LEAF_RANK_XL)
            launch_items(k_leaf_rank_num<RANK_L2BLOCK, W18, RANK_SMALL, RANK_L2EPT, 1, CI, V>, RANK_L2BLOCK, n, s, L,
                         items, width, o);
        else if (narrow)  // (16 waves were no faster here)
            launch_items(k_leaf_rank_num<RANK_BLOCK, W17, RANK_NNZ_MAX, RANK_EPT, 1, CI, V>, RANK_BLOCK, n, s, L, items,
                         width, o);
        else  // 73 KB of LDS: two groups per CU, 16 waves each
            launch_items(k_leaf_rank_num<RANK_X2BLOCK, W18, RANK_NNZ_MAX, RANK_X2EPT, 2, CI, V>, RANK_X2BLOCK, n, s, L,
                         items, width, o);
        break;
    }
    default: break;
    }
}

void leaf_numeric(const LeafSet &L, int bin, const LeafTask *items, int64_t n, int64_t width64, void *c_col, bool ci64,
                  int slot_width_log2, void *c_val, int32_t *err, int32_t *counter, hipStream_t s) {
    const int width = (int)(width64 < ((int64_t)1 << 30) ? width64 : ((int64_t)1 << 30));
    with_types(ci64, L.v32, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        LeafDst<CI, V> o{static_cast<CI *>(c_col), static_cast<V *>(c_val), err, slot_width_log2};
        leaf_numeric_typed<CI, V>(L, bin, items, n, width, o, counter, s);
    });
}

void slot_scan(int64_t *slot, int64_t n_heavy, int64_t n_slots, const int64_t *heavy_rows, int64_t *row_nnz,
               hipStream_t s) {
    if (n_heavy <= 0) return;
    GM_REQUIRE(n_heavy < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "too many heavy rows for one panel");
    hipLaunchKernelGGL(k_slot_scan, dim3((unsigned)n_heavy), dim3(SLOT_BLOCK), 0, s, slot, n_slots, heavy_rows,
                       row_nnz);
    GM_CHECK_LAUNCH();
}

int64_t tau_limit() {
    int64_t t = HN_CAP[3] < RANK_NNZ_MAX ? HN_CAP[3] : RANK_NNZ_MAX;
    return t < SORT_CAP[2] ? t : SORT_CAP[2];
}

// Rows of more products take the heavy path even when they are below tau:
// one 512-thread group per CU sorting up to 6912 products in LDS is slower
// than expanding and splitting them.
int64_t light_row_limit() { return SORT_CAP[1]; }

}  // namespace gm
