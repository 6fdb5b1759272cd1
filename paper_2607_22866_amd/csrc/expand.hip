// Outer-product expansion of the heavy rows into the intermediate matrix
// C-hat (Section III-B, Eq. outer, Algorithm 4).
//
// The flattened product space of all slices (slice s = column k of the
// masked A times row k of B, sliceOffsets = exclusive scan of
// nnz(A~[:,k]) * nnz(B[k,:])) is cut into equal tiles, one per work group,
// so every work group reads and writes the same number of products.
// Within a tile the products form "segments": one per A~ entry, a run of
// consecutive entries of one B row (partial at the tile's two ends, the
// excess of Algorithm 4). Each segment reserves its run in its C-hat row
// with one atomic add on that row's cursor, then the products are written
// with consecutive lanes on consecutive addresses.
//
// gfx950 specifics: per-tile slice lookups are precomputed by a separate,
// fully parallel kernel (no serial binary search at work-group start);
// segments are processed in batches of one per thread with their slice
// pointers staged in LDS; tiles are remapped so each XCD works on a
// contiguous range of slices (B rows reused from that XCD's L2); stores are
// cached, so the L2 merges the partial lines at the edges of short runs.
#include "host.hpp"

namespace gm {

namespace {

constexpr int EXP_BLOCK = 256;
constexpr int64_t EXP_TILE = 8192;
constexpr int EXP_ILP = 4;

struct TileInfo {
    int64_t s0;    // slice containing the tile's first product
    int64_t a0;    // A~ entry of the tile's first product
    int64_t nseg;  // A~ entries (segments) the tile touches
};

__global__ void k_expand_tiles(Csr B, const int64_t *col_ptr, const int64_t *slice_off, const int32_t *slice_k,
                               int64_t n_slices, int64_t total, int64_t n_tiles, TileInfo *info) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n_tiles;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t g0 = t * EXP_TILE;
        const int64_t g1 = g0 + EXP_TILE < total ? g0 + EXP_TILE : total;
        const int64_t s0 = find_row(slice_off, 0, n_slices + 1, g0);
        const int64_t s1 = find_row(slice_off, s0, n_slices + 1, g1 - 1);
        const int32_t k0 = slice_k[s0], k1 = slice_k[s1];
        const int64_t L0 = B.rp[k0 + 1] - B.rp[k0], L1 = B.rp[k1 + 1] - B.rp[k1];
        const int64_t a0 = col_ptr[s0] + (g0 - slice_off[s0]) / L0;
        const int64_t a1 = col_ptr[s1] + (g1 - 1 - slice_off[s1]) / L1;
        info[t] = TileInfo{s0, a0, a1 - a0 + 1};
    }
}

template <typename CI, typename V>
__global__ __launch_bounds__(EXP_BLOCK) void k_expand(CsrV<CI, V> B, const int64_t *col_ptr, const int64_t *slice_off,
                                                      const int32_t *slice_k, const int32_t *row_h,
                                                      const V *a_val, int64_t n_slices, int64_t total,
                                                      int64_t n_tiles, const TileInfo *info, int64_t *cursor,
                                                      int32_t *chat_col, V *chat_val) {
    __shared__ int64_t cp[EXP_BLOCK + 1];   // col_ptr window of the current batch's slices
    __shared__ int32_t seg_lo[EXP_BLOCK + 1];  // tile-local first product of each segment
    __shared__ int64_t seg_dst[EXP_BLOCK];  // C-hat position minus tile-local index
    __shared__ int64_t seg_src[EXP_BLOCK];  // B position minus tile-local index
    __shared__ V seg_a[EXP_BLOCK];
    __shared__ int64_t next_base;

    const int tid = threadIdx.x;
    const int64_t tile = xcd_tile(blockIdx.x, n_tiles);
    const int64_t g0 = tile * EXP_TILE;
    const int64_t g1 = g0 + EXP_TILE < total ? g0 + EXP_TILE : total;
    const TileInfo ti = info[tile];
    int64_t sbase = ti.s0;

    for (int64_t b = 0; b < ti.nseg; b += EXP_BLOCK) {
        const int nb = (int)(ti.nseg - b < EXP_BLOCK ? ti.nseg - b : EXP_BLOCK);
        // The batch's entries lie in slices [sbase, sbase + nb): each slice
        // it touches holds at least one of its nb entries.
        for (int q = tid; q <= nb; q += EXP_BLOCK) cp[q] = sbase + q <= n_slices ? col_ptr[sbase + q] : INT64_MAX;
        __syncthreads();
        if (tid < nb) {
            const int64_t e = ti.a0 + b + tid;
            const int64_t s = sbase + find_row(cp, 0, nb + 1, e);
            const int32_t k = slice_k[s];
            const int64_t bstart = B.rp[k], L = B.rp[k + 1] - bstart;
            const int64_t seg_g = slice_off[s] + (e - cp[s - sbase]) * L;
            const int64_t lo = seg_g > g0 ? seg_g : g0;
            const int64_t hi = seg_g + L < g1 ? seg_g + L : g1;
            const int64_t loc = lo - g0;
            const int64_t dst =
                (int64_t)atomicAdd((unsigned long long *)&cursor[row_h[e]], (unsigned long long)(hi - lo));
            seg_lo[tid] = (int32_t)loc;
            seg_dst[tid] = dst - loc;
            seg_src[tid] = bstart + (lo - seg_g) - loc;
            seg_a[tid] = a_val[e];
            if (tid == nb - 1) {
                seg_lo[nb] = (int32_t)(hi - g0);
                next_base = s;
            }
        }
        __syncthreads();
        const int t0 = seg_lo[0], t1 = seg_lo[nb];
        // EXP_ILP products per thread per pass, all loads issued before any
        // store; the segment of a product is the last one starting at or
        // before it (searched from the previous product's segment)
        int q_prev = 0;
        for (int tb = t0 + tid; tb < t1; tb += EXP_BLOCK * EXP_ILP) {
            int32_t c[EXP_ILP];
            V bv[EXP_ILP], av[EXP_ILP];
            int64_t d[EXP_ILP];
#pragma unroll
            for (int u = 0; u < EXP_ILP; ++u) {
                const int t = tb + u * EXP_BLOCK;
                if (t < t1) {
                    const int q = (int)find_row(seg_lo, q_prev, nb, t);
                    q_prev = q;
                    const int64_t src = seg_src[q] + t;
                    c[u] = (int32_t)B.ci[src];  // C.m < 2^31 on this path
                    bv[u] = B.v[src];
                    av[u] = seg_a[q];
                    d[u] = seg_dst[q] + t;
                }
            }
#pragma unroll
            for (int u = 0; u < EXP_ILP; ++u) {
                if (tb + u * EXP_BLOCK < t1) {
                    chat_col[d[u]] = c[u];
                    chat_val[d[u]] = av[u] * bv[u];
                }
            }
        }
        sbase = next_base;
        __syncthreads();
    }
}

// Expansion fused with the first level's split. The tiles and segments are
// those of k_expand; each segment (one A~ entry times a clipped run of its B
// row) is cut further at the first-level chunk boundaries of that B row
// (bnd: per slice, offsets of the first column of every chunk), giving
// "runs" that all go to one (heavy row, chunk) output row. Runs stay in
// product order (the B row is sorted), so the nonempty runs of a batch tile
// a contiguous range of tile-local products. Each nonempty run reserves its
// range with one atomic add on cursor[h * nc + c] (the output row's next
// free position); the products are written with the chunk-local column.
//
// A product finds its run in constant time: the nonempty runs are
// compacted, their first products are marked in a tile-wide bitmap, and a
// product's run is the number of marks at or before it, minus one (word
// prefix counts plus one popcount), with no per-product search.
constexpr int EXP_WORDS = (int)(EXP_TILE / 32);
static_assert(EXP_WORDS == EXP_BLOCK, "one bitmap word per thread");

template <typename CI, typename V>
__global__ __launch_bounds__(EXP_BLOCK) void k_expand_split(
    CsrV<CI, V> B, const int64_t *col_ptr, const int64_t *slice_off, const int32_t *slice_k, const int32_t *row_h,
    const V *a_val, int64_t n_slices, int64_t total, int64_t n_tiles, const TileInfo *info, const int32_t *bnd,
    int nc, int shift, int64_t *cursor, int32_t *out_col, V *out_val) {
    __shared__ int64_t cp[EXP_BLOCK + 1];
    __shared__ int64_t sg_b[EXP_BLOCK];     // B.rp[k] of the segment's slice
    __shared__ int64_t sg_hc[EXP_BLOCK];    // heavy row * nc
    __shared__ V sg_a[EXP_BLOCK];
    __shared__ int32_t sg_s[EXP_BLOCK];     // slice
    __shared__ int32_t sg_loc[EXP_BLOCK];   // tile-local index of the segment's first product
    __shared__ int32_t sg_off[EXP_BLOCK];   // its offset in the B row
    __shared__ int32_t sg_end[EXP_BLOCK];   // offset one past the segment's last product
    __shared__ int32_t sg_c[EXP_BLOCK];     // chunk of the first product
    __shared__ int32_t run_base[EXP_BLOCK + 1];
    __shared__ int64_t rn_dst[EXP_BLOCK];   // output position minus tile-local index (compacted runs)
    __shared__ int64_t rn_src[EXP_BLOCK];   // B position minus tile-local index
    __shared__ V rn_a[EXP_BLOCK];
    __shared__ uint32_t start_bits[EXP_WORDS];
    __shared__ int32_t word_pre[EXP_WORDS];
    __shared__ int32_t scan_sm[EXP_BLOCK / GM_WAVE];
    __shared__ int32_t range[2];
    __shared__ int64_t next_base;

    const int tid = threadIdx.x;
    const int64_t tile = xcd_tile(blockIdx.x, n_tiles);
    const int64_t g0 = tile * EXP_TILE;
    const int64_t g1 = g0 + EXP_TILE < total ? g0 + EXP_TILE : total;
    const TileInfo ti = info[tile];
    const int32_t mask = (int32_t)((1u << shift) - 1u);
    int64_t sbase = ti.s0;

    for (int64_t b = 0; b < ti.nseg; b += EXP_BLOCK) {
        const int nb = (int)(ti.nseg - b < EXP_BLOCK ? ti.nseg - b : EXP_BLOCK);
        for (int q = tid; q <= nb; q += EXP_BLOCK) cp[q] = sbase + q <= n_slices ? col_ptr[sbase + q] : INT64_MAX;
        __syncthreads();
        int nr = 0;
        if (tid < nb) {
            const int64_t e = ti.a0 + b + tid;
            const int64_t s = sbase + find_row(cp, 0, nb + 1, e);
            const int32_t k = slice_k[s];
            const int64_t bstart = B.rp[k], L = B.rp[k + 1] - bstart;
            const int64_t seg_g = slice_off[s] + (e - cp[s - sbase]) * L;
            const int64_t lo = seg_g > g0 ? seg_g : g0;
            const int64_t hi = seg_g + L < g1 ? seg_g + L : g1;
            const int32_t off0 = (int32_t)(lo - seg_g), off1 = (int32_t)(hi - seg_g);
            const int32_t c0 = (int32_t)(B.ci[bstart + off0] >> shift);
            const int32_t c1 = (int32_t)(B.ci[bstart + off1 - 1] >> shift);
            nr = c1 - c0 + 1;
            sg_b[tid] = bstart;
            sg_hc[tid] = (int64_t)row_h[e] * nc;
            sg_a[tid] = a_val[e];
            sg_s[tid] = (int32_t)s;
            sg_loc[tid] = (int32_t)(lo - g0);
            sg_off[tid] = off0;
            sg_end[tid] = off1;
            sg_c[tid] = c0;
            if (tid == nb - 1) next_base = s;
        }
        int n_runs = 0;
        const int rbase = block_excl_scan<EXP_BLOCK, int>(nr, scan_sm, &n_runs);
        run_base[tid] = rbase;
        if (tid == 0) run_base[EXP_BLOCK] = n_runs;
        __syncthreads();

        for (int rb = 0; rb < n_runs; rb += EXP_BLOCK) {
            const int nrb = n_runs - rb < EXP_BLOCK ? n_runs - rb : EXP_BLOCK;
            start_bits[tid] = 0u;
            int32_t loc = 0, len = 0;
            int64_t dst = 0, src = 0;
            V av = 0;
            if (tid < nrb) {
                const int gr = rb + tid;
                const int q = (int)find_row(run_base, 0, nb, gr);
                const int c = sg_c[q] + (gr - run_base[q]);
                const int32_t *bq = bnd + (int64_t)sg_s[q] * (nc + 1);
                const int32_t b_lo = bq[c], b_hi = bq[c + 1];
                // first and last runs are clipped to the segment; inner runs
                // are whole chunks of the B row (possibly empty)
                const int32_t lo_r = b_lo > sg_off[q] ? b_lo : sg_off[q];
                const int32_t hi_r = b_hi < sg_end[q] ? b_hi : sg_end[q];
                len = hi_r > lo_r ? hi_r - lo_r : 0;
                loc = sg_loc[q] + (lo_r - sg_off[q]);
                if (len > 0)
                    dst = (int64_t)atomicAdd((unsigned long long *)&cursor[sg_hc[q] + c], (unsigned long long)len);
                src = sg_b[q] + lo_r;
                av = sg_a[q];
            }
            // compact the nonempty runs (block_excl_scan synchronizes, so the
            // bitmap is clear before it is marked)
            int n_ne = 0;
            const int slot = block_excl_scan<EXP_BLOCK, int>(len > 0 ? 1 : 0, scan_sm, &n_ne);
            if (len > 0) {
                rn_dst[slot] = dst - loc;
                rn_src[slot] = src - loc;
                rn_a[slot] = av;
                atomicOr(&start_bits[loc >> 5], 1u << (loc & 31));
                if (slot == 0) range[0] = loc;
                if (slot == n_ne - 1) range[1] = loc + len;
            }
            __syncthreads();
            word_pre[tid] = block_excl_scan<EXP_BLOCK, int>(__popc(start_bits[tid]), scan_sm);
            __syncthreads();
            const int t0 = n_ne > 0 ? range[0] : 0, t1 = n_ne > 0 ? range[1] : 0;
            for (int tb = t0 + tid; tb < t1; tb += EXP_BLOCK * EXP_ILP) {
                CI c[EXP_ILP];
                V bv[EXP_ILP], a[EXP_ILP];
                int64_t d[EXP_ILP];
#pragma unroll
                for (int u = 0; u < EXP_ILP; ++u) {
                    const int t = tb + u * EXP_BLOCK;
                    if (t < t1) {
                        const int w = t >> 5, bit = t & 31;
                        const uint32_t below = bit == 31 ? ~0u : (2u << bit) - 1u;
                        const int q = word_pre[w] + __popc(start_bits[w] & below) - 1;
                        const int64_t sp = rn_src[q] + t;
                        c[u] = B.ci[sp];
                        bv[u] = B.v[sp];
                        a[u] = rn_a[q];
                        d[u] = rn_dst[q] + t;
                    }
                }
#pragma unroll
                for (int u = 0; u < EXP_ILP; ++u) {
                    if (tb + u * EXP_BLOCK < t1) {
                        out_col[d[u]] = (int32_t)(c[u] & (CI)mask);
                        out_val[d[u]] = a[u] * bv[u];
                    }
                }
            }
            __syncthreads();
        }
        sbase = next_base;
        __syncthreads();
    }
}

}  // namespace

int64_t expand_tile_words(int64_t total) {
    static_assert(sizeof(TileInfo) == 3 * sizeof(int64_t), "TileInfo layout");
    return 3 * ((total + EXP_TILE - 1) / EXP_TILE);
}

void expand_tiles(const Csr &B, const SliceArrays &sl, int64_t total, int64_t *info_words, hipStream_t s) {
    if (total <= 0 || sl.n_slices <= 0) return;
    const int64_t n_tiles = (total + EXP_TILE - 1) / EXP_TILE;
    GM_REQUIRE(n_tiles < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "expansion: too many tiles for one panel");
    hipLaunchKernelGGL(k_expand_tiles, dim3(grid_for(n_tiles, 256, 65536)), dim3(256), 0, s, B, sl.col_ptr,
                       sl.slice_off, sl.slice_k, sl.n_slices, total, n_tiles, (TileInfo *)info_words);
    GM_CHECK_LAUNCH();
}

void expand(const Csr &B, const SliceArrays &sl, int64_t total, const int64_t *info_words, int64_t *chat_cursor,
            int32_t *chat_col, void *chat_val, hipStream_t s) {
    if (total <= 0 || sl.n_slices <= 0) return;
    GM_REQUIRE(B.n_cols < ((int64_t)1 << 31), GMAGNUS_ERROR_UNSUPPORTED,
               "C-hat row by row holds whole columns: B must have fewer than 2^31 columns");
    const int64_t n_tiles = (total + EXP_TILE - 1) / EXP_TILE;
    with_types(B, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        hipLaunchKernelGGL((k_expand<CI, V>), dim3((unsigned)n_tiles), dim3(EXP_BLOCK), 0, s, typed<CI, V>(B),
                           sl.col_ptr, sl.slice_off, sl.slice_k, sl.row_h, static_cast<const V *>(sl.a_val),
                           sl.n_slices, total, n_tiles, (const TileInfo *)info_words, chat_cursor, chat_col,
                           static_cast<V *>(chat_val));
        GM_CHECK_LAUNCH();
    });
}

void expand_split(const Csr &B, const SliceArrays &sl, int64_t total, const int64_t *info_words, const int32_t *bnd,
                  int nc, int shift, int64_t *cursor, int32_t *out_col, void *out_val, hipStream_t s) {
    if (total <= 0 || sl.n_slices <= 0) return;
    GM_REQUIRE(nc >= 1 && nc < GM_WAVE && shift >= 0 && shift < 31, GMAGNUS_ERROR_UNSUPPORTED,
               "fused expansion: unsupported first-level chunking");
    const int64_t n_tiles = (total + EXP_TILE - 1) / EXP_TILE;
    with_types(B, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        hipLaunchKernelGGL((k_expand_split<CI, V>), dim3((unsigned)n_tiles), dim3(EXP_BLOCK), 0, s, typed<CI, V>(B),
                           sl.col_ptr, sl.slice_off, sl.slice_k, sl.row_h, static_cast<const V *>(sl.a_val),
                           sl.n_slices, total, n_tiles, (const TileInfo *)info_words, bnd, nc, shift, cursor, out_col,
                           static_cast<V *>(out_val));
        GM_CHECK_LAUNCH();
    });
}

}  // namespace gm
