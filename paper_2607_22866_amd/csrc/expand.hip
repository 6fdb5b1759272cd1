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
// contiguous range of slices (B rows reused from that XCD's L2); C-hat is
// written with non-temporal stores (it is read back only by the next pass).
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

__global__ __launch_bounds__(EXP_BLOCK) void k_expand(Csr B, const int64_t *col_ptr, const int64_t *slice_off,
                                                      const int32_t *slice_k, const int32_t *row_h,
                                                      const double *a_val, int64_t n_slices, int64_t total,
                                                      int64_t n_tiles, const TileInfo *info, int64_t *cursor,
                                                      int32_t *chat_col, double *chat_val) {
    __shared__ int64_t cp[EXP_BLOCK + 1];   // col_ptr window of the current batch's slices
    __shared__ int32_t seg_lo[EXP_BLOCK + 1];  // tile-local first product of each segment
    __shared__ int64_t seg_dst[EXP_BLOCK];  // C-hat position minus tile-local index
    __shared__ int64_t seg_src[EXP_BLOCK];  // B position minus tile-local index
    __shared__ double seg_a[EXP_BLOCK];
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
            double bv[EXP_ILP], av[EXP_ILP];
            int64_t d[EXP_ILP];
#pragma unroll
            for (int u = 0; u < EXP_ILP; ++u) {
                const int t = tb + u * EXP_BLOCK;
                if (t < t1) {
                    const int q = (int)find_row(seg_lo, q_prev, nb, t);
                    q_prev = q;
                    const int64_t src = seg_src[q] + t;
                    c[u] = B.ci[src];
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
            int32_t *chat_col, double *chat_val, hipStream_t s) {
    if (total <= 0 || sl.n_slices <= 0) return;
    const int64_t n_tiles = (total + EXP_TILE - 1) / EXP_TILE;
    hipLaunchKernelGGL(k_expand, dim3((unsigned)n_tiles), dim3(EXP_BLOCK), 0, s, B, sl.col_ptr, sl.slice_off,
                       sl.slice_k, sl.row_h, sl.a_val, sl.n_slices, total, n_tiles, (const TileInfo *)info_words,
                       chat_cursor, chat_col, chat_val);
    GM_CHECK_LAUNCH();
}

}  // namespace gm
