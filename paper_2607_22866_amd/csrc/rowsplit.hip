// Expansion fused with the first level's split, in chunk-major row order
// (Section III-B, Algorithm 4, with the level-0 split of Algorithm 5).
//
// The first level's output is laid out chunk-major: region (c, h) holds the
// products of heavy row h whose column falls in level-0 chunk c, regions in
// the order of the heavy/light partition of the (c, h) counts. Inside region
// (c, h) the products are ordered by the row's A~ entries (row order) and,
// per entry e = (h, k), by position in the chunk-c part of B[k,:]. So every
// product has a fixed place:
//
//   out_ptr[r] + pre[e][c] + j,
//
// where pre[e][c] is the exclusive prefix, over the entries of row h before
// e, of their chunk-c part sizes (a segmented scan over the row-ordered
// entries, one lane per chunk). The expansion cuts the output range itself
// into equal tiles: a tile writes one contiguous range of the output with no
// atomics, and reads, per (entry, chunk) segment, a contiguous piece of a B
// row. Concurrent tiles work on one chunk at a time, so the B data in use is
// one chunk's share of the B rows, which the caches can hold.
//
// Since a tile covers at most a few heavy regions, the next level's
// histogram ((region, sub-chunk) counts of the regions that stay heavy) is
// taken in LDS during the write and flushed with one atomic per counter.
#include "host.hpp"

namespace gm {

namespace {

constexpr int RS_BLOCK = 256;
constexpr int64_t RS_TILE = 8192;
constexpr int RS_ILP = 4;
constexpr int RS_WORDS = (int)(RS_TILE / 32);
static_assert(RS_WORDS == RS_BLOCK, "one bitmap word per thread");
constexpr int PRE_ENTRIES = 256;  // entries per wave in the offset scan
constexpr int RS_HREG = 8;        // heavy regions per tile with LDS counters (more go to global atomics)
constexpr int RS_NEXT_MAX = 64;   // next-level chunks

__global__ void k_heavy_entries(Csr A, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
                                const int64_t *a_heavy_ptr, int64_t total, const int32_t *k_to_slice,
                                RowEntries ent) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t h = find_row(a_heavy_ptr, 0, n_heavy + 1, e);
        const int64_t j = A.rp[r0 + heavy_rows[h]] + (e - a_heavy_ptr[h]);
        const int32_t k = A.ci[j];
        ent.k[e] = k;
        ent.s[e] = k_to_slice[k];
        ent.h[e] = (int32_t)h;
        ent.a[e] = A.v[j];
    }
}

// chunk-c size of entry e (0 when its B row is empty)
GM_DEV int32_t entry_chunk_size(const int32_t *bnd, int32_t s, int nc, int c) {
    if (s < 0) return 0;
    const int32_t *bq = bnd + (int64_t)s * (nc + 1);
    return bq[c + 1] - bq[c];
}

// Offset scan, pass 1: per wave of PRE_ENTRIES entries, lane c sums the
// chunk-c sizes of the wave's last row segment; the wave's first and last
// rows are recorded.
__global__ __launch_bounds__(256) void k_pre_agg(RowEntries ent, int64_t n_ent, const int32_t *bnd, int nc,
                                                 int64_t *agg, int32_t *wfirst, int32_t *wlast) {
    const int lane = threadIdx.x & (GM_WAVE - 1);
    const int64_t w = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / GM_WAVE;
    const int64_t e0 = w * PRE_ENTRIES;
    if (e0 >= n_ent) return;  // uniform across the wave
    const int64_t e1 = e0 + PRE_ENTRIES < n_ent ? e0 + PRE_ENTRIES : n_ent;
    int32_t cur = ent.h[e0];
    int64_t acc = 0;
    for (int64_t eb = e0; eb < e1; eb += GM_WAVE) {
        const int64_t e = eb + lane;
        const int32_t hl = e < e1 ? ent.h[e] : -1;
        const int32_t sl = e < e1 ? ent.s[e] : -1;
        const int cnt = (int)(e1 - eb < GM_WAVE ? e1 - eb : GM_WAVE);
        for (int q = 0; q < cnt; ++q) {
            const int32_t hq = __shfl(hl, q, GM_WAVE), sq = __shfl(sl, q, GM_WAVE);
            if (hq != cur) {
                acc = 0;
                cur = hq;
            }
            if (lane < nc) acc += entry_chunk_size(bnd, sq, nc, lane);
        }
    }
    if (lane < nc) agg[w * nc + lane] = acc;
    if (lane == 0) {
        wfirst[w] = ent.h[e0];
        wlast[w] = cur;
    }
}

// Offset scan, pass 2: carry[w][c] = the chunk-c total of the entries of
// wave w's first row that lie in earlier waves. A segmented scan over the
// waves (a row boundary resets it), one work group per chunk: each thread
// scans a contiguous range of waves, thread 0 chains the ranges.
constexpr int PRE_CARRY_BLOCK = 1024;

__global__ __launch_bounds__(PRE_CARRY_BLOCK) void k_pre_carry(const int64_t *agg, const int32_t *wfirst,
                                                               const int32_t *wlast, int64_t n_waves, int nc,
                                                               int64_t *carry) {
    __shared__ int64_t t_val[PRE_CARRY_BLOCK];
    __shared__ int32_t t_reset[PRE_CARRY_BLOCK];
    const int c = blockIdx.x, tid = threadIdx.x;
    const int64_t per = (n_waves + PRE_CARRY_BLOCK - 1) / PRE_CARRY_BLOCK;
    const int64_t w0 = tid * per, w1 = w0 + per < n_waves ? w0 + per : n_waves;
    // X[w]: total of the row that is open at the end of wave w; it restarts
    // at w when w holds a row boundary or its first row starts at w
    int64_t x = 0;
    int any_reset = 0;
    for (int64_t w = w0; w < w1; ++w) {
        const bool reset = wfirst[w] != wlast[w] || w == 0 || wlast[w - 1] != wfirst[w];
        x = agg[w * nc + c] + (reset ? 0 : x);
        any_reset |= reset;
    }
    t_val[tid] = x;
    t_reset[tid] = any_reset || w0 >= w1;
    __syncthreads();
    if (tid == 0) {
        // exclusive chain over the threads' ranges: value entering each range
        int64_t run = 0;
        for (int t = 0; t < PRE_CARRY_BLOCK; ++t) {
            const int64_t v = t_val[t];
            const int r = t_reset[t];
            t_val[t] = run;
            const int64_t t_begin = (int64_t)t * per;
            if (t_begin < n_waves) run = r ? v : run + v;
        }
    }
    __syncthreads();
    x = t_val[tid];  // X of the wave before w0
    for (int64_t w = w0; w < w1; ++w) {
        const bool cont = w > 0 && wlast[w - 1] == wfirst[w];
        carry[w * nc + c] = cont ? x : 0;
        const bool reset = wfirst[w] != wlast[w] || w == 0 || !cont;
        x = agg[w * nc + c] + (reset ? 0 : x);
    }
}

// Offset scan, pass 3: pre[e * nc + c] = exclusive prefix of the chunk-c
// sizes over the earlier entries of e's row.
__global__ __launch_bounds__(256) void k_pre_write(RowEntries ent, int64_t n_ent, const int32_t *bnd, int nc,
                                                   const int64_t *carry, uint32_t *pre) {
    const int lane = threadIdx.x & (GM_WAVE - 1);
    const int64_t w = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / GM_WAVE;
    const int64_t e0 = w * PRE_ENTRIES;
    if (e0 >= n_ent) return;
    const int64_t e1 = e0 + PRE_ENTRIES < n_ent ? e0 + PRE_ENTRIES : n_ent;
    int32_t cur = ent.h[e0];
    int64_t acc = lane < nc ? carry[w * nc + lane] : 0;
    for (int64_t eb = e0; eb < e1; eb += GM_WAVE) {
        const int64_t e = eb + lane;
        const int32_t hl = e < e1 ? ent.h[e] : -1;
        const int32_t sl = e < e1 ? ent.s[e] : -1;
        const int cnt = (int)(e1 - eb < GM_WAVE ? e1 - eb : GM_WAVE);
        for (int q = 0; q < cnt; ++q) {
            const int32_t hq = __shfl(hl, q, GM_WAVE), sq = __shfl(sl, q, GM_WAVE);
            if (hq != cur) {
                acc = 0;
                cur = hq;
            }
            if (lane < nc) {
                pre[(eb + q) * nc + lane] = (uint32_t)acc;
                acc += entry_chunk_size(bnd, sq, nc, lane);
            }
        }
    }
}

// Per output region r (partition order): chunk, first entry of its row and
// number of entries (the row's segments), from the chunk-major index.
__global__ void k_region_records(const int64_t *perm, int64_t n_out, int64_t n_heavy, const int64_t *a_heavy_ptr,
                                 int32_t *reg_c, int64_t *reg_efirst, int64_t *reg_ne) {
    for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < n_out; r += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = perm[r];
        const int64_t h = i % n_heavy;
        reg_c[r] = (int32_t)(i / n_heavy);
        reg_efirst[r] = a_heavy_ptr[h];
        reg_ne[r] = a_heavy_ptr[h + 1] - a_heavy_ptr[h];
    }
}

// Segment of output position g: region r (largest with out_ptr[r] <= g) and
// the entry of r's row whose chunk part holds g (largest e with pre <= g - start).
GM_DEV int64_t segment_of(int64_t g, const int64_t *out_ptr, int64_t n_out, const int64_t *seg_base,
                          const int32_t *reg_c, const int64_t *reg_efirst, const int64_t *reg_ne, const uint32_t *pre,
                          int nc, int64_t *region) {
    const int64_t r = find_row(out_ptr, 0, n_out + 1, g);
    const int64_t o = g - out_ptr[r];
    const int c = reg_c[r];
    int64_t lo = reg_efirst[r], hi = lo + reg_ne[r];
    while (hi - lo > 1) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if ((int64_t)pre[mid * nc + c] <= o)
            lo = mid;
        else
            hi = mid;
    }
    *region = r;
    return seg_base[r] + (lo - reg_efirst[r]);
}

struct RsTile {
    int64_t r0;    // region of the tile's first product
    int64_t s0;    // its first segment
    int64_t nseg;  // segments the tile touches
};

__global__ void k_rs_tiles(const int64_t *out_ptr, int64_t n_out, const int64_t *seg_base, const int32_t *reg_c,
                           const int64_t *reg_efirst, const int64_t *reg_ne, const uint32_t *pre, int nc,
                           int64_t total, int64_t n_tiles, RsTile *info) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n_tiles;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t g0 = t * RS_TILE;
        const int64_t g1 = g0 + RS_TILE < total ? g0 + RS_TILE : total;
        int64_t r0, r1;
        const int64_t s0 = segment_of(g0, out_ptr, n_out, seg_base, reg_c, reg_efirst, reg_ne, pre, nc, &r0);
        const int64_t s1 = segment_of(g1 - 1, out_ptr, n_out, seg_base, reg_c, reg_efirst, reg_ne, pre, nc, &r1);
        info[t] = RsTile{r0, s0, s1 - s0 + 1};
    }
}

struct RsArgs {
    Csr B;
    RowEntries ent;
    const uint32_t *pre;
    const int32_t *bnd;
    const int64_t *out_ptr;
    const int64_t *seg_base;
    const int32_t *reg_c;
    const int64_t *reg_efirst;
    int64_t n_out;
    int64_t n_heavy_out;  // regions [0, n_heavy_out) stay heavy
    int64_t total;
    int64_t n_tiles;
    const RsTile *info;
    int nc, shift;
    int next_nc, next_shift;  // next level (0: none)
    int64_t *next_counts;     // n_heavy_out * next_nc
    int32_t *out_col;
    double *out_val;
};

__global__ __launch_bounds__(RS_BLOCK) void k_expand_rows(RsArgs a) {
    __shared__ int64_t sb[RS_BLOCK + 2];   // seg_base window of the batch's regions
    __shared__ int64_t rn_src[RS_BLOCK];   // compacted non-empty segments: B position minus tile-local index
    __shared__ double rn_a[RS_BLOCK];
    __shared__ int32_t rn_reg[RS_BLOCK];
    __shared__ uint32_t start_bits[RS_WORDS];
    __shared__ int32_t word_pre[RS_WORDS];
    __shared__ int32_t hist[RS_HREG * RS_NEXT_MAX];
    __shared__ int32_t scan_sm[RS_BLOCK / GM_WAVE];
    __shared__ int32_t range[2];
    __shared__ int64_t next_rb;

    const int tid = threadIdx.x, lane = tid & (GM_WAVE - 1);
    const int64_t tile = blockIdx.x;  // chunk-major order: concurrent tiles share one chunk's B data
    const int64_t g0 = tile * RS_TILE;
    const int64_t g1 = g0 + RS_TILE < a.total ? g0 + RS_TILE : a.total;
    const RsTile ti = a.info[tile];
    const int32_t mask = (int32_t)((1u << a.shift) - 1u);
    const bool fuse_next = a.next_counts != nullptr;
    const int64_t hreg0 = ti.r0;  // heavy-region slots are regions hreg0 .. hreg0 + RS_HREG - 1
    if (fuse_next)
        for (int q = tid; q < RS_HREG * a.next_nc; q += RS_BLOCK) hist[q] = 0;
    const uint64_t le_mask = lanemask_lt() | (uint64_t(1) << lane);
    int64_t rb = ti.r0;

    for (int64_t b = 0; b < ti.nseg; b += RS_BLOCK) {
        const int nb = (int)(ti.nseg - b < RS_BLOCK ? ti.nseg - b : RS_BLOCK);
        const int64_t sfirst = ti.s0 + b;
        // every region holds at least one segment and the batch starts in
        // region rb or rb + 1, so its segments lie in regions [rb, rb + nb]
        for (int q = tid; q <= nb + 1; q += RS_BLOCK) sb[q] = rb + q <= a.n_out ? a.seg_base[rb + q] : INT64_MAX;
        start_bits[tid] = 0u;
        __syncthreads();
        int32_t loc = -1, len = 0, reg = -1;
        int64_t src = 0;
        double av = 0.0;
        if (tid < nb) {
            const int64_t S = sfirst + tid;
            const int64_t r = rb + find_row(sb, 0, nb + 2, S);
            const int c = a.reg_c[r];
            const int64_t e = a.reg_efirst[r] + (S - sb[r - rb]);
            const bool last = S + 1 == sb[r - rb + 1];
            const int64_t start = a.out_ptr[r];
            const int64_t seg_g = start + a.pre[e * a.nc + c];
            const int64_t seg_e = last ? a.out_ptr[r + 1] : start + a.pre[(e + 1) * a.nc + c];
            const int64_t lo = seg_g > g0 ? seg_g : g0;
            const int64_t hi = seg_e < g1 ? seg_e : g1;
            if (hi > lo) {
                const int32_t s = a.ent.s[e];
                src = a.B.rp[a.ent.k[e]] + a.bnd[(int64_t)s * (a.nc + 1) + c] + (lo - seg_g);
                av = a.ent.a[e];
                loc = (int32_t)(lo - g0);
                len = (int32_t)(hi - lo);
                reg = (fuse_next && r < a.n_heavy_out) ? (int32_t)(r - hreg0) : -1;
                if (reg >= RS_HREG) reg = RS_HREG + (int32_t)(r - hreg0);  // counted with global atomics
            }
            if (tid == nb - 1) next_rb = r;
        }
        // compact the non-empty segments and mark their first products
        int n_ne = 0;
        const int slot = block_excl_scan<RS_BLOCK, int>(len > 0 ? 1 : 0, scan_sm, &n_ne);
        if (len > 0) {
            rn_src[slot] = src - loc;
            rn_a[slot] = av;
            rn_reg[slot] = reg;
            atomicOr(&start_bits[loc >> 5], 1u << (loc & 31));
            if (slot == 0) range[0] = loc;
            if (slot == n_ne - 1) range[1] = loc + len;
        }
        __syncthreads();
        word_pre[tid] = block_excl_scan<RS_BLOCK, int>(__popc(start_bits[tid]), scan_sm);
        __syncthreads();
        const int t0 = n_ne > 0 ? range[0] : 0, t1 = n_ne > 0 ? range[1] : 0;
        // uniform trip count (ballots below need the whole wave)
        for (int tb = t0; tb < t1; tb += RS_BLOCK * RS_ILP) {
            int32_t col[RS_ILP], rg[RS_ILP];
            double bv[RS_ILP], am[RS_ILP];
#pragma unroll
            for (int u = 0; u < RS_ILP; ++u) {
                const int t = tb + u * RS_BLOCK + tid;
                rg[u] = -1;
                col[u] = -1;
                if (t < t1) {
                    const int w = t >> 5, bit = t & 31;
                    const uint32_t below = bit == 31 ? ~0u : (2u << bit) - 1u;
                    const int q = word_pre[w] + __popc(start_bits[w] & below) - 1;
                    const int64_t sp = rn_src[q] + t;
                    col[u] = a.B.ci[sp] & mask;
                    bv[u] = a.B.v[sp];
                    am[u] = rn_a[q];
                    rg[u] = rn_reg[q];
                }
            }
#pragma unroll
            for (int u = 0; u < RS_ILP; ++u) {
                const int t = tb + u * RS_BLOCK + tid;
                if (t < t1) {
                    a.out_col[g0 + t] = col[u];
                    a.out_val[g0 + t] = am[u] * bv[u];
                }
                if (fuse_next) {
                    // next-level (region, sub-chunk) counts, one LDS atomic per run of equal keys
                    const int key = rg[u] >= 0 ? rg[u] * a.next_nc + (col[u] >> a.next_shift) : -1;
                    const int kprev = __shfl_up(key, 1, GM_WAVE);
                    const uint64_t starts = ballot(lane == 0 || key != kprev);
                    if (key >= 0 && ((starts >> lane) & 1)) {
                        const uint64_t above = starts & ~le_mask;
                        const int n = (above ? __ffsll((long long)above) - 1 : GM_WAVE) - lane;
                        if (rg[u] < RS_HREG)
                            atomicAdd(&hist[key], n);
                        else
                            atomicAdd((unsigned long long *)&a.next_counts[(hreg0 + rg[u] - RS_HREG) * a.next_nc +
                                                                           (col[u] >> a.next_shift)],
                                      (unsigned long long)n);
                    }
                }
            }
        }
        rb = next_rb;
        __syncthreads();
    }
    if (fuse_next) {
        for (int q = tid; q < RS_HREG * a.next_nc; q += RS_BLOCK) {
            const int v = hist[q];
            if (v) {
                const int64_t r = hreg0 + q / a.next_nc;
                atomicAdd((unsigned long long *)&a.next_counts[r * a.next_nc + q % a.next_nc], (unsigned long long)v);
            }
        }
    }
}

}  // namespace

void heavy_entries(const Csr &A, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0, const int64_t *a_heavy_ptr,
                   int64_t nnz_heavy_all, const int32_t *k_to_slice, const RowEntries &ent, hipStream_t s) {
    if (n_heavy <= 0 || nnz_heavy_all <= 0) return;
    hipLaunchKernelGGL(k_heavy_entries, dim3(grid_for(nnz_heavy_all, 256, 65536)), dim3(256), 0, s, A, heavy_rows,
                       n_heavy, r0, a_heavy_ptr, nnz_heavy_all, k_to_slice, ent);
    GM_CHECK_LAUNCH();
}

int64_t entry_offset_waves(int64_t n_ent) { return (n_ent + PRE_ENTRIES - 1) / PRE_ENTRIES; }

void entry_offsets(const RowEntries &ent, int64_t n_ent, const int32_t *bnd, int nc, int64_t *agg, int32_t *wfirst,
                   int32_t *wlast, int64_t *carry, uint32_t *pre, hipStream_t s) {
    if (n_ent <= 0) return;
    GM_REQUIRE(nc >= 1 && nc < GM_WAVE, GMAGNUS_ERROR_UNSUPPORTED, "level-0 chunk count must be below 64");
    const int64_t waves = entry_offset_waves(n_ent);
    const unsigned blocks = grid_for(waves, 4, (int64_t)1 << 30);
    hipLaunchKernelGGL(k_pre_agg, dim3(blocks), dim3(256), 0, s, ent, n_ent, bnd, nc, agg, wfirst, wlast);
    GM_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_pre_carry, dim3(nc), dim3(PRE_CARRY_BLOCK), 0, s, agg, wfirst, wlast, waves, nc, carry);
    GM_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_pre_write, dim3(blocks), dim3(256), 0, s, ent, n_ent, bnd, nc, carry, pre);
    GM_CHECK_LAUNCH();
}

void region_records(const int64_t *perm, int64_t n_out, int64_t n_heavy, const int64_t *a_heavy_ptr, int32_t *reg_c,
                    int64_t *reg_efirst, int64_t *reg_ne, hipStream_t s) {
    if (n_out <= 0) return;
    hipLaunchKernelGGL(k_region_records, dim3(grid_for(n_out, 256, 65536)), dim3(256), 0, s, perm, n_out, n_heavy,
                       a_heavy_ptr, reg_c, reg_efirst, reg_ne);
    GM_CHECK_LAUNCH();
}

int64_t rows_tile_words(int64_t total) {
    static_assert(sizeof(RsTile) == 3 * sizeof(int64_t), "RsTile layout");
    return 3 * ((total + RS_TILE - 1) / RS_TILE);
}

bool rows_next_fits(int next_nc) { return next_nc <= RS_NEXT_MAX; }

void expand_rows(const Csr &B, const RowEntries &ent, const uint32_t *pre, const int32_t *bnd, const int64_t *out_ptr,
                 const int64_t *seg_base, const int32_t *reg_c, const int64_t *reg_efirst, const int64_t *reg_ne,
                 int64_t n_out, int64_t n_heavy_out, int64_t total, int nc, int shift, int next_nc, int next_shift,
                 int64_t *next_counts, int64_t *tile_words, int32_t *out_col, double *out_val, hipStream_t s) {
    if (total <= 0) return;
    GM_REQUIRE(nc >= 1 && nc < GM_WAVE && shift >= 0 && shift < 31, GMAGNUS_ERROR_UNSUPPORTED,
               "fused expansion: unsupported first-level chunking");
    GM_REQUIRE(next_counts == nullptr || (next_nc >= 1 && next_nc <= RS_NEXT_MAX), GMAGNUS_ERROR_UNSUPPORTED,
               "fused expansion: unsupported next-level chunking");
    const int64_t n_tiles = (total + RS_TILE - 1) / RS_TILE;
    GM_REQUIRE(n_tiles < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "expansion: too many tiles for one panel");
    RsTile *info = (RsTile *)tile_words;
    hipLaunchKernelGGL(k_rs_tiles, dim3(grid_for(n_tiles, 256, 65536)), dim3(256), 0, s, out_ptr, n_out, seg_base,
                       reg_c, reg_efirst, reg_ne, pre, nc, total, n_tiles, info);
    GM_CHECK_LAUNCH();
    RsArgs a{B,       ent,  pre,   bnd,   out_ptr,   seg_base,   reg_c,       reg_efirst, n_out,  n_heavy_out,
             total,   n_tiles, info, nc,  shift,     next_nc,    next_shift,  next_counts, out_col, out_val};
    hipLaunchKernelGGL(k_expand_rows, dim3((unsigned)n_tiles), dim3(RS_BLOCK), 0, s, a);
    GM_CHECK_LAUNCH();
}

}  // namespace gm
