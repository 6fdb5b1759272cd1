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
//   out_ptr[r] + pre[c][e] + j,
//
// where pre[c][e] is the exclusive prefix, over the entries of row h before
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

template <typename CI, typename V>
__global__ void k_heavy_entries(CsrV<CI, V> A, const int64_t *b_rp, const int64_t *heavy_rows, int64_t n_heavy,
                                int64_t r0, const int64_t *a_heavy_ptr, int64_t total, const int32_t *k_to_slice,
                                RowEntries ent) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t h = find_row(a_heavy_ptr, 0, n_heavy + 1, e);
        const int64_t j = A.rp[r0 + heavy_rows[h]] + (e - a_heavy_ptr[h]);
        const int32_t k = (int32_t)A.ci[j];
        ent.k[e] = k;
        ent.s[e] = k_to_slice[k];
        ent.h[e] = (int32_t)h;
        ent.b0[e] = b_rp[k];
        static_cast<V *>(ent.a)[e] = A.v[j];
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

// Offset scan, pass 3: pb[c * n_ent + e] = (exclusive prefix of the chunk-c
// sizes over the earlier entries of e's row, offset of the chunk-c part in
// e's B row). Chunk-major, so the expansion reads consecutive entries of a
// region from consecutive places. Lane = entry: for every chunk a wave takes a
// segmented scan (by row) of its 64 entries' chunk sizes and stores 64
// consecutive pairs. The sums are taken modulo 2^32 (DPP scan): the offsets
// inside one (chunk, row) region are below 2^32, so the stored values are
// exact. Lane c keeps the chunk-c total of the row that is open at the end of
// the group (pass 2's carry at the wave's first row).
GM_DEV uint32_t wave_incl_scan_u32(uint32_t x) {
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);  // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);  // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);  // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);  // row_shr:8
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
    return x;
}

// (NC > 0: the chunk count fixed at compile time, so a lane's chunk bounds
// are read once into registers; NC = 0: any count, read per chunk)
template <int NC>
__global__ __launch_bounds__(256) void k_pre_write(RowEntries ent, int64_t n_ent, const int32_t *bnd, int nc_rt,
                                                   const int64_t *carry, uint2 *pb) {
    const int nc = NC > 0 ? NC : nc_rt;
    const int lane = threadIdx.x & (GM_WAVE - 1);
    const int64_t w = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / GM_WAVE;
    const int64_t e0 = w * PRE_ENTRIES;
    if (e0 >= n_ent) return;  // uniform across the wave
    const int64_t e1 = e0 + PRE_ENTRIES < n_ent ? e0 + PRE_ENTRIES : n_ent;
    uint32_t open = lane < nc ? (uint32_t)carry[w * nc + lane] : 0u;  // lane c: chunk c of the open row
    int32_t hopen = ent.h[e0];                                        // the open row
    const uint64_t le_mask = lanemask_lt() | (uint64_t(1) << lane);
    for (int64_t eb = e0; eb < e1; eb += GM_WAVE) {
        const int cnt = (int)(e1 - eb < GM_WAVE ? e1 - eb : GM_WAVE);
        const bool in = lane < cnt;
        const int64_t e = eb + lane;
        const int32_t h = in ? ent.h[e] : -1;
        const int32_t sl = in ? ent.s[e] : -1;
        const int32_t *bq = bnd + (int64_t)(sl < 0 ? 0 : sl) * (nc + 1);
        const int32_t hp = prev_lane(h, hopen);
        const uint64_t heads = ballot(h != hp);
        const uint64_t mine = heads & le_mask;
        const bool cont = mine == 0;  // no row start at or before this lane: the open row continues
        const int seg0 = cont ? 0 : 63 - __clzll((long long)mine);
        auto chunk = [&](int c, uint32_t lo, uint32_t size) {
            const uint32_t incl = wave_incl_scan_u32(size);
            const uint32_t before = (uint32_t)__shfl((int)incl, seg0 > 0 ? seg0 - 1 : 0, GM_WAVE);
            const uint32_t carry_c = (uint32_t)__builtin_amdgcn_readlane((int)open, c);
            const uint32_t excl = incl - size - (seg0 > 0 ? before : 0u) + (cont ? carry_c : 0u);
            if (in) pb[(int64_t)c * n_ent + e] = make_uint2(excl, lo);
            const uint32_t last = (uint32_t)__builtin_amdgcn_readlane((int)(excl + size), cnt - 1);
            if (lane == c) open = last;
        };
        if constexpr (NC > 0) {
            uint32_t bv[NC + 1];
#pragma unroll
            for (int c = 0; c <= NC; ++c) bv[c] = sl >= 0 ? (uint32_t)bq[c] : 0u;
#pragma unroll
            for (int c = 0; c < NC; ++c) chunk(c, bv[c], bv[c + 1] - bv[c]);
        } else {
            for (int c = 0; c < nc; ++c) {
                uint32_t lo = 0, size = 0;
                if (sl >= 0) {
                    lo = (uint32_t)bq[c];
                    size = (uint32_t)bq[c + 1] - lo;
                }
                chunk(c, lo, size);
            }
        }
        hopen = __builtin_amdgcn_readlane(h, cnt - 1);
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
                          const int32_t *reg_c, const int64_t *reg_efirst, const int64_t *reg_ne, const uint2 *pb,
                          int64_t n_ent, int64_t *region) {
    const int64_t r = find_row(out_ptr, 0, n_out + 1, g);
    const int64_t o = g - out_ptr[r];
    const int c = reg_c[r];
    int64_t lo = reg_efirst[r], hi = lo + reg_ne[r];
    while (hi - lo > 1) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if ((int64_t)pb[(int64_t)c * n_ent + mid].x <= o)
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
                           const int64_t *reg_efirst, const int64_t *reg_ne, const uint2 *pb, int64_t n_ent,
                           int64_t total, int64_t n_tiles, RsTile *info) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n_tiles;
         t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t g0 = t * RS_TILE;
        const int64_t g1 = g0 + RS_TILE < total ? g0 + RS_TILE : total;
        int64_t r0, r1;
        const int64_t s0 = segment_of(g0, out_ptr, n_out, seg_base, reg_c, reg_efirst, reg_ne, pb, n_ent, &r0);
        const int64_t s1 = segment_of(g1 - 1, out_ptr, n_out, seg_base, reg_c, reg_efirst, reg_ne, pb, n_ent, &r1);
        info[t] = RsTile{r0, s0, s1 - s0 + 1};
    }
}

template <typename CI, typename V>
struct RsArgs {
    CsrV<CI, V> B;
    RowEntries ent;
    const uint2 *pb;
    int64_t n_ent;
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
    V *out_val;
};

template <typename CI, typename V>
__global__ __launch_bounds__(RS_BLOCK) void k_expand_rows(RsArgs<CI, V> a) {
    __shared__ int64_t sb[RS_BLOCK + 2];   // seg_base window of the batch's regions
    __shared__ int64_t rn_src[RS_BLOCK];   // compacted non-empty segments: B position minus tile-local index
    __shared__ V rn_a[RS_BLOCK];
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
    const CI mask = (CI)((1u << a.shift) - 1u);
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
        V av = 0;
        if (tid < nb) {
            const int64_t S = sfirst + tid;
            const int64_t r = rb + find_row(sb, 0, nb + 2, S);
            const int c = a.reg_c[r];
            const int64_t e = a.reg_efirst[r] + (S - sb[r - rb]);
            const bool last = S + 1 == sb[r - rb + 1];
            const int64_t start = a.out_ptr[r];
            const uint2 pe = a.pb[(int64_t)c * a.n_ent + e];
            const int64_t seg_g = start + pe.x;
            const int64_t seg_e = last ? a.out_ptr[r + 1] : start + a.pb[(int64_t)c * a.n_ent + e + 1].x;
            const int64_t lo = seg_g > g0 ? seg_g : g0;
            const int64_t hi = seg_e < g1 ? seg_e : g1;
            if (hi > lo) {
                src = a.ent.b0[e] + pe.y + (lo - seg_g);
                av = static_cast<const V *>(a.ent.a)[e];
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
            V bv[RS_ILP], am[RS_ILP];
            // as in the two-level kernel: every load of the thread's products in flight together
            int qs[RS_ILP];
            int64_t sp[RS_ILP];
#pragma unroll
            for (int u = 0; u < RS_ILP; ++u) {
                const int t = tb + u * RS_BLOCK + tid < t1 ? tb + u * RS_BLOCK + tid : t1 - 1;
                const int w = t >> 5, bit = t & 31;
                const uint32_t below = bit == 31 ? ~0u : (2u << bit) - 1u;
                qs[u] = word_pre[w] + __popc(start_bits[w] & below) - 1;
                sp[u] = rn_src[qs[u]] + t;
            }
            CI cb[RS_ILP];
#pragma unroll
            for (int u = 0; u < RS_ILP; ++u) {
                cb[u] = a.B.ci[sp[u]];
                bv[u] = a.B.v[sp[u]];
            }
#pragma unroll
            for (int u = 0; u < RS_ILP; ++u) {
                const bool ok = tb + u * RS_BLOCK + tid < t1;
                col[u] = ok ? (int32_t)(cb[u] & mask) : -1;
                am[u] = rn_a[qs[u]];
                rg[u] = ok ? rn_reg[qs[u]] : -1;
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
                    const int kprev = prev_lane(key, key);
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


// ---------------------------------------------------------------------------
// Two levels in one pass. When the hierarchy has two levels, the heavy
// regions of the first level are not written out: each tile of the
// chunk-major expansion splits its products of heavy regions by the second
// level's chunk in LDS (ranks over the wave's runs of equal keys, one scan,
// one atomic per nonempty (region, chunk) reserving the tile's range in that
// final chunk, a permutation through LDS) and writes them straight into the
// final chunks; products of light regions (themselves final chunks) are
// written at their first-level place. The second level's counts, needed to
// lay out the final chunks beforehand, come from the structure: per slice
// the boundaries of its B row at every fine chunk (first-level chunk times
// second-level chunk), and per heavy row the sum over its entries of their
// fine chunk sizes. The outputs are written with nontemporal stores: they
// are read again only by a later kernel, and keeping them out of the caches
// leaves room for the B rows that the tiles gather (measured: a tile loop
// that gathers from a 170 MB table while streaming its output out runs 15 %
// faster with nontemporal stores).

// Fine boundaries: bndf[s * (nf + 1) + f] = offset in B[k,:] of the first
// column >= f << fshift (f = 0..nf), for the slices whose B row is longer
// than FB_SHORT (the fine counts read the columns of the shorter rows
// instead: at most FB_SHORT reads against nf + 1). One wave per slice; lane i
// searches the boundaries i, i + 64, ... (PER of them), all its searches
// stepping together so their loads overlap (a hub row's searches would
// otherwise be PER dependent chains of about 17 loads each, one after the
// other). Each search starts from its first-level chunk's part of the row
// (the slice's coarse bounds), about five steps shorter than the whole row.
constexpr int FB_SHORT = 64;
// Rows of at most FB_STREAM elements are read once instead: their columns
// (FB_ILP loads per lane in flight) are counted per fine chunk in the wave's
// LDS histogram, one add per run of equal chunks (the row is sorted), and the
// boundaries are the histogram's exclusive scan, written in one coalesced
// pass: about len / (64 * FB_ILP) rounds of loads instead of a dozen
// dependent search steps.
constexpr int FB_STREAM = 4096, FB_ILP = 8, FB_MAXF = 1024, FB_WAVES = 4;

template <int PER, typename CI>
__global__ __launch_bounds__(FB_WAVES * GM_WAVE) void k_fine_bounds(CsrV<CI, NoV> B, const int32_t *slice_k,
                                                                    int64_t n_slices, int nf, int fshift,
                                                                    const int32_t *sbnd, int nc, int32_t *bndf) {
    __shared__ int32_t hist_all[FB_WAVES][FB_MAXF];
    const int lane = threadIdx.x & (GM_WAVE - 1);
    int32_t *hist = hist_all[threadIdx.x / GM_WAVE];
    const int nc1 = nf / nc;
    const int64_t nwaves = (int64_t)gridDim.x * (blockDim.x / GM_WAVE);
    for (int64_t s = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / GM_WAVE; s < n_slices; s += nwaves) {
        const int32_t k = slice_k[s];
        const int64_t b0 = B.rp[k], len = B.rp[k + 1] - b0;
        if (len <= FB_SHORT) continue;
        int32_t *out = bndf + s * (nf + 1);
        const int32_t *cb = sbnd + s * (nc + 1);  // the row's first-level chunk bounds
        const CI *row = B.ci + b0;
        if (len <= FB_STREAM) {  // uniform over the wave
            for (int f = lane; f < nf; f += GM_WAVE) hist[f] = 0;
            wave_lds_fence();
            for (int p0 = 0; p0 < (int)len; p0 += GM_WAVE * FB_ILP) {
                int fc[FB_ILP];
#pragma unroll
                for (int u = 0; u < FB_ILP; ++u) {
                    const int p = p0 + u * GM_WAVE + lane;
                    const int64_t f = p < (int)len ? ((int64_t)row[p] >> fshift) : -1;
                    fc[u] = f < nf ? (int)f : nf - 1;  // (a column past C's width would be invalid input)
                }
#pragma unroll
                for (int u = 0; u < FB_ILP; ++u) {
                    const int fp = prev_lane(fc[u], -2);
                    const uint64_t starts = ballot(fc[u] >= 0 && fc[u] != fp);
                    if (fc[u] >= 0 && ((starts >> lane) & 1)) {
                        const uint64_t above = starts & ~((lanemask_lt() << 1) | 1ull);
                        const int left = (int)len - (p0 + u * GM_WAVE);  // elements of this batch in the row
                        const int end = above ? __ffsll((long long)above) - 1 : (left < GM_WAVE ? left : GM_WAVE);
                        atomicAdd(&hist[fc[u]], end - lane);
                    }
                }
            }
            wave_lds_fence();
            // boundary f = elements in fine chunks below f: lane l scans the
            // counters [l * per, l * per + per), then adds the lanes before it
            const int per = (nf + 1 + GM_WAVE - 1) / GM_WAVE;
            const int f0 = lane * per;
            int32_t tot = 0;
            for (int j = 0; j < per; ++j) {
                const int f = f0 + j;
                if (f < nf) tot += hist[f];
            }
            int32_t run = wave_incl_scan<int32_t>(tot) - tot;
            for (int j = 0; j < per; ++j) {
                const int f = f0 + j;
                if (f <= nf) out[f] = run;
                if (f < nf) run += hist[f];
            }
            wave_lds_fence();  // the counters are read before the next slice clears them
            continue;
        }
        for (int f0 = 0; f0 <= nf; f0 += PER * GM_WAVE) {  // PER boundaries per lane at a time
            int32_t lo[PER], hi[PER];
#pragma unroll
            for (int j = 0; j < PER; ++j) {
                const int f = f0 + lane + j * GM_WAVE;
                // boundary f lies inside its first-level chunk's part of the row
                const int c = f < nf ? f / nc1 : nc;
                lo[j] = f <= nf ? cb[c] : 0;
                hi[j] = f < nf ? cb[c + 1] : lo[j];  // f = nf: the row's end; past nf: empty
            }
            // bit length of the widest range: that many halvings close every search
            int32_t rng = 0;
#pragma unroll
            for (int j = 0; j < PER; ++j) rng = hi[j] - lo[j] > rng ? hi[j] - lo[j] : rng;
            for (int d = GM_WAVE / 2; d >= 1; d >>= 1) {
                const int32_t o = __shfl_xor(rng, d, GM_WAVE);
                rng = o > rng ? o : rng;
            }
            const int steps = 32 - __clz(rng);
            for (int st = 0; st < steps; ++st) {
#pragma unroll
                for (int j = 0; j < PER; ++j) {
                    const int32_t mid = (lo[j] + hi[j]) >> 1;
                    const bool go = lo[j] < hi[j];
                    const CI col = go ? row[mid] : (CI)0;
                    const bool below = (int64_t)col < ((int64_t)(f0 + lane + j * GM_WAVE) << fshift);
                    if (go) {
                        if (below)
                            lo[j] = mid + 1;
                        else
                            hi[j] = mid;
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < PER; ++j)
                if (f0 + lane + j * GM_WAVE <= nf) out[f0 + lane + j * GM_WAVE] = lo[j];
        }
    }
}

// F[h * nf + f] += fine chunk f's products of heavy row h: each work group
// takes FC_ENTRIES consecutive row-ordered entries, thread t owns the fine
// chunks t, t + FC_BLOCK, ... for entries with long B rows (sizes from the
// fine boundaries, loaded for FC_U entries at a time so that their loads are
// in flight together), the waves take turns to histogram the columns of
// short B rows in LDS, and a row's counts are flushed with one atomic per
// nonzero counter when the row changes.
constexpr int FC_BLOCK = 256, FC_ENTRIES = 256, FC_MAXF = 1024, FC_U = 8;

template <typename CI, int FPT>  // FPT: fine chunks per thread, nf <= FPT * FC_BLOCK
__global__ __launch_bounds__(FC_BLOCK) void k_fine_counts(CsrV<CI, NoV> B, RowEntries ent, int64_t n_ent,
                                                          const int32_t *bndf, int nf, int fshift, int64_t *F) {
    static_assert(FPT * FC_BLOCK <= FC_MAXF, "the short rows' counters hold every fine chunk");
    __shared__ int32_t es[FC_ENTRIES], eh[FC_ENTRIES], el[FC_ENTRIES];
    __shared__ int64_t eb[FC_ENTRIES];
    __shared__ int32_t sh[FC_MAXF];  // the current row's counts from short B rows
    const int tid = threadIdx.x, lane = tid & (GM_WAVE - 1);
    const int64_t e0 = blockIdx.x * (int64_t)FC_ENTRIES;
    const int ne = (int)(n_ent - e0 < FC_ENTRIES ? n_ent - e0 : FC_ENTRIES);
    if (tid < ne) {
        const int32_t sl = ent.s[e0 + tid];
        es[tid] = sl;
        eh[tid] = ent.h[e0 + tid];
        int64_t b0 = 0, len = 0;
        if (sl >= 0) {
            const int32_t k = ent.k[e0 + tid];
            b0 = B.rp[k];
            len = B.rp[k + 1] - b0;
        }
        eb[tid] = b0;
        el[tid] = (int32_t)(len < INT32_MAX ? len : INT32_MAX);
    }
    for (int f = tid; f < FC_MAXF; f += FC_BLOCK) sh[f] = 0;
    __syncthreads();
    int64_t acc[FPT];
#pragma unroll
    for (int j = 0; j < FPT; ++j) acc[j] = 0;
    // adds row h's counts to F and clears them (all threads)
    auto flush = [&](int32_t h) {
        __syncthreads();
#pragma unroll
        for (int j = 0; j < FPT; ++j) {
            const int f = tid + j * FC_BLOCK;
            if (f < nf) {
                const int64_t v = acc[j] + sh[f];
                if (v) atomicAdd((unsigned long long *)&F[(int64_t)h * nf + f], (unsigned long long)v);
                sh[f] = 0;
            }
            acc[j] = 0;
        }
        __syncthreads();
    };
    int32_t cur = eh[0];
    for (int i0 = 0; i0 < ne; i0 += FC_U) {
        // the fine boundaries of the long B rows among the next FC_U entries,
        // loaded with no branch between the loads (a slot with nothing to
        // read loads bndf[0] and is dropped), so that they are in flight together
        int32_t lo[FC_U][FPT], hi[FC_U][FPT];
#pragma unroll
        for (int u = 0; u < FC_U; ++u) {
            const int i = i0 + u < ne ? i0 + u : ne - 1;
            const bool lng = es[i] >= 0 && el[i] > FB_SHORT;
            const int32_t *bq = bndf + (int64_t)(lng ? es[i] : 0) * (nf + 1);
#pragma unroll
            for (int j = 0; j < FPT; ++j) {
                const int f = tid + j * FC_BLOCK;
                const bool ok = lng && f < nf;
                lo[u][j] = *(ok ? bq + f : bndf);
                hi[u][j] = *(ok ? bq + f + 1 : bndf);
            }
        }
#pragma unroll
        for (int u = 0; u < FC_U; ++u) {
            const int i = i0 + u;
            if (i >= ne) break;  // uniform
            const int32_t h = eh[i];
            if (h != cur) {  // uniform: flush the row's counts
                flush(cur);
                cur = h;
            }
            const int32_t sl = es[i], len = el[i];
            if (sl < 0 || len == 0) continue;
            if (len > FB_SHORT) {
#pragma unroll
                for (int j = 0; j < FPT; ++j)
                    if (tid + j * FC_BLOCK < nf) acc[j] += hi[u][j] - lo[u][j];
            } else if (tid / GM_WAVE == (i & (FC_BLOCK / GM_WAVE - 1))) {
                // short B rows go to the waves in turn; one lane per element, a
                // run of equal chunks adds its length once
                const int f = lane < len ? (int)(B.ci[eb[i] + lane] >> fshift) : -1;
                const int fp = prev_lane(f, -2);
                const uint64_t starts = ballot(f >= 0 && f != fp);
                if (f >= 0 && ((starts >> lane) & 1)) {
                    const uint64_t above = starts & ~((lanemask_lt() << 1) | 1ull);
                    const int end = above ? __ffsll((long long)above) - 1 : (len < GM_WAVE ? len : GM_WAVE);
                    atomicAdd(&sh[f], end - lane);
                }
            }
        }
    }
    flush(cur);
}

// counts1[r * nc1 + c1] = F[h * nf + c * nc1 + c1] for the heavy regions r of
// the first level (perm: region -> c * n_heavy + h).
__global__ void k_level1_counts(const int64_t *perm, int64_t n_regions, int64_t n_heavy, const int64_t *F, int nf,
                                int nc1, int64_t *counts1) {
    const int64_t n = n_regions * nc1;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / nc1, c1 = i - r * nc1;
        const int64_t x = perm[r];
        const int64_t c = x / n_heavy, h = x - c * n_heavy;
        counts1[i] = F[h * nf + c * nc1 + c1];
    }
}

constexpr int RS2_SUB = 1024;                 // products split per sub-batch
constexpr int RS2_E = RS2_SUB / RS_BLOCK;     // per thread
constexpr int RS2_KMAX = 1024;                // keys: heavy regions per tile times second-level chunks
constexpr int RS2_NW = RS_BLOCK / GM_WAVE;

struct Rs2Layout {
    int whist, key_start, key_delta, col, val, key, total;
};
__host__ __device__ inline Rs2Layout rs2_layout(int K, int vsize) {
    Rs2Layout L;
    int o = 0;
    L.key_delta = o;  o += 8 * K;
    L.val = o;        o += vsize * RS2_SUB;
    L.whist = o;      o += 4 * RS2_NW * K;
    L.key_start = o;  o += 4 * (K + 1);
    L.col = o;        o += 2 * RS2_SUB;  // final chunks' columns: 16 bits
    L.key = o;        o += 2 * RS2_SUB;
    L.total = (o + 15) & ~15;
    return L;
}

template <typename CI, typename V>
struct Rs2Args {
    CsrV<CI, V> B;
    RowEntries ent;
    const uint2 *pb;
    int64_t n_ent;
    const int64_t *out_ptr;  // first level's region pointers
    const int64_t *seg_base;
    const int32_t *reg_c;
    const int64_t *reg_efirst;
    int64_t n_out;
    int64_t n_heavy_out;     // regions [0, n_heavy_out) are split again
    int64_t total;
    int64_t n_tiles;
    const RsTile *info;
    int nc, shift;           // first level
    int nc1, shift1, R;      // second level; heavy regions a tile can touch
    int64_t *cursor1;        // next free place of second-level output row r * nc1 + c1
    int64_t n_out1_elems;    // size of the second level's output
    int32_t *err;            // set when a key or a place falls outside its range (a bug)
    int32_t *out_col0;       // first level (light regions)
    V *out_val0;
    uint16_t *out_col1;      // second level (final chunks: at most 2^16 columns)
    V *out_val1;
};

template <typename CI, typename V>
__global__ __launch_bounds__(RS_BLOCK) void k_expand_rows2(Rs2Args<CI, V> a) {
    __shared__ int64_t sb[RS_BLOCK + 2];
    __shared__ int32_t rn_src[RS_BLOCK];  // B position minus tile-local index (B has fewer than 2^31 entries)
    __shared__ V rn_a[RS_BLOCK];
    __shared__ int32_t rn_reg[RS_BLOCK];   // region minus the tile's first region
    __shared__ uint32_t start_bits[RS_WORDS];
    __shared__ int32_t word_pre[RS_WORDS];
    __shared__ int32_t scan_sm[RS_BLOCK / GM_WAVE];
    __shared__ int32_t range[2];
    __shared__ int64_t next_rb;
    extern __shared__ __align__(16) unsigned char rs2_smem[];

    const int K = a.R * a.nc1;
    const Rs2Layout Lo = rs2_layout(K, (int)sizeof(V));
    int64_t *key_delta = (int64_t *)(rs2_smem + Lo.key_delta);
    V *val_buf = (V *)(rs2_smem + Lo.val);
    int32_t *whist = (int32_t *)(rs2_smem + Lo.whist);
    int32_t *key_start = (int32_t *)(rs2_smem + Lo.key_start);
    uint16_t *col_buf = (uint16_t *)(rs2_smem + Lo.col);
    uint16_t *key_buf = (uint16_t *)(rs2_smem + Lo.key);

    const int tid = threadIdx.x, lane = tid & (GM_WAVE - 1), w = tid / GM_WAVE;
    const int64_t tile = blockIdx.x;  // chunk-major order
    const int64_t g0 = tile * RS_TILE;
    const int64_t g1 = g0 + RS_TILE < a.total ? g0 + RS_TILE : a.total;
    const RsTile ti = a.info[tile];
    const CI mask = (CI)((1u << a.shift) - 1u);
    const int32_t mask1 = (int32_t)((1u << a.shift1) - 1u);
    const int64_t rt = ti.r0;  // keys are (region - rt) * nc1 + second-level chunk
    const bool tile_heavy = rt < a.n_heavy_out;  // uniform over the work group
    const uint64_t le_mask = lanemask_lt() | (uint64_t(1) << lane);
    int32_t *wh = whist + w * K;
    for (int k = tid; k < RS2_NW * K; k += RS_BLOCK) whist[k] = 0;
    int64_t rb = ti.r0;

    for (int64_t b = 0; b < ti.nseg; b += RS_BLOCK) {
        const int nb = (int)(ti.nseg - b < RS_BLOCK ? ti.nseg - b : RS_BLOCK);
        const int64_t sfirst = ti.s0 + b;
        for (int q = tid; q <= nb + 1; q += RS_BLOCK) sb[q] = rb + q <= a.n_out ? a.seg_base[rb + q] : INT64_MAX;
        start_bits[tid] = 0u;
        __syncthreads();
        int32_t loc = -1, len = 0, reg = 0;
        int64_t src = 0;
        V av = 0;
        if (tid < nb) {
            const int64_t S = sfirst + tid;
            const int64_t r = rb + find_row(sb, 0, nb + 2, S);
            const int c = a.reg_c[r];
            const int64_t e = a.reg_efirst[r] + (S - sb[r - rb]);
            const bool last = S + 1 == sb[r - rb + 1];
            const int64_t start = a.out_ptr[r];
            const uint2 pe = a.pb[(int64_t)c * a.n_ent + e];
            const int64_t seg_g = start + pe.x;
            const int64_t seg_e = last ? a.out_ptr[r + 1] : start + a.pb[(int64_t)c * a.n_ent + e + 1].x;
            const int64_t lo = seg_g > g0 ? seg_g : g0;
            const int64_t hi = seg_e < g1 ? seg_e : g1;
            if (hi > lo) {
                src = a.ent.b0[e] + pe.y + (lo - seg_g);
                av = static_cast<const V *>(a.ent.a)[e];
                loc = (int32_t)(lo - g0);
                len = (int32_t)(hi - lo);
                reg = (int32_t)(r - rt);
            }
            if (tid == nb - 1) next_rb = r;
        }
        int n_ne = 0;
        const int slot = block_excl_scan<RS_BLOCK, int>(len > 0 ? 1 : 0, scan_sm, &n_ne);
        if (len > 0) {
            rn_src[slot] = (int32_t)(src - loc);
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
        // sub-batches of RS2_SUB products (uniform trip count: ballots and
        // barriers need the whole work group)
        for (int sbt = t0; sbt < t1; sbt += RS2_SUB) {
            int32_t col[RS2_E];
            V val[RS2_E];
            int key[RS2_E];
            // segments and B positions of the thread's products, then all their
            // loads with no branch in between (past the end a thread re-reads the
            // sub-batch's last product and drops it), so they are in flight together
            int qs[RS2_E];
            int64_t sp[RS2_E];
#pragma unroll
            for (int u = 0; u < RS2_E; ++u) {
                const int t = sbt + u * RS_BLOCK + tid < t1 ? sbt + u * RS_BLOCK + tid : t1 - 1;
                const int wd = t >> 5, bit = t & 31;
                const uint32_t below = bit == 31 ? ~0u : (2u << bit) - 1u;
                qs[u] = word_pre[wd] + __popc(start_bits[wd] & below) - 1;
                sp[u] = rn_src[qs[u]] + t;
            }
            CI cb[RS2_E];
            V bb[RS2_E];
#pragma unroll
            for (int u = 0; u < RS2_E; ++u) {
                cb[u] = a.B.ci[sp[u]];
                bb[u] = a.B.v[sp[u]];
            }
#pragma unroll
            for (int u = 0; u < RS2_E; ++u) {
                key[u] = -1;
                col[u] = 0;
                val[u] = 0;
                if (sbt + u * RS_BLOCK + tid < t1) {
                    const int q = qs[u];
                    col[u] = (int32_t)(cb[u] & mask);
                    val[u] = rn_a[q] * bb[u];
                    const int rl = rn_reg[q];
                    if (rt + rl < a.n_heavy_out) {
                        key[u] = rl * a.nc1 + (col[u] >> a.shift1);
                        if (key[u] >= K) {
                            atomicOr(a.err, 8);
                            key[u] = -1;
                        }
                    } else {
                        key[u] = -2;  // light region: a final chunk of the first level
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < RS2_E; ++u) {
                if (key[u] == -2) {
                    const int64_t d = g0 + sbt + u * RS_BLOCK + tid;
                    __builtin_nontemporal_store(col[u], &a.out_col0[d]);
                    __builtin_nontemporal_store(val[u], &a.out_val0[d]);
                    key[u] = -1;
                }
            }
            // the split: only tiles that hold heavy regions (heavy regions come
            // first, so a tile whose first region is light holds none)
            if (tile_heavy) {
                // ranks inside (wave, key) buckets, one LDS atomic per run of equal keys
                int rank[RS2_E];
#pragma unroll
                for (int u = 0; u < RS2_E; ++u) {
                    const int k = key[u];
                    const int kprev = prev_lane(k, k);
                    // lane 0 always starts a run: its bit is set after the ballot
                    // (the whole wave is active here), which keeps the ballot
                    // a single comparison
                    const uint64_t starts = ballot(k != kprev) | 1ull;
                    const int first = 63 - __clzll((long long)(starts & le_mask));
                    const uint64_t above = starts & ~le_mask;
                    const int rl = (above ? __ffsll((long long)above) - 1 : GM_WAVE) - first;
                    int base = 0;
                    if (k >= 0 && lane == first) base = atomicAdd(&wh[k], rl);
                    base = __shfl(base, first, GM_WAVE);
                    rank[u] = base + (lane - first);
                }
                __syncthreads();
                // exclusive scan over the buckets in (key, wave) order
                {
                    const int M = RS2_NW * K;
                    const int per = (M + RS_BLOCK - 1) / RS_BLOCK;
                    int sum = 0;
                    for (int q = 0; q < per; ++q) {
                        const int idx = tid * per + q;
                        if (idx < M) sum += whist[(idx % RS2_NW) * K + idx / RS2_NW];
                    }
                    int tot = 0;
                    int run = block_excl_scan<RS_BLOCK>(sum, scan_sm, &tot);
                    for (int q = 0; q < per; ++q) {
                        const int idx = tid * per + q;
                        if (idx < M) {
                            const int ad = (idx % RS2_NW) * K + idx / RS2_NW;
                            const int v = whist[ad];
                            whist[ad] = run;
                            if (idx % RS2_NW == 0) key_start[idx / RS2_NW] = run;
                            run += v;
                        }
                    }
                    if (tid == 0) key_start[K] = tot;
                }
                __syncthreads();
                // reserve each key's range in its final chunk
                for (int k = tid; k < K; k += RS_BLOCK) {
                    const int cnt = key_start[k + 1] - key_start[k];
                    if (cnt > 0) {
                        const int64_t row = (rt + k / a.nc1) * a.nc1 + (k % a.nc1);
                        const int64_t d = (int64_t)atomicAdd((unsigned long long *)&a.cursor1[row], (unsigned long long)cnt);
                        key_delta[k] = d - key_start[k];
                    }
                }
#pragma unroll
                for (int u = 0; u < RS2_E; ++u) {
                    if (key[u] >= 0) {
                        const int pos = wh[key[u]] + rank[u];
                        col_buf[pos] = (uint16_t)(col[u] & mask1);
                        val_buf[pos] = val[u];
                        key_buf[pos] = (uint16_t)key[u];
                    }
                }
                __syncthreads();
                const int nh = key_start[K];
                for (int p = tid; p < nh; p += RS_BLOCK) {
                    const int64_t d = key_delta[key_buf[p]] + p;
                    if (d < 0 || d >= a.n_out1_elems) {
                        atomicOr(a.err, 8);
                        continue;
                    }
                    __builtin_nontemporal_store(col_buf[p], &a.out_col1[d]);
                    __builtin_nontemporal_store(val_buf[p], &a.out_val1[d]);
                }
                for (int k = tid; k < RS2_NW * K; k += RS_BLOCK) whist[k] = 0;
                __syncthreads();
            }
        }
        rb = next_rb;
        __syncthreads();
    }
}

}  // namespace

void heavy_entries(const Csr &A, const Csr &B, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
                   const int64_t *a_heavy_ptr, int64_t nnz_heavy_all, const int32_t *k_to_slice, const RowEntries &ent,
                   hipStream_t s) {
    if (n_heavy <= 0 || nnz_heavy_all <= 0) return;
    with_types(A, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        hipLaunchKernelGGL((k_heavy_entries<CI, V>), dim3(grid_for(nnz_heavy_all, 256, 65536)), dim3(256), 0, s,
                           typed<CI, V>(A), B.rp, heavy_rows, n_heavy, r0, a_heavy_ptr, nnz_heavy_all, k_to_slice,
                           ent);
        GM_CHECK_LAUNCH();
    });
}

int64_t entry_offset_waves(int64_t n_ent) { return (n_ent + PRE_ENTRIES - 1) / PRE_ENTRIES; }

void entry_offsets(const RowEntries &ent, int64_t n_ent, const int32_t *bnd, int nc, int64_t *agg, int32_t *wfirst,
                   int32_t *wlast, int64_t *carry, uint2 *pb, hipStream_t s) {
    if (n_ent <= 0) return;
    GM_REQUIRE(nc >= 1 && nc < GM_WAVE, GMAGNUS_ERROR_UNSUPPORTED, "level-0 chunk count must be below 64");
    const int64_t waves = entry_offset_waves(n_ent);
    const unsigned blocks = grid_for(waves, 4, (int64_t)1 << 30);
    hipLaunchKernelGGL(k_pre_agg, dim3(blocks), dim3(256), 0, s, ent, n_ent, bnd, nc, agg, wfirst, wlast);
    GM_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_pre_carry, dim3(nc), dim3(PRE_CARRY_BLOCK), 0, s, agg, wfirst, wlast, waves, nc, carry);
    GM_CHECK_LAUNCH();
    if (nc == 32)
        hipLaunchKernelGGL(k_pre_write<32>, dim3(blocks), dim3(256), 0, s, ent, n_ent, bnd, nc, carry, pb);
    else
        hipLaunchKernelGGL(k_pre_write<0>, dim3(blocks), dim3(256), 0, s, ent, n_ent, bnd, nc, carry, pb);
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

void expand_rows(const Csr &B, const RowEntries &ent, const uint2 *pb, int64_t n_ent, const int64_t *out_ptr,
                 const int64_t *seg_base, const int32_t *reg_c, const int64_t *reg_efirst, const int64_t *reg_ne,
                 int64_t n_out, int64_t n_heavy_out, int64_t total, int nc, int shift, int next_nc, int next_shift,
                 int64_t *next_counts, int64_t *tile_words, int32_t *out_col, void *out_val, hipStream_t s) {
    if (total <= 0) return;
    GM_REQUIRE(nc >= 1 && nc < GM_WAVE && shift >= 0 && shift < 31, GMAGNUS_ERROR_UNSUPPORTED,
               "fused expansion: unsupported first-level chunking");
    GM_REQUIRE(next_counts == nullptr || (next_nc >= 1 && next_nc <= RS_NEXT_MAX), GMAGNUS_ERROR_UNSUPPORTED,
               "fused expansion: unsupported next-level chunking");
    const int64_t n_tiles = (total + RS_TILE - 1) / RS_TILE;
    GM_REQUIRE(n_tiles < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "expansion: too many tiles for one panel");
    RsTile *info = (RsTile *)tile_words;
    hipLaunchKernelGGL(k_rs_tiles, dim3(grid_for(n_tiles, 256, 65536)), dim3(256), 0, s, out_ptr, n_out, seg_base,
                       reg_c, reg_efirst, reg_ne, pb, n_ent, total, n_tiles, info);
    GM_CHECK_LAUNCH();
    with_types(B, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        RsArgs<CI, V> a{typed<CI, V>(B), ent,        pb,          n_ent,       out_ptr, seg_base,
                        reg_c,           reg_efirst, n_out,       n_heavy_out, total,   n_tiles,
                        info,            nc,         shift,       next_nc,     next_shift, next_counts,
                        out_col,         static_cast<V *>(out_val)};
        hipLaunchKernelGGL((k_expand_rows<CI, V>), dim3((unsigned)n_tiles), dim3(RS_BLOCK), 0, s, a);
        GM_CHECK_LAUNCH();
    });
}

// ------------------------------------------------------------ two levels
int64_t fine_bounds_words(int64_t n_slices, int nf) { return n_slices * (nf + 1); }

void fine_bounds(const Csr &B, const int32_t *slice_k, int64_t n_slices, int nf, int fshift, const int32_t *sbnd,
                 int nc, int32_t *bndf, hipStream_t s) {
    if (n_slices <= 0) return;
    GM_REQUIRE(nf >= 1 && nf <= FC_MAXF && nf <= FB_MAXF && (int64_t)B.nnz < ((int64_t)1 << 31),
               GMAGNUS_ERROR_UNSUPPORTED, "fine boundaries: too many fine chunks or B too large");
    GM_REQUIRE(nc >= 1 && nf % nc == 0, GMAGNUS_ERROR_UNSUPPORTED, "fine boundaries: fine chunks must refine the first level");
    // 9 boundaries per lane cover nf = 512 (R-MAT 22's 32 x 16 chunks) in one round
    with_index_type(B.ci64, [&](auto ci) {
        using CI = decltype(ci);
        hipLaunchKernelGGL((k_fine_bounds<9, CI>), dim3(grid_for(n_slices, FB_WAVES, 65536)), dim3(FB_WAVES * GM_WAVE),
                           0, s, typed<CI, NoV>(B), slice_k, n_slices, nf, fshift, sbnd, nc, bndf);
        GM_CHECK_LAUNCH();
    });
}

void fine_counts(const Csr &B, const RowEntries &ent, int64_t n_ent, const int32_t *bndf, int nf, int fshift,
                 int64_t n_heavy, int64_t *F, hipStream_t s) {
    fill<int64_t>(F, 0, n_heavy * nf, s);
    if (n_ent <= 0) return;
    GM_REQUIRE(nf >= 1 && nf <= FC_MAXF, GMAGNUS_ERROR_UNSUPPORTED, "fine counts: too many fine chunks");
    const int64_t blocks = (n_ent + FC_ENTRIES - 1) / FC_ENTRIES;
    GM_REQUIRE(blocks < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "fine counts: too many entries");
    with_index_type(B.ci64, [&](auto ci) {
        using CI = decltype(ci);
        if (nf <= 2 * FC_BLOCK)
            hipLaunchKernelGGL((k_fine_counts<CI, 2>), dim3((unsigned)blocks), dim3(FC_BLOCK), 0, s,
                               typed<CI, NoV>(B), ent, n_ent, bndf, nf, fshift, F);
        else
            hipLaunchKernelGGL((k_fine_counts<CI, FC_MAXF / FC_BLOCK>), dim3((unsigned)blocks), dim3(FC_BLOCK), 0, s,
                               typed<CI, NoV>(B), ent, n_ent, bndf, nf, fshift, F);
        GM_CHECK_LAUNCH();
    });
}

void level1_counts(const int64_t *perm, int64_t n_regions, int64_t n_heavy, const int64_t *F, int nf, int nc1,
                   int64_t *counts1, hipStream_t s) {
    if (n_regions <= 0) return;
    hipLaunchKernelGGL(k_level1_counts, dim3(grid_for(n_regions * nc1, 256, 65536)), dim3(256), 0, s, perm, n_regions,
                       n_heavy, F, nf, nc1, counts1);
    GM_CHECK_LAUNCH();
}

int rows2_regions(int64_t tau) {
    // heavy regions hold more than tau products: a tile meets at most this many
    return (int)((RS_TILE - 1 + tau) / (tau + 1)) + 1;
}

bool rows2_fits(int64_t tau, int nc1, int nf) {
    const int64_t K = (int64_t)rows2_regions(tau) * nc1;
    return K <= RS2_KMAX && nf <= FC_MAXF && nc1 >= 1;
}

void expand_rows2(const Csr &B, const RowEntries &ent, const uint2 *pb, int64_t n_ent,
                  const int64_t *out_ptr, const int64_t *seg_base, const int32_t *reg_c, const int64_t *reg_efirst,
                  const int64_t *reg_ne, int64_t n_out, int64_t n_heavy_out, int64_t total, int nc, int shift,
                  int nc1, int shift1, int64_t tau, int64_t *cursor1, int64_t n_out1_elems, int32_t *err,
                  int64_t *tile_words, int32_t *out_col0, void *out_val0, uint16_t *out_col1, void *out_val1,
                  hipStream_t s) {
    if (total <= 0) return;
    GM_REQUIRE(nc >= 1 && nc < GM_WAVE && shift >= 0 && shift < 31 && shift1 >= 0 && shift1 <= shift && shift1 <= 16,
               GMAGNUS_ERROR_UNSUPPORTED, "two-level expansion: unsupported chunking");
    const int R = rows2_regions(tau);
    const int K = R * nc1;
    GM_REQUIRE(K <= RS2_KMAX && K < 65536, GMAGNUS_ERROR_UNSUPPORTED, "two-level expansion: too many keys");
    GM_REQUIRE((int64_t)B.nnz < ((int64_t)1 << 31), GMAGNUS_ERROR_UNSUPPORTED,
               "two-level expansion: B positions are kept in 32 bits");
    const int64_t n_tiles = (total + RS_TILE - 1) / RS_TILE;
    GM_REQUIRE(n_tiles < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "expansion: too many tiles for one panel");
    RsTile *info = (RsTile *)tile_words;
    hipLaunchKernelGGL(k_rs_tiles, dim3(grid_for(n_tiles, 256, 65536)), dim3(256), 0, s, out_ptr, n_out, seg_base,
                       reg_c, reg_efirst, reg_ne, pb, n_ent, total, n_tiles, info);
    GM_CHECK_LAUNCH();
    with_types(B, [&](auto ci, auto v) {
        using CI = decltype(ci);
        using V = decltype(v);
        const int lds = rs2_layout(K, (int)sizeof(V)).total;
        allow_dynamic_lds((const void *)k_expand_rows2<CI, V>, rs2_layout(RS2_KMAX, (int)sizeof(V)).total);
        Rs2Args<CI, V> a{typed<CI, V>(B), ent,      pb,      n_ent,       out_ptr,  seg_base,
                         reg_c,           reg_efirst, n_out, n_heavy_out, total,    n_tiles,
                         info,            nc,       shift,   nc1,         shift1,   R,
                         cursor1,         n_out1_elems, err, out_col0,    static_cast<V *>(out_val0), out_col1,
                         static_cast<V *>(out_val1)};
        hipLaunchKernelGGL((k_expand_rows2<CI, V>), dim3((unsigned)n_tiles), dim3(RS_BLOCK), lds, s, a);
        GM_CHECK_LAUNCH();
    });
}

}  // namespace gm
