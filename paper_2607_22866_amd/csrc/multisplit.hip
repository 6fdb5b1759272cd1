// Hierarchical multisplit of the heavy rows (Section III-C, Algorithm 3's
// reorder loop, Algorithm 5): per level a histogram of (row, chunk) counts,
// the heavy/light chunk partition (ThreshPartition, heavy chunks first) and
// the multisplit that permutes every row of C-hat into its column chunks,
// with columns shifted into the chunk's local range.
//
// gfx950 design of the multisplit work group (one tile of consecutive
// elements, at most `group_rows` rows since every input row holds more than
// tau elements):
//  * elements are loaded coalesced into registers, E per thread;
//  * each element's rank inside its (wave, key) bucket comes from wave64
//    ballots (the lanes holding the same key form a peer mask; rank =
//    popcount of lower peers), accumulated in wave-private LDS counters, so
//    no LDS atomics are needed and the local order is stable;
//  * one scan over the (key, wave) counters gives every bucket its local
//    offset; one global atomic per nonempty key reserves its output range;
//  * elements are permuted through LDS and written back with consecutive
//    lanes on consecutive addresses of each output chunk;
//  * the next level's (chunk, sub-chunk) histogram is accumulated during the
//    write-out for the chunks that stay heavy, so levels after the first need
//    no separate histogram pass.
#include "host.hpp"

namespace gm {

namespace {

constexpr int MS_KMAX = 1024;     // keys = group_rows * n_chunks (powers of two)
constexpr int MS_RMAX = 16;       // rows per tile
constexpr int MS_NEXT_MAX = 64;   // next-level chunks for the fused histogram

// Row containing the first element of every tile.
__global__ void k_tile_rows(const int64_t *in_ptr, int64_t n_in, int64_t te, int64_t n_tiles, int64_t *tile_row) {
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n_tiles;
         t += (int64_t)gridDim.x * blockDim.x)
        tile_row[t] = find_row(in_ptr, 0, n_in + 1, t * te);
}

GM_DEV int local_row(const int64_t *rb, int R, int64_t i) {
    int lr = 0;
    while (lr + 1 < R && rb[lr + 1] <= i) ++lr;
    return lr;
}

// Histogram of a level's input (Algorithm 3, Histogram): counts[r * n_chunks
// + c] = number of elements of row r with column >> shift == c. Rows are
// made of sorted B-row runs, so equal keys come in runs over consecutive
// lanes: the first lane of each run adds the run's length with one LDS
// atomic (no same-address atomics within a wave). Tiles are larger than the
// multisplit's (the work group keeps only R * n_chunks counters).
constexpr int HIST_BLOCK = 256;
constexpr int HIST_ILP = 4;
constexpr int HIST_NTILES = 6;
constexpr int64_t HIST_TILES[HIST_NTILES] = {16384, 8192, 4096, 2048, 1024, 512};

__global__ __launch_bounds__(HIST_BLOCK) void k_histogram(int64_t n_in, int64_t elems, const int64_t *in_ptr,
                                                          const int64_t *tile_row, int64_t te, int64_t n_tiles,
                                                          const int32_t *in_col, int n_chunks, int shift, int R,
                                                          int64_t *counts) {
    __shared__ int32_t cnt[MS_KMAX];
    __shared__ int64_t rb[MS_RMAX + 1];
    const int tid = threadIdx.x, lane = tid & (GM_WAVE - 1);
    const int64_t tile = xcd_tile(blockIdx.x, n_tiles);
    const int64_t g0 = tile * te;
    const int64_t g1 = g0 + te < elems ? g0 + te : elems;
    const int64_t r0 = tile_row[tile];
    const int K = R * n_chunks;
    if (tid <= R) rb[tid] = r0 + tid <= n_in ? in_ptr[r0 + tid] : INT64_MAX;
    for (int k = tid; k < K; k += HIST_BLOCK) cnt[k] = 0;
    __syncthreads();
    const uint64_t le_mask = lanemask_lt() | (uint64_t(1) << lane);
    // every lane runs the same iterations (ballots need the whole wave)
    for (int64_t pb = g0; pb < g1; pb += HIST_BLOCK * HIST_ILP) {
        int32_t c[HIST_ILP];
#pragma unroll
        for (int u = 0; u < HIST_ILP; ++u) {
            const int64_t p = pb + u * HIST_BLOCK + tid;
            c[u] = p < g1 ? __builtin_nontemporal_load(&in_col[p]) : -1;
        }
#pragma unroll
        for (int u = 0; u < HIST_ILP; ++u) {
            const int64_t p = pb + u * HIST_BLOCK + tid;
            const int k = c[u] >= 0 ? local_row(rb, R, p) * n_chunks + (c[u] >> shift) : -1;
            const int kprev = prev_lane(k, k);
            const uint64_t starts = ballot(lane == 0 || k != kprev);
            if (k >= 0 && ((starts >> lane) & 1)) {
                const uint64_t above = starts & ~le_mask;
                const int len = (above ? __ffsll((long long)above) - 1 : GM_WAVE) - lane;
                atomicAdd(&cnt[k], len);
            }
        }
    }
    __syncthreads();
    for (int k = tid; k < K; k += HIST_BLOCK) {
        const int v = cnt[k];
        if (v) atomicAdd((unsigned long long *)&counts[(r0 + k / n_chunks) * n_chunks + k % n_chunks],
                         (unsigned long long)v);
    }
}

// Tile of the histogram pass: the largest whose rows fit the counters.
struct HistTile {
    int64_t te;
    int R;
};
HistTile hist_tile(const LevelGeom &g, int64_t tau) {
    for (int i = 0; i < HIST_NTILES; ++i) {
        const int64_t te = HIST_TILES[i];
        const int R = (int)ceil_pow2((te - 1 + tau - 1) / tau + 1);  // input rows hold more than tau elements
        if (R <= MS_RMAX && R * g.n_chunks <= MS_KMAX) return HistTile{te, R};
    }
    throw Error{GMAGNUS_ERROR_UNSUPPORTED, "histogram: tau too small for its tile sizes"};
}

// Dynamic LDS layout of one multisplit work group (byte offsets); the
// arrays whose size depends on the level (keys, next-level histogram) are
// sized exactly, so small levels leave room for more work groups per CU.
struct MsLayout {
    int val, key_delta, key_out, rb, col, whist, key_start, next_hist, scan, total;
};

__host__ __device__ inline MsLayout ms_layout(int te, int nw, int K, int next, int R) {
    MsLayout L;
    int o = 0;
    L.val = o;        o += 8 * te;
    L.key_delta = o;  o += 8 * K;
    L.key_out = o;    o += 8 * K;
    L.rb = o;         o += 8 * (R + 1);
    L.col = o;        o += 4 * te;
    L.whist = o;      o += 4 * nw * K;
    L.key_start = o;  o += 4 * (K + 1);
    L.next_hist = o;  o += 4 * K * next;
    L.scan = o;       o += 4 * nw;
    L.total = o;
    return L;
}

// (the value buffer keeps 8 bytes per element for either value type)
template <int BLOCK, int TE, typename V>
__global__ __launch_bounds__(BLOCK) void k_multisplit(int64_t n_in, int64_t elems, const int64_t *in_ptr,
                                                      const int64_t *tile_row, int64_t n_tiles,
                                                      const int32_t *in_col, const V *in_val, int n_chunks,
                                                      int cbits, int shift, int R, int rbits, const int64_t *x_map,
                                                      int64_t *cursor, int32_t *out_col, V *out_val,
                                                      int64_t n_heavy_out, int next_chunks, int next_shift,
                                                      int64_t *next_counts) {
    constexpr int NW = BLOCK / GM_WAVE;
    constexpr int E = TE / BLOCK;
    extern __shared__ __align__(16) unsigned char ms_smem[];
    const int K = R << cbits;
    const bool fuse_next = next_counts != nullptr;
    const MsLayout Lo = ms_layout(TE, NW, K, fuse_next ? next_chunks : 0, R);
    V *val_buf = (V *)(ms_smem + Lo.val);
    int64_t *key_delta = (int64_t *)(ms_smem + Lo.key_delta);  // global position - local position
    int64_t *key_out = (int64_t *)(ms_smem + Lo.key_out);      // output chunk row
    int64_t *rb = (int64_t *)(ms_smem + Lo.rb);
    int32_t *col_buf = (int32_t *)(ms_smem + Lo.col);
    int32_t *whist = (int32_t *)(ms_smem + Lo.whist);  // [wave][key] counts, then offsets
    int32_t *key_start = (int32_t *)(ms_smem + Lo.key_start);
    int32_t *next_hist = (int32_t *)(ms_smem + Lo.next_hist);
    int32_t *scan_sm = (int32_t *)(ms_smem + Lo.scan);

    const int tid = threadIdx.x, lane = tid & (GM_WAVE - 1), w = tid / GM_WAVE;
    const int64_t tile = xcd_tile(blockIdx.x, n_tiles);
    const int64_t g0 = tile * (int64_t)TE;
    const int n = (int)(elems - g0 < TE ? elems - g0 : TE);
    const int64_t r0 = tile_row[tile];
    const int32_t mask = (int32_t)((1u << shift) - 1u);
    (void)rbits;

    if (tid <= R) rb[tid] = r0 + tid <= n_in ? in_ptr[r0 + tid] : INT64_MAX;
    for (int k = tid; k < NW * K; k += BLOCK) whist[k] = 0;
    if (fuse_next)
        for (int q = tid; q < K * next_chunks; q += BLOCK) next_hist[q] = 0;
    __syncthreads();

    int32_t col[E];
    V val[E];
    int key[E];
    int rank[E];
#pragma unroll
    for (int j = 0; j < E; ++j) {
        const int p = j * BLOCK + tid;
        const bool valid = p < n;
        col[j] = valid ? __builtin_nontemporal_load(&in_col[g0 + p]) : 0;
        val[j] = valid ? __builtin_nontemporal_load(&in_val[g0 + p]) : (V)0;
        key[j] = valid ? (local_row(rb, R, g0 + p) << cbits) | (col[j] >> shift) : -1;
    }
    // Ranks inside (wave, key) buckets. Rows of C-hat are made of sorted B-row
    // segments, so equal keys come in runs over consecutive lanes: each run's
    // first lane reserves the run's length in the wave-private counter with
    // one LDS atomic and the run's lanes take consecutive ranks. The next
    // level's (key, sub-chunk) counts are taken the same way, per run.
    int32_t *wh = whist + w * K;
    const uint64_t le_mask = lanemask_lt() | (uint64_t(1) << lane);
#pragma unroll
    for (int j = 0; j < E; ++j) {
        const int k = key[j];
        const int kprev = prev_lane(k, k);
        const uint64_t starts = ballot(lane == 0 || k != kprev);
        const int first = 63 - __clzll((long long)(starts & le_mask));
        const uint64_t above = starts & ~le_mask;
        const int len = (above ? __ffsll((long long)above) - 1 : GM_WAVE) - first;
        int base = 0;
        if (k >= 0 && lane == first) base = atomicAdd(&wh[k], len);
        base = __shfl(base, first, GM_WAVE);
        rank[j] = base + (lane - first);
        if (fuse_next) {
            const int k2 = k >= 0 ? k * next_chunks + ((col[j] & mask) >> next_shift) : -1;
            const int k2prev = prev_lane(k2, k2);
            const uint64_t s2 = ballot(lane == 0 || k2 != k2prev);
            const uint64_t a2 = s2 & ~le_mask;
            if (k2 >= 0 && ((s2 >> lane) & 1)) {
                const int len2 = (a2 ? __ffsll((long long)a2) - 1 : GM_WAVE) - lane;
                atomicAdd(&next_hist[k2], len2);
            }
        }
    }
    __syncthreads();

    // exclusive scan over buckets in (key, wave) order
    {
        const int M = NW * K;
        const int per = (M + BLOCK - 1) / BLOCK;
        int sum = 0;
        for (int q = 0; q < per; ++q) {
            const int idx = tid * per + q;
            if (idx < M) sum += whist[(idx % NW) * K + idx / NW];
        }
        int run = block_excl_scan<BLOCK>(sum, scan_sm);
        for (int q = 0; q < per; ++q) {
            const int idx = tid * per + q;
            if (idx < M) {
                const int a = (idx % NW) * K + idx / NW;
                const int v = whist[a];
                whist[a] = run;
                if (idx % NW == 0) key_start[idx / NW] = run;
                run += v;
            }
        }
        if (tid == 0) key_start[K] = n;
    }
    __syncthreads();

    // reserve each key's range in its output chunk
    for (int k = tid; k < K; k += BLOCK) {
        const int cnt = key_start[k + 1] - key_start[k];
        if (cnt > 0) {
            const int64_t r = r0 + (k >> cbits);
            const int64_t orow = x_map[r * n_chunks + (k & (n_chunks - 1))];
            const int64_t d = (int64_t)atomicAdd((unsigned long long *)&cursor[orow], (unsigned long long)cnt);
            key_delta[k] = d - key_start[k];
            key_out[k] = orow;
        }
    }
    // permute into LDS
#pragma unroll
    for (int j = 0; j < E; ++j) {
        if (key[j] >= 0) {
            const int pos = wh[key[j]] + rank[j];
            col_buf[pos] = col[j];
            val_buf[pos] = val[j];
        }
    }
    __syncthreads();

    // coalesced write-out; the local row of position p is the last row whose
    // first key starts at or before p
    for (int p = tid; p < n; p += BLOCK) {
        const int32_t c = col_buf[p];
        int lr = 0;
        while (lr + 1 < R && key_start[(lr + 1) << cbits] <= p) ++lr;
        const int k = (lr << cbits) | (c >> shift);
        const int64_t d = key_delta[k] + p;
        const int32_t lc = c & mask;
        out_col[d] = lc;  // cached stores: the L2 merges the partial lines at chunk-run edges
        out_val[d] = val_buf[p];
    }
    if (fuse_next) {
        // counts of the chunks that stay heavy go to the next level
        for (int q = tid; q < K * next_chunks; q += BLOCK) {
            const int v = next_hist[q];
            const int k = q / next_chunks;
            if (v && key_out[k] < n_heavy_out) {
                atomicAdd((unsigned long long *)&next_counts[key_out[k] * next_chunks + q % next_chunks],
                          (unsigned long long)v);
            }
        }
    }
}

__global__ void k_chunk_classes(const int64_t *counts, int64_t n, int64_t tau, int last, uint8_t *cls) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        cls[i] = (!last && counts[i] > tau) ? 0 : 1;
}

__global__ void k_chunk_reorder(const int64_t *counts, const int64_t *inv, int64_t n, int n_chunks,
                                const int64_t *origin_in, int64_t stride, int64_t cmajor_rows, int64_t *out_cnt,
                                int64_t *origin_out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t o = inv[i];
        const int64_t h = cmajor_rows ? i % cmajor_rows : i / n_chunks;
        const int64_t c = cmajor_rows ? i / cmajor_rows : i % n_chunks;
        out_cnt[o] = counts[i];
        origin_out[o] = origin_in[h] + c * stride;
    }
}

constexpr int MS_NTILES = 4;
constexpr int64_t MS_TILES[MS_NTILES] = {2048, 4096, 1024, 512};
constexpr int MS_LDS_MAX = 160 * 1024;

template <int BLOCK, int TE>
int ms_lds_bytes(int K, int next, int R) {
    return ms_layout(TE, BLOCK / GM_WAVE, K, next, R).total;
}

template <int BLOCK, int TE, typename V>
void launch_multisplit(const LevelGeom &g, const int64_t *in_ptr, const int64_t *tile_row, const int32_t *in_col,
                       const V *in_val, const int64_t *x_map, int64_t *cursor, int32_t *out_col,
                       V *out_val, int64_t n_heavy_out, int64_t *next_counts, int cbits, int rbits,
                       hipStream_t s) {
    const int64_t n_tiles = (g.elems + TE - 1) / TE;
    GM_REQUIRE(n_tiles < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "multisplit: too many tiles");
    const int K = g.group_rows << cbits;
    const int lds = ms_lds_bytes<BLOCK, TE>(K, next_counts ? g.next_chunks : 0, g.group_rows);
    GM_REQUIRE(lds <= MS_LDS_MAX, GMAGNUS_ERROR_UNSUPPORTED, "multisplit: work-group LDS above 160 KB");
    allow_dynamic_lds((const void *)k_multisplit<BLOCK, TE, V>, MS_LDS_MAX);
    hipLaunchKernelGGL((k_multisplit<BLOCK, TE, V>), dim3((unsigned)n_tiles), dim3(BLOCK), lds, s, g.n_in, g.elems,
                       in_ptr, tile_row, n_tiles, in_col, in_val, g.n_chunks, cbits, g.shift, g.group_rows, rbits,
                       x_map, cursor, out_col, out_val, n_heavy_out, g.next_chunks, g.next_shift, next_counts);
    GM_CHECK_LAUNCH();
}

}  // namespace

int multisplit_tile_count() { return MS_NTILES; }
int64_t multisplit_tile_elems(int i) { return MS_TILES[i]; }
int multisplit_max_keys() { return MS_KMAX; }
int multisplit_max_rows() { return MS_RMAX; }
bool multisplit_next_fits(int keys, int next_chunks) {
    return next_chunks <= MS_NEXT_MAX && 4 * keys * next_chunks <= 32 * 1024;
}

int64_t histogram_tiles(const LevelGeom &g, int64_t tau) {
    const HistTile ht = hist_tile(g, tau);
    return (g.elems + ht.te - 1) / ht.te;
}

void histogram(const LevelGeom &g, int64_t tau, const int64_t *in_ptr, const int32_t *in_col, int64_t *tile_row,
               int64_t *counts, hipStream_t s) {
    fill<int64_t>(counts, 0, g.n_in * g.n_chunks, s);
    if (g.elems <= 0) return;
    const HistTile ht = hist_tile(g, tau);
    const int64_t n_tiles = (g.elems + ht.te - 1) / ht.te;
    GM_REQUIRE(n_tiles < (int64_t)1 << 31, GMAGNUS_ERROR_UNSUPPORTED, "histogram: too many tiles");
    hipLaunchKernelGGL(k_tile_rows, dim3(grid_for(n_tiles, 256, 65536)), dim3(256), 0, s, in_ptr, g.n_in, ht.te,
                       n_tiles, tile_row);
    GM_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_histogram, dim3((unsigned)n_tiles), dim3(HIST_BLOCK), 0, s, g.n_in, g.elems, in_ptr,
                       tile_row, ht.te, n_tiles, in_col, g.n_chunks, g.shift, ht.R, counts);
    GM_CHECK_LAUNCH();
}

void tile_rows(const LevelGeom &g, const int64_t *in_ptr, int64_t *tile_row, hipStream_t s) {
    if (g.elems <= 0) return;
    const int64_t n_tiles = (g.elems + g.group_elems - 1) / g.group_elems;
    hipLaunchKernelGGL(k_tile_rows, dim3(grid_for(n_tiles, 256, 65536)), dim3(256), 0, s, in_ptr, g.n_in,
                       g.group_elems, n_tiles, tile_row);
    GM_CHECK_LAUNCH();
}

void chunk_classes(const int64_t *counts, int64_t n, int64_t tau, bool last, uint8_t *cls, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_chunk_classes, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, counts, n, tau, (int)last,
                       cls);
    GM_CHECK_LAUNCH();
}

void chunk_reorder(const int64_t *counts, const int64_t *inv, int64_t n, int n_chunks, const int64_t *origin_in,
                   int64_t stride, int64_t cmajor_rows, int64_t *out_cnt, int64_t *origin_out, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_chunk_reorder, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, counts, inv, n, n_chunks,
                       origin_in, stride, cmajor_rows, out_cnt, origin_out);
    GM_CHECK_LAUNCH();
}

void multisplit(const LevelGeom &g, const int64_t *in_ptr, const int64_t *tile_row, const int32_t *in_col,
                const void *in_val_v, bool v32, const int64_t *x_map, int64_t *cursor, int32_t *out_col, void *out_val_v,
                int64_t n_heavy_out, int64_t *next_counts, hipStream_t s) {
    if (g.elems <= 0) return;
    const int cbits = ilog2(g.n_chunks);
    const int rbits = ilog2(g.group_rows);
    GM_REQUIRE((1 << cbits) == g.n_chunks && (1 << rbits) == g.group_rows, GMAGNUS_ERROR_INVALID_VALUE,
               "multisplit: chunk and row counts must be powers of two");
    GM_REQUIRE(g.group_rows <= MS_RMAX && (g.group_rows << cbits) <= MS_KMAX, GMAGNUS_ERROR_UNSUPPORTED,
               "multisplit: too many keys per work group");
    const bool fuse = next_counts != nullptr && n_heavy_out > 0 && g.next_chunks > 0;
    if (fuse)
        GM_REQUIRE(multisplit_next_fits(g.group_rows << cbits, g.next_chunks), GMAGNUS_ERROR_UNSUPPORTED,
                   "multisplit: next-level histogram does not fit");
    int64_t *nc = fuse ? next_counts : nullptr;
    with_value_type(v32, [&](auto v) {
        using V = decltype(v);
        const V *in_val = static_cast<const V *>(in_val_v);
        V *out_val = static_cast<V *>(out_val_v);
    switch (g.group_elems) {
    case 1024:
        launch_multisplit<128, 1024, V>(g, in_ptr, tile_row, in_col, in_val, x_map, cursor, out_col, out_val,
                                     n_heavy_out, nc, cbits, rbits, s);
        break;
    case 4096:
        launch_multisplit<256, 4096, V>(g, in_ptr, tile_row, in_col, in_val, x_map, cursor, out_col, out_val,
                                     n_heavy_out, nc, cbits, rbits, s);
        break;
    case 2048:
        launch_multisplit<256, 2048, V>(g, in_ptr, tile_row, in_col, in_val, x_map, cursor, out_col, out_val,
                                     n_heavy_out, nc, cbits, rbits, s);
        break;
    case 512:
        launch_multisplit<256, 512, V>(g, in_ptr, tile_row, in_col, in_val, x_map, cursor, out_col, out_val,
                                    n_heavy_out, nc, cbits, rbits, s);
        break;
    default: throw Error{GMAGNUS_ERROR_INVALID_VALUE, "multisplit: unsupported tile size"};
    }
    });
}

}  // namespace gm
