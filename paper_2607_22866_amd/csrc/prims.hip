// Device-wide primitives: three-pass exclusive scan of int64 values and a
// stable multi-class partition built on it (the flagged partitions of
// Algorithm 3: light/heavy rows, slices, heavy/light chunks, bins).
#include "host.hpp"

namespace gm {

namespace {

constexpr int SCAN_BLOCK = 256;
constexpr int SCAN_ITEMS = 8;
constexpr int64_t SCAN_TILE = SCAN_BLOCK * SCAN_ITEMS;

struct PlainIn {
    const int64_t *p;
    GM_DEV int64_t operator()(int64_t i) const { return p[i]; }
};
struct GatherIn {
    const int64_t *p;
    const int64_t *idx;
    GM_DEV int64_t operator()(int64_t i) const { return p[idx[i]]; }
};

template <class In>
__global__ __launch_bounds__(SCAN_BLOCK) void k_scan_reduce(In in, int64_t n, int64_t *partial) {
    __shared__ int64_t sm[SCAN_BLOCK / GM_WAVE];
    const int64_t base = blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j)
        if (base + j < n) s += in(base + j);
    s = block_reduce_sum<SCAN_BLOCK>(s, sm);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

// One block scans the tile sums in place (exclusive) and writes the total
// after the last tile sum.
__global__ __launch_bounds__(1024) void k_scan_partials(int64_t *partial, int64_t n_tiles) {
    __shared__ int64_t sm[1024 / GM_WAVE];
    __shared__ int64_t carry;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int64_t b = 0; b < n_tiles; b += 1024) {
        const int64_t i = b + threadIdx.x;
        int64_t x = i < n_tiles ? partial[i] : 0;
        int64_t tot;
        int64_t ex = block_excl_scan<1024>(x, sm, &tot);
        const int64_t c = carry;
        if (i < n_tiles) partial[i] = c + ex;
        __syncthreads();
        if (threadIdx.x == 0) carry = c + tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[n_tiles] = carry;
}

template <class In>
__global__ __launch_bounds__(SCAN_BLOCK) void k_scan_apply(In in, int64_t n, const int64_t *partial, int64_t *out) {
    __shared__ int64_t sm[SCAN_BLOCK / GM_WAVE];
    const int64_t base = blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
    int64_t v[SCAN_ITEMS];
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) {
        v[j] = base + j < n ? in(base + j) : 0;
        s += v[j];
    }
    int64_t run = partial[blockIdx.x] + block_excl_scan<SCAN_BLOCK>(s, sm);
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) {
        if (base + j < n) out[base + j] = run;
        run += v[j];
    }
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) out[n] = partial[gridDim.x];
}

// Small inputs: one work group walks the array in pieces of 8192 with a
// running carry (one launch instead of three; below ~16K items the launches
// cost more than the work).
constexpr int SCAN1_BLOCK = 1024;
constexpr int64_t SCAN1_MAX = 16384;

template <class In>
__global__ __launch_bounds__(SCAN1_BLOCK) void k_scan_single(In in, int64_t n, int64_t *out) {
    __shared__ int64_t sm[SCAN1_BLOCK / GM_WAVE];
    int64_t carry = 0;
    for (int64_t b0 = 0; b0 < n; b0 += (int64_t)SCAN1_BLOCK * SCAN_ITEMS) {
        const int64_t base = b0 + threadIdx.x * SCAN_ITEMS;
        int64_t v[SCAN_ITEMS];
        int64_t sum = 0;
#pragma unroll
        for (int j = 0; j < SCAN_ITEMS; ++j) {
            v[j] = base + j < n ? in(base + j) : 0;
            sum += v[j];
        }
        int64_t tot;
        int64_t run = carry + block_excl_scan<SCAN1_BLOCK>(sum, sm, &tot);
#pragma unroll
        for (int j = 0; j < SCAN_ITEMS; ++j) {
            if (base + j < n) out[base + j] = run;
            run += v[j];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) out[n] = carry;
}

template <class In>
void scan_impl(In in, int64_t n, int64_t *out, int64_t *scratch, hipStream_t s) {
    if (n <= 0) {
        fill<int64_t>(out, 0, 1, s);
        return;
    }
    if (n <= SCAN1_MAX) {
        hipLaunchKernelGGL(k_scan_single<In>, dim3(1), dim3(SCAN1_BLOCK), 0, s, in, n, out);
        GM_CHECK_LAUNCH();
        return;
    }
    const int64_t tiles = (n + SCAN_TILE - 1) / SCAN_TILE;
    hipLaunchKernelGGL(k_scan_reduce<In>, dim3((unsigned)tiles), dim3(SCAN_BLOCK), 0, s, in, n, scratch);
    GM_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(1024), 0, s, scratch, tiles);
    GM_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_scan_apply<In>, dim3((unsigned)tiles), dim3(SCAN_BLOCK), 0, s, in, n, scratch, out);
    GM_CHECK_LAUNCH();
}

// ---------------------------------------------------------------- partition
constexpr int PART_BLOCK = 256;
constexpr int PART_ITEMS = 16;
constexpr int64_t PART_TILE = PART_BLOCK * PART_ITEMS;
constexpr int PART_MAX_CLASSES = 16;

__global__ __launch_bounds__(PART_BLOCK) void k_part_count(const uint8_t *cls, int64_t n, int nc, int64_t n_tiles,
                                                           int64_t *tile_count) {
    __shared__ int cnt[PART_MAX_CLASSES];
    if (threadIdx.x < PART_MAX_CLASSES) cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = blockIdx.x * PART_TILE;
    for (int j = 0; j < PART_ITEMS; ++j) {
        const int64_t i = base + j * PART_BLOCK + threadIdx.x;
        if (i < n) atomicAdd(&cnt[cls[i]], 1);
    }
    __syncthreads();
    if (threadIdx.x < nc) tile_count[threadIdx.x * n_tiles + blockIdx.x] = cnt[threadIdx.x];
}

// Each thread owns PART_ITEMS consecutive items; per-class counts of the
// threads are scanned in thread order (four 16-bit class counters per int64
// word), so positions are stable in item order. base_off[c]: position of the
// tile's first item of class c.
GM_DEV void part_tile_scatter(const uint8_t *cls, int64_t n, int nc, int64_t tile, const int64_t *base_off,
                              int64_t *sm, int64_t *perm, int64_t *inv, int64_t *tile_tot = nullptr) {
    const int64_t base = tile * PART_TILE + (int64_t)threadIdx.x * PART_ITEMS;
    uint8_t c[PART_ITEMS];
#pragma unroll
    for (int j = 0; j < PART_ITEMS; ++j) c[j] = base + j < n ? cls[base + j] : 0xFF;
    int prefix[PART_MAX_CLASSES];
#pragma unroll
    for (int g = 0; g < PART_MAX_CLASSES / 4; ++g) {
        if (4 * g >= nc) {  // nc is uniform over the block
#pragma unroll
            for (int q = 0; q < 4; ++q) prefix[4 * g + q] = 0;
            continue;
        }
        uint64_t packed = 0;
#pragma unroll
        for (int j = 0; j < PART_ITEMS; ++j) {
            const int q = (int)c[j] - 4 * g;
            if (c[j] != 0xFF && q >= 0 && q < 4) packed += uint64_t(1) << (16 * q);
        }
        int64_t tot = 0;
        const uint64_t ex = (uint64_t)block_excl_scan<PART_BLOCK>((int64_t)packed, sm, &tot);
#pragma unroll
        for (int q = 0; q < 4; ++q) prefix[4 * g + q] = (int)((ex >> (16 * q)) & 0xFFFF);
        if (tile_tot && threadIdx.x < 4) tile_tot[4 * g + threadIdx.x] = ((uint64_t)tot >> (16 * threadIdx.x)) & 0xFFFF;
    }
    __syncthreads();
    int run[PART_MAX_CLASSES];
#pragma unroll
    for (int q = 0; q < PART_MAX_CLASSES; ++q) run[q] = 0;
#pragma unroll
    for (int j = 0; j < PART_ITEMS; ++j) {
        if (c[j] == 0xFF) continue;
        int r = 0, p = 0;
#pragma unroll
        for (int q = 0; q < PART_MAX_CLASSES; ++q)
            if (q == c[j]) {
                r = run[q]++;
                p = prefix[q];
            }
        const int64_t pos = base_off[c[j]] + p + r;
        perm[pos] = base + j;
        if (inv) inv[base + j] = pos;
    }
}

__global__ __launch_bounds__(PART_BLOCK) void k_part_scatter(const uint8_t *cls, int64_t n, int nc, int64_t n_tiles,
                                                             const int64_t *tile_off, int64_t *perm, int64_t *inv) {
    __shared__ int64_t sm[PART_BLOCK / GM_WAVE];
    __shared__ int64_t base_off[PART_MAX_CLASSES];
    if (threadIdx.x < nc) base_off[threadIdx.x] = tile_off[threadIdx.x * n_tiles + blockIdx.x];
    part_tile_scatter(cls, n, nc, blockIdx.x, base_off, sm, perm, inv);
}

// Small inputs: one work group counts the classes, then scatters tile by tile
// with running per-class offsets (one launch instead of six).
constexpr int64_t PART1_MAX = 16384;

__global__ __launch_bounds__(PART_BLOCK) void k_part_single(const uint8_t *cls, int64_t n, int nc, int64_t *perm,
                                                            int64_t *inv, int64_t *class_start) {
    __shared__ int64_t sm[PART_BLOCK / GM_WAVE];
    __shared__ int64_t off[PART_MAX_CLASSES + 1];
    __shared__ int64_t tile_tot[PART_MAX_CLASSES];
    // class counts in one pass: per thread two 32-bit counters per int64 word
    // (no LDS atomics: a few classes would serialise them)
    constexpr int NG = PART_MAX_CLASSES / 2;
    uint64_t packed[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) packed[g] = 0;
    for (int64_t i = threadIdx.x; i < n; i += PART_BLOCK) {
        const int c = cls[i];
#pragma unroll
        for (int g = 0; g < NG; ++g) packed[g] += (c >> 1) == g ? uint64_t(1) << (32 * (c & 1)) : 0;
    }
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        if (2 * g >= nc) break;  // nc is uniform over the block
        const int64_t tot = block_reduce_sum<PART_BLOCK>((int64_t)packed[g], sm);
        if (threadIdx.x < 2 && 2 * g + (int)threadIdx.x < nc)
            off[2 * g + threadIdx.x + 1] = ((uint64_t)tot >> (32 * threadIdx.x)) & 0xFFFFFFFFu;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        off[0] = 0;
        for (int c = 0; c < nc; ++c) off[c + 1] += off[c];
        for (int c = 0; c <= nc; ++c) class_start[c] = off[c];
    }
    __syncthreads();
    const int64_t tiles = (n + PART_TILE - 1) / PART_TILE;
    for (int64_t t = 0; t < tiles; ++t) {
        part_tile_scatter(cls, n, nc, t, off, sm, perm, inv, tile_tot);
        __syncthreads();
        if (threadIdx.x < nc) off[threadIdx.x] += tile_tot[threadIdx.x];  // running offsets past this tile
        __syncthreads();
    }
}

__global__ void k_class_starts(const int64_t *tile_off, int nc, int64_t n_tiles, int64_t *class_start) {
    const int c = threadIdx.x;
    if (c <= nc) class_start[c] = tile_off[(int64_t)c * n_tiles];
}

}  // namespace

int64_t scan_scratch_elems(int64_t n) { return (n + SCAN_TILE - 1) / SCAN_TILE + 2; }

void scan_i64(const int64_t *in, int64_t n, int64_t *out, int64_t *scratch, hipStream_t s) {
    scan_impl(PlainIn{in}, n, out, scratch, s);
}

void scan_gather_i64(const int64_t *in, const int64_t *idx, int64_t n, int64_t *out, int64_t *scratch,
                     hipStream_t s) {
    scan_impl(GatherIn{in, idx}, n, out, scratch, s);
}

int64_t partition_scratch_elems(int64_t n, int nc) {
    const int64_t tiles = (n + PART_TILE - 1) / PART_TILE;
    const int64_t m = tiles * nc;
    return m + (m + 1) + scan_scratch_elems(m);
}

void partition_u8(const uint8_t *cls, int64_t n, int nc, int64_t *perm, int64_t *inv, int64_t *class_start,
                  int64_t *scratch, hipStream_t s) {
    GM_REQUIRE(nc >= 1 && nc <= PART_MAX_CLASSES, GMAGNUS_ERROR_INVALID_VALUE, "partition: too many classes");
    const int64_t tiles = (n + PART_TILE - 1) / PART_TILE;
    if (n <= 0) {
        fill<int64_t>(class_start, 0, nc + 1, s);
        return;
    }
    if (n <= PART1_MAX) {
        hipLaunchKernelGGL(k_part_single, dim3(1), dim3(PART_BLOCK), 0, s, cls, n, nc, perm, inv, class_start);
        GM_CHECK_LAUNCH();
        return;
    }
    const int64_t m = tiles * nc;
    int64_t *tile_count = scratch;
    int64_t *tile_off = scratch + m;
    int64_t *sc = tile_off + m + 1;
    hipLaunchKernelGGL(k_part_count, dim3((unsigned)tiles), dim3(PART_BLOCK), 0, s, cls, n, nc, tiles, tile_count);
    GM_CHECK_LAUNCH();
    scan_i64(tile_count, m, tile_off, sc, s);
    hipLaunchKernelGGL(k_part_scatter, dim3((unsigned)tiles), dim3(PART_BLOCK), 0, s, cls, n, nc, tiles, tile_off,
                       perm, inv);
    GM_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_class_starts, dim3(1), dim3(64), 0, s, tile_off, nc, tiles, class_start);
    GM_CHECK_LAUNCH();
}

}  // namespace gm
