// Streaming bandwidth probe: the measured peak that the paper's
// speed-of-light figures divide by (Section IV-C measures it with a copy
// kernel). Grid-stride loops over 16-byte elements, each wave touching
// 1 KiB of consecutive memory per access; variants for ordinary and
// nontemporal loads and stores. A gather variant reads random 128-byte lines
// of a working set of a given size, the access of the expansion's B-row
// gathers, so its rate against the working-set size shows which sizes the
// L2s (4 MB per XCD) and the Infinity Cache serve faster than HBM.
#include "host.hpp"

namespace gm {
namespace {

constexpr int PROBE_BLOCK = 256;

struct alignas(16) V2 {
    double x, y;
};

__global__ __launch_bounds__(PROBE_BLOCK) void k_probe_read(const V2 *__restrict__ a, int64_t n, double *sink) {
    double s = 0.0;
    for (int64_t i = blockIdx.x * (int64_t)PROBE_BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * PROBE_BLOCK) {
        const V2 v = a[i];
        s += v.x + v.y;
    }
    if (s == -1.0) sink[0] = s;  // keeps the loads; never true for the filled buffer
}

__global__ __launch_bounds__(PROBE_BLOCK) void k_probe_read_nt(const V2 *__restrict__ a, int64_t n, double *sink) {
    double s = 0.0;
    for (int64_t i = blockIdx.x * (int64_t)PROBE_BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * PROBE_BLOCK) {
        const double *p = &a[i].x;
        s += __builtin_nontemporal_load(p) + __builtin_nontemporal_load(p + 1);
    }
    if (s == -1.0) sink[0] = s;
}

__global__ __launch_bounds__(PROBE_BLOCK) void k_probe_write(V2 *__restrict__ a, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)PROBE_BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * PROBE_BLOCK)
        a[i] = V2{1.0, (double)i};
}

__global__ __launch_bounds__(PROBE_BLOCK) void k_probe_write_nt(V2 *__restrict__ a, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)PROBE_BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * PROBE_BLOCK) {
        double *p = &a[i].x;
        __builtin_nontemporal_store(1.0, p);
        __builtin_nontemporal_store((double)i, p + 1);
    }
}

// Each group of 8 lanes reads one random line of the working set (16 bytes a
// lane), four lines in flight per lane; xorshift32 line indices (the 8 lanes
// of a group share the generator, so they read the same line).
constexpr unsigned GATHER_GRID = 2048;
constexpr int GATHER_ITERS = 512;  // 2048 groups x 256 lanes x 512 x 16 B = 4 GiB per run

__global__ __launch_bounds__(PROBE_BLOCK) void k_probe_gather(const V2 *__restrict__ a, uint32_t lines_mask,
                                                              double *sink) {
    const int lane = threadIdx.x & 7;
    uint32_t x = ((blockIdx.x * PROBE_BLOCK + threadIdx.x) >> 3) * 2654435761u + 0x9E3779B9u;
    double s = 0.0;
    for (int it = 0; it < GATHER_ITERS; it += 4) {
        V2 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            x ^= x << 13;
            x ^= x >> 17;
            x ^= x << 5;
            v[u] = a[(uint64_t)(x & lines_mask) * 8 + lane];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) s += v[u].x + v[u].y;
    }
    if (s == -1.0) sink[0] = s;
}

__global__ __launch_bounds__(PROBE_BLOCK) void k_probe_copy(const V2 *__restrict__ a, V2 *__restrict__ b, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)PROBE_BLOCK + threadIdx.x; i < n; i += (int64_t)gridDim.x * PROBE_BLOCK)
        b[i] = a[i];
}

}  // namespace
}  // namespace gm

using namespace gm;

extern "C" gmagnus_status_t gmagnus_bandwidth_probe(int32_t kind, void *dst, const void *src, int64_t bytes,
                                                    int32_t grid, int32_t reps, void *hip_stream, double *ms) {
    try {
        GM_REQUIRE(kind >= GMAGNUS_PROBE_READ && kind <= GMAGNUS_PROBE_GATHER, GMAGNUS_ERROR_INVALID_VALUE,
                   "unknown probe kind");
        GM_REQUIRE(kind != GMAGNUS_PROBE_GATHER ||
                       (bytes >= 4096 && bytes <= ((int64_t)1 << 37) && (bytes & (bytes - 1)) == 0),
                   GMAGNUS_ERROR_INVALID_VALUE, "gather probe: the working set must be a power of two, 4 KiB .. 128 GiB");
        GM_REQUIRE(ms != nullptr && reps >= 1 && bytes >= 16 && bytes % 16 == 0, GMAGNUS_ERROR_INVALID_VALUE,
                   "probe: bytes must be a positive multiple of 16, reps >= 1, ms not NULL");
        const bool reads = kind != GMAGNUS_PROBE_WRITE && kind != GMAGNUS_PROBE_WRITE_NT;
        const bool writes = kind != GMAGNUS_PROBE_READ && kind != GMAGNUS_PROBE_READ_NT && kind != GMAGNUS_PROBE_GATHER;
        GM_REQUIRE((!reads || src) && dst, GMAGNUS_ERROR_INVALID_VALUE, "probe: NULL buffer");
        GM_REQUIRE(((uintptr_t)dst % 16) == 0 && ((uintptr_t)src % 16) == 0, GMAGNUS_ERROR_INVALID_VALUE,
                   "probe: buffers must be 16-byte aligned");
        (void)writes;
        const int64_t n = bytes / 16;
        const unsigned g = grid > 0 ? (unsigned)grid : grid_for(n, PROBE_BLOCK, 16384);
        hipStream_t s = (hipStream_t)hip_stream;
        hipEvent_t e0, e1;
        GM_HIP(hipEventCreate(&e0));
        GM_HIP(hipEventCreate(&e1));
        struct EvGuard {
            hipEvent_t a, b;
            ~EvGuard() {
                (void)hipEventDestroy(a);
                (void)hipEventDestroy(b);
            }
        } guard{e0, e1};
        // for the read kernels dst is the sink (one double, never written for the filled buffer)
        auto launch = [&]() {
            switch (kind) {
            case GMAGNUS_PROBE_READ:
                hipLaunchKernelGGL(k_probe_read, dim3(g), dim3(PROBE_BLOCK), 0, s, (const V2 *)src, n, (double *)dst);
                break;
            case GMAGNUS_PROBE_READ_NT:
                hipLaunchKernelGGL(k_probe_read_nt, dim3(g), dim3(PROBE_BLOCK), 0, s, (const V2 *)src, n,
                                   (double *)dst);
                break;
            case GMAGNUS_PROBE_WRITE:
                hipLaunchKernelGGL(k_probe_write, dim3(g), dim3(PROBE_BLOCK), 0, s, (V2 *)dst, n);
                break;
            case GMAGNUS_PROBE_WRITE_NT:
                hipLaunchKernelGGL(k_probe_write_nt, dim3(g), dim3(PROBE_BLOCK), 0, s, (V2 *)dst, n);
                break;
            case GMAGNUS_PROBE_GATHER:
                hipLaunchKernelGGL(k_probe_gather, dim3(GATHER_GRID), dim3(PROBE_BLOCK), 0, s, (const V2 *)src,
                                   (uint32_t)(bytes / 128 - 1), (double *)dst);
                break;
            default:
                hipLaunchKernelGGL(k_probe_copy, dim3(g), dim3(PROBE_BLOCK), 0, s, (const V2 *)src, (V2 *)dst, n);
            }
            GM_CHECK_LAUNCH();
        };
        launch();  // warm-up
        GM_HIP(hipEventRecord(e0, s));
        for (int r = 0; r < reps; ++r) launch();
        GM_HIP(hipEventRecord(e1, s));
        GM_HIP(hipEventSynchronize(e1));
        float t = 0.f;
        GM_HIP(hipEventElapsedTime(&t, e0, e1));
        *ms = (double)t / reps;
        return GMAGNUS_SUCCESS;
    } catch (const Error &e) {
        set_last_error(e.msg);
        return e.status;
    }
}
