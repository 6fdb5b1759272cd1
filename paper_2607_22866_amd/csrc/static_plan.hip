// Plans whose device workspace is a static device array: for callers that
// cannot allocate device memory (code under HIP graph capture, serving loops
// that forbid allocation, harnesses that do). gmagnus_plan_static builds the
// same plan as gmagnus_plan, with every workspace block carved from
// `scratch`, a file-scope device array each device holds from the first call
// on it until the process ends. Later symbolic, numeric and update_values
// calls on such a plan allocate nothing either, and its host reads go
// through pageable memory instead of a pinned staging buffer.
//
// The array is managed as a first-fit free list (blocks of 256-byte
// multiples, coalesced on release), so plans that coexist on one device take
// disjoint blocks and never share memory; together they are bounded by the
// array's size. The blocks' contents are whatever the last plan left there:
// every buffer a plan reads is written by that plan first, as with memory
// from hipMalloc.
#include <map>
#include <mutex>

#include "host.hpp"

namespace {

constexpr size_t STATIC_WORKSPACE_BYTES = (size_t)GMAGNUS_STATIC_WORKSPACE_MIB << 20;
constexpr int MAX_DEVICES = 64;
// setup work a plan holds for every row of its panel (row products, column
// spans, bins, permutation, prefix sums), a lower bound of its workspace
constexpr int64_t SETUP_BYTES_PER_ROW = 41;

__device__ __align__(256) unsigned char scratch[STATIC_WORKSPACE_BYTES];

struct Arena {
    unsigned char *base = nullptr;     // the device's address of `scratch` (hipGetSymbolAddress)
    std::map<size_t, size_t> free_;    // offset -> bytes
    std::map<size_t, size_t> used_;    // offset -> bytes
};

std::mutex g_mutex;
Arena g_arena[MAX_DEVICES];

// Address of this device's array, looked up once per device with the device
// current. Host code uses only this address, never the array's name.
Arena &arena_for_current_device() {
    int dev = 0;
    GM_HIP(hipGetDevice(&dev));
    GM_REQUIRE(dev >= 0 && dev < MAX_DEVICES, GMAGNUS_ERROR_UNSUPPORTED, "device index beyond the static workspace table");
    std::lock_guard<std::mutex> lk(g_mutex);
    Arena &a = g_arena[dev];
    if (!a.base) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            throw gm::Error{GMAGNUS_ERROR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e)};
        a.base = static_cast<unsigned char *>(ptr);
        a.free_.clear();
        a.used_.clear();
        a.free_[0] = STATIC_WORKSPACE_BYTES;
    }
    return a;
}

void *arena_alloc(size_t bytes, void * /*stream*/, void *ctx) {
    Arena &a = *static_cast<Arena *>(ctx);
    bytes = (bytes + 255) & ~(size_t)255;
    std::lock_guard<std::mutex> lk(g_mutex);
    for (auto it = a.free_.begin(); it != a.free_.end(); ++it) {
        if (it->second < bytes) continue;
        const size_t off = it->first, len = it->second;
        a.free_.erase(it);
        if (len > bytes) a.free_[off + bytes] = len - bytes;
        a.used_[off] = bytes;
        return a.base + off;
    }
    return nullptr;
}

void arena_free(void *p, void * /*stream*/, void *ctx) {
    Arena &a = *static_cast<Arena *>(ctx);
    std::lock_guard<std::mutex> lk(g_mutex);
    auto u = a.used_.find((size_t)(static_cast<unsigned char *>(p) - a.base));
    if (u == a.used_.end()) return;
    size_t off = u->first, len = u->second;
    a.used_.erase(u);
    auto next = a.free_.lower_bound(off);
    if (next != a.free_.end() && off + len == next->first) {
        len += next->second;
        next = a.free_.erase(next);
    }
    if (next != a.free_.begin()) {
        auto prev = std::prev(next);
        if (prev->first + prev->second == off) {
            prev->second += len;
            return;
        }
    }
    a.free_[off] = len;
}

}  // namespace

extern "C" gmagnus_status_t gmagnus_plan_static(gmagnus_plan_t *out, const gmagnus_csr_t *A, const gmagnus_csr_t *B,
                                                const gmagnus_options_t *opts, void *hip_stream) {
    if (out) *out = nullptr;
    gmagnus_options_t o;
    Arena *arena = nullptr;
    try {
        GM_REQUIRE(out != nullptr, GMAGNUS_ERROR_INVALID_VALUE, "NULL plan output");
        if (opts) {
            GM_REQUIRE(opts->struct_size == sizeof(gmagnus_options_t), GMAGNUS_ERROR_INVALID_VALUE,
                       "options.struct_size mismatch");
            GM_REQUIRE(opts->alloc == nullptr && opts->free == nullptr, GMAGNUS_ERROR_INVALID_VALUE,
                       "a static-workspace plan takes no allocator callbacks");
            o = *opts;
        } else {
            gmagnus_options_init(&o);
        }
        GM_REQUIRE(A != nullptr, GMAGNUS_ERROR_INVALID_VALUE, "A is NULL");
        const int64_t r1 = o.row_end > 0 ? o.row_end : A->n_rows;
        const int64_t rows = r1 - o.row_begin;
        GM_REQUIRE(rows <= (int64_t)(STATIC_WORKSPACE_BYTES / SETUP_BYTES_PER_ROW), GMAGNUS_ERROR_UNSUPPORTED,
                   "a panel of " + std::to_string(rows) + " rows needs more than the static workspace of " +
                       std::to_string(STATIC_WORKSPACE_BYTES) + " bytes per device holds (at most " +
                       std::to_string(STATIC_WORKSPACE_BYTES / SETUP_BYTES_PER_ROW) +
                       " rows per panel, fewer for heavy rows)");
        arena = &arena_for_current_device();
    } catch (const gm::Error &e) {
        gm::set_last_error(e.msg);
        return e.status;
    }
    o.alloc = arena_alloc;
    o.free = arena_free;
    o.alloc_ctx = arena;
    if (o.workspace_limit_bytes <= 0 || o.workspace_limit_bytes > (int64_t)STATIC_WORKSPACE_BYTES)
        o.workspace_limit_bytes = (int64_t)STATIC_WORKSPACE_BYTES;
    gmagnus_matrix_t a{}, b{};
    if (A) a = gmagnus_matrix_t{A->n_rows, A->n_cols, A->nnz, A->row_ptr, A->col_idx, A->val, GMAGNUS_INDEX_INT32,
                                GMAGNUS_VALUE_FP64};
    if (B) b = gmagnus_matrix_t{B->n_rows, B->n_cols, B->nnz, B->row_ptr, B->col_idx, B->val, GMAGNUS_INDEX_INT32,
                                GMAGNUS_VALUE_FP64};
    return gm::make_plan(out, &a, B ? &b : nullptr, &o, hip_stream, true);
}
