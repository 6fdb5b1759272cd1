// Host orchestration of the SpGEMM C = A*B (Algorithm 3) behind the C ABI of
// gmagnus.h: parameter selection (Section III-D), the setup phase, the heavy
// path (masked CSC, outer product, hierarchical multisplit, final chunks) on
// one HIP stream and the light path on another, the C row-pointer scan, and
// the numeric phase. Also the library's caching device allocator.
#include <algorithm>
#include <cstring>
#include <functional>
#include <map>
#include <memory>
#include <mutex>

#include "host.hpp"

namespace gm {

// ------------------------------------------------------------ last error
static thread_local std::string g_last_error;
void set_last_error(const std::string &msg) { g_last_error = msg; }

// --------------------------------------------------------- caching allocator
namespace {
struct DeviceCache {
    std::mutex m;
    std::multimap<std::pair<int, size_t>, void *> free_blocks;  // (device, bytes) -> block
    std::map<void *, std::pair<int, size_t>> sizes;             // all blocks handed out
};
DeviceCache &cache() {
    static DeviceCache *c = new DeviceCache();  // never destroyed: outlives static plans
    return *c;
}

size_t round_bytes(size_t b) {
    if (b < ((size_t)1 << 20)) return (b + 255) & ~(size_t)255;
    if (b >= ((size_t)1 << 30)) {
        // eight size classes per power of two: row panels of slightly
        // different sizes then ask for the same block, which the cache hands
        // back, instead of a fresh hipMalloc of tens of GB (about a second)
        size_t top = (size_t)1 << 30;
        while (top * 2 <= b) top *= 2;
        const size_t step = top / 8;
        return (b + step - 1) / step * step;
    }
    const size_t g = (size_t)2 << 20;
    return (b + g - 1) / g * g;
}

void *cache_alloc(size_t bytes) {
    int dev = 0;
    GM_HIP(hipGetDevice(&dev));
    bytes = round_bytes(bytes);
    DeviceCache &c = cache();
    {
        std::lock_guard<std::mutex> lk(c.m);
        auto it = c.free_blocks.lower_bound({dev, bytes});
        // reuse a block up to 25% (+2 MiB) larger than asked, or up to twice
        // as large for blocks of 1 GiB and more (a fresh hipMalloc of that size
        // stalls the host far longer than the memory it would save is worth)
        const size_t slack = bytes >= ((size_t)1 << 30) ? bytes : bytes / 4 + ((size_t)2 << 20);
        if (it != c.free_blocks.end() && it->first.first == dev && it->first.second <= bytes + slack) {
            void *p = it->second;
            c.free_blocks.erase(it);
            return p;
        }
    }
    void *p = nullptr;
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        cache_release();
        e = hipMalloc(&p, bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            throw Error{GMAGNUS_ERROR_OUT_OF_MEMORY, "device allocation of " + std::to_string(bytes) + " bytes failed"};
        }
    }
    std::lock_guard<std::mutex> lk(c.m);
    c.sizes[p] = {dev, bytes};
    return p;
}

void cache_free(void *p) {
    DeviceCache &c = cache();
    std::lock_guard<std::mutex> lk(c.m);
    auto it = c.sizes.find(p);
    if (it == c.sizes.end()) return;
    c.free_blocks.insert({it->second, p});
}
}  // namespace

void cache_release() {
    DeviceCache &c = cache();
    std::lock_guard<std::mutex> lk(c.m);
    for (auto &kv : c.free_blocks) {
        (void)hipFree(kv.second);
        c.sizes.erase(kv.second);
    }
    c.free_blocks.clear();
}

void Workspace::give_back(const Block &b) {
    if (ufree_)
        ufree_(b.p, (void *)stream_, uctx_);
    else
        cache_free(b.p);
    owned_ -= b.bytes;
}

void allow_dynamic_lds(const void *kernel, int bytes) {
    static std::mutex m;
    static std::map<std::pair<int, const void *>, int> done;  // (device, kernel) -> bytes allowed
    int dev = 0;
    GM_HIP(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lk(m);
    auto it = done.find({dev, kernel});
    if (it != done.end() && it->second >= bytes) return;
    GM_HIP(hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
    done[{dev, kernel}] = bytes;
}

void *Workspace::alloc_bytes(size_t bytes) {
    const size_t want = round_bytes(bytes);
    for (size_t i = 0; i < spare_.size(); ++i)
        if (spare_[i].bytes >= want && spare_[i].bytes <= want + want / 4 + ((size_t)2 << 20)) {
            Block b = spare_[i];
            spare_[i] = spare_.back();
            spare_.pop_back();
            blocks_.push_back(b);
            in_use_ += b.bytes;
            return b.p;
        }
    if (limit_ && owned_ + want > limit_) {
        // blocks this plan freed count against the limit too: return them first
        for (auto &b : spare_) give_back(b);
        spare_.clear();
        if (owned_ + want > limit_)
            throw Error{GMAGNUS_ERROR_OUT_OF_MEMORY,
                        "workspace limit of " + std::to_string(limit_) + " bytes reached: " + std::to_string(owned_) +
                            " bytes in use, " + std::to_string(want) + " more requested"};
    }
    void *p = nullptr;
    if (ualloc_) {
        p = ualloc_(want, (void *)stream_, uctx_);
        if (!p)
            throw Error{GMAGNUS_ERROR_OUT_OF_MEMORY, "the workspace allocator returned NULL for " +
                                                         std::to_string(want) + " bytes (" + std::to_string(owned_) +
                                                         " bytes held by the plan)"};
    } else {
        try {
            p = cache_alloc(want);
        } catch (const Error &) {
            // give this plan's spare blocks back and retry once
            for (auto &b : spare_) give_back(b);
            spare_.clear();
            p = cache_alloc(want);
        }
    }
    blocks_.push_back({p, want});
    in_use_ += want;
    owned_ += want;
    peak_ = std::max(peak_, owned_);
    return p;
}

void Workspace::free(void *p) {
    if (!p || hold_) return;
    for (size_t i = 0; i < blocks_.size(); ++i)
        if (blocks_[i].p == p) {
            in_use_ -= blocks_[i].bytes;
            spare_.push_back(blocks_[i]);
            blocks_[i] = blocks_.back();
            blocks_.pop_back();
            return;
        }
}

void Workspace::release_all() {
    for (auto *v : {&blocks_, &spare_})
        for (auto &b : *v) give_back(b);
    blocks_.clear();
    spare_.clear();
    in_use_ = 0;
    owned_ = 0;
}

// --------------------------------------------------------------- planner
namespace {
constexpr int64_t S_ROWPTR = 8, S_HISTO = 4, ALPHA = 2, N_SUBGROUPS = 16;
constexpr int64_t MIN_LOCAL_CHUNK = 64;  // mean elements per local chunk of a multisplit group
constexpr int MAX_DENSE_LOG2 = 13;       // 8192 fp64 values + bitmap per work group
constexpr int MAX_CHUNKS_LOG2 = 6;       // chunks per level the multisplit kernel supports

// Largest column count of C for an index type. With int64 columns every
// multisplit level stores chunk-local columns in 32 bits: 2^35 columns in 32
// first-level chunks leave chunks of 2^30 columns.
int64_t max_columns(int64_t s_col) { return s_col == 8 ? ((int64_t)1 << 35) : ((int64_t)1 << 31) - 1; }

// s_col / s_val: byte sizes of the column index and value types.
void compute_params(int64_t c_m, int64_t s_lm, int64_t S_COL, int64_t S_VAL, const gmagnus_options_t *o,
                    gmagnus_params_t *p) {
    GM_REQUIRE(c_m >= 1 && c_m <= max_columns(S_COL), GMAGNUS_ERROR_INVALID_VALUE,
               S_COL == 8 ? "C must have 1..2^35 columns" : "C must have 1..2^31-1 columns");
    GM_REQUIRE(s_lm >= 1024, GMAGNUS_ERROR_INVALID_VALUE, "local memory size below 1 KB");
    std::memset(p, 0, sizeof(*p));
    // tau: alpha*tau hash slots of (column, value) fill the local memory
    int64_t tau = s_lm / (ALPHA * (S_COL + S_VAL));
    // dense width: one value and one bitmap bit per column, with alpha headroom
    int64_t W = floor_pow2((8 * s_lm) / (ALPHA * (8 * S_VAL + 1)));
    if (o && o->tau > 0) tau = o->tau;
    if (o && o->dense_width_log2 > 0) {
        GM_REQUIRE(o->dense_width_log2 >= 5 && o->dense_width_log2 <= MAX_DENSE_LOG2, GMAGNUS_ERROR_INVALID_VALUE,
                   "dense width must be 2^5 .. 2^13");
        W = int64_t(1) << o->dense_width_log2;
    }
    W = std::min<int64_t>(W, int64_t(1) << MAX_DENSE_LOG2);
    const int64_t req = std::max<int64_t>(1, ceil_pow2(c_m) / W);
    // half of local memory holds the locally permuted elements of a multisplit group
    const int64_t min_group = s_lm / (2 * (S_COL + S_VAL));
    const int64_t group_rows = (min_group - 1 + tau - 1) / tau + 1;
    // the light accumulators hold at most tau_limit() products per row
    tau = std::min<int64_t>(tau, tau_limit());
    const int64_t eq = (s_lm - min_group * (S_COL + S_VAL) - S_HISTO) / (group_rows * (N_SUBGROUPS * S_HISTO + S_ROWPTR));
    int64_t cmax = std::min(floor_pow2(eq), floor_pow2(min_group / (group_rows * MIN_LOCAL_CHUNK)));
    if (o && o->chunks_max_log2 > 0) cmax = int64_t(1) << o->chunks_max_log2;
    cmax = std::max<int64_t>(2, std::min<int64_t>(cmax, int64_t(1) << MAX_CHUNKS_LOG2));
    p->tau = tau;
    p->dense_width = W;
    p->chunks_required = req;
    p->chunks_max = cmax;
    p->min_group_elems = min_group;
    p->group_rows = group_rows;
    if (req == 1) {
        p->n_levels = 0;
    } else if (req <= cmax) {
        p->n_levels = 1;
        p->v_chunks[0] = (int32_t)req;
    } else {
        const int lr = ilog2(req), lm = ilog2(cmax);
        const int levels = (lr + lm - 1) / lm;
        GM_REQUIRE(levels <= GMAGNUS_MAX_LEVELS, GMAGNUS_ERROR_UNSUPPORTED, "too many multisplit levels");
        p->n_levels = levels;
        for (int i = 0; i < levels - 1; ++i) p->v_chunks[i] = (int32_t)cmax;
        p->v_chunks[levels - 1] = (int32_t)(req >> (lm * (levels - 1)));
    }
}
}  // namespace

}  // namespace gm

using namespace gm;

// ------------------------------------------------------------------ plan
namespace {
struct Timed;
}

struct LeafLevel {
    LeafSet set;
    int64_t width = 0;
    int64_t *leaf_nnz = nullptr;
    int64_t *items_sym = nullptr, *items_num = nullptr;
    int64_t bins_sym[LEAF_NBINS + 1] = {0};
    int64_t bins_num[LEAF_NBINS + 1] = {0};
    int64_t elems = 0;
};

struct TimedEvent {
    int cls;
    hipEvent_t a, b;
};

struct gmagnus_plan_s {
    Csr A{}, B{};
    int64_t r0 = 0, r1 = 0, n = 0;
    gmagnus_options_t opts{};
    gmagnus_params_t params{};
    hipStream_t stream = nullptr, s_heavy = nullptr, s_light = nullptr;
    bool own_streams = false;
    std::unique_ptr<Workspace> ws;
    int32_t *err = nullptr;  // device consistency flags
    // setup
    int64_t *ip = nullptr;
    void *minc = nullptr, *maxc = nullptr;  // B's column type
    int64_t vsize = 8, csize = 4;          // bytes of a value and of a column index
    int64_t *perm = nullptr;          // rows grouped by symbolic light bin (heavy class included)
    int64_t bins_sym[LIGHT_NBINS + 1] = {0};
    int64_t *perm_num = nullptr;      // rows grouped by numeric bin
    int64_t bins_num[LIGHT_NBINS + 1] = {0};
    int64_t n_heavy = 0;
    const int64_t *heavy_rows = nullptr;
    int64_t *chat_ptr = nullptr;      // n_heavy + 1
    int64_t products_total = 0, products_heavy = 0;
    int64_t nnz_heavy = 0;            // A entries of the heavy rows
    // symbolic
    int64_t *row_nnz = nullptr;
    int64_t n_slots = 1;
    int n_slots_log2 = 0, slot_width_log2 = 0;
    int64_t *slot = nullptr;
    std::vector<LeafLevel> leaves;
    // value-producing launches of the heavy path in their order, recorded
    // under GMAGNUS_FLAG_KEEP_PATTERN and replayed by gmagnus_update_values
    std::vector<std::function<void(const Csr &, const Csr &, hipStream_t)>> replay;
    bool symbolic_done = false;
    int64_t c_nnz = 0;
    gmagnus_plan_info_t info{};
    std::vector<TimedEvent> timers;
    std::vector<Timed *> open_timers;  // timed scopes open now, innermost last
    bool timing = false;
    bool no_alloc = false;  // workspace from the caller's callbacks only, host reads through pageable memory

    ~gmagnus_plan_s() {
        (void)hipStreamSynchronize(stream);
        if (s_heavy && s_heavy != stream) (void)hipStreamSynchronize(s_heavy);
        if (s_light && s_light != stream) (void)hipStreamSynchronize(s_light);
        for (auto &t : timers) {
            (void)hipEventDestroy(t.a);
            (void)hipEventDestroy(t.b);
        }
        ws.reset();
        if (own_streams) {
            (void)hipStreamDestroy(s_heavy);
            (void)hipStreamDestroy(s_light);
        }
    }
};

namespace {

// Records events around a group of launches of one kernel class. Scopes do
// not overlap in time: opening a scope pauses the one already open (its
// interval ends where the inner one starts and resumes where it ends), and a
// host read pauses every open scope for the time the host waits, so each
// class's time is device time between its own launches, and the classes'
// times add up to no more than the wall time.
struct Timed {
    gmagnus_plan_s *p;
    int cls;
    hipStream_t s;
    hipEvent_t a = nullptr;
    Timed(gmagnus_plan_s *p_, int cls_, hipStream_t s_) : p(p_), cls(cls_), s(s_) {
        if (!p->timing) return;
        if (!p->open_timers.empty()) p->open_timers.back()->pause();
        p->open_timers.push_back(this);
        resume();
    }
    ~Timed() {
        if (!p->timing) return;
        pause();
        p->open_timers.pop_back();
        if (!p->open_timers.empty()) p->open_timers.back()->resume();
    }
    Timed(const Timed &) = delete;
    Timed &operator=(const Timed &) = delete;
    void resume() {
        if (hipEventCreate(&a) != hipSuccess) {
            a = nullptr;
            return;
        }
        if (hipEventRecord(a, s) != hipSuccess) {
            (void)hipEventDestroy(a);
            a = nullptr;
        }
    }
    void pause() {
        if (!a) return;
        hipEvent_t b = nullptr;
        if (hipEventCreate(&b) == hipSuccess && hipEventRecord(b, s) == hipSuccess) {
            p->timers.push_back({cls, a, b});
        } else {
            (void)hipEventDestroy(a);
            if (b) (void)hipEventDestroy(b);
        }
        a = nullptr;
    }
};

// The plan whose entry point is running (set for the duration of each entry
// point that runs a plan's phases): host reads pause its timed scopes, and
// read through pageable memory for plans that must not allocate.
thread_local gmagnus_plan_s *t_plan = nullptr;
struct TimedPlanScope {
    gmagnus_plan_s *prev;
    explicit TimedPlanScope(gmagnus_plan_s *p) : prev(t_plan) { t_plan = p; }
    ~TimedPlanScope() { t_plan = prev; }
};

// Pinned host staging for the small device-to-host reads of counts and bin
// boundaries (a copy into pageable memory goes through the runtime's own
// staging and costs more per read). One buffer per host thread: every read
// has completed when its call returns, so reads never overlap on it. The
// buffer lives until the process ends.
constexpr int READ_SLOTS = 64;

int64_t *read_buffer() {
    thread_local int64_t *buf = nullptr;
    if (!buf) GM_HIP(hipHostMalloc((void **)&buf, sizeof(int64_t) * READ_SLOTS, hipHostMallocDefault));
    return buf;
}

// Several reads, one stream synchronisation: add() queues a copy into the
// staging buffer, wait() synchronises once and copies the values out.
class HostReads {
  public:
    explicit HostReads(hipStream_t s)
        : s_(s), buf_(t_plan && t_plan->no_alloc ? local_ : read_buffer()) {}
    ~HostReads() { resume_timers(); }
    void add(const int64_t *dev, int n, int64_t *host) {
        GM_REQUIRE(used_ + n <= READ_SLOTS && n_ < MAXR, GMAGNUS_ERROR_INVALID_VALUE, "too many host reads at once");
        // the open timed scopes stop before the copies and resume after the host's wait
        if (!tp_ && t_plan && t_plan->timing && !t_plan->open_timers.empty()) {
            tp_ = t_plan;
            tp_->open_timers.back()->pause();  // the innermost scope is the one running
        }
        GM_HIP(hipMemcpyAsync(buf_ + used_, dev, sizeof(int64_t) * n, hipMemcpyDeviceToHost, s_));
        r_[n_++] = Read{host, n, used_};
        used_ += n;
    }
    // whether `reads` more reads of `values` values in all fit before a wait() is needed
    bool room(int values, int reads) const { return used_ + values <= READ_SLOTS && n_ + reads <= MAXR; }
    void wait() {
        GM_HIP(hipStreamSynchronize(s_));
        resume_timers();
        for (int i = 0; i < n_; ++i)
            for (int j = 0; j < r_[i].n; ++j) r_[i].host[j] = buf_[r_[i].at + j];
        n_ = used_ = 0;
    }

  private:
    struct Read {
        int64_t *host;
        int n, at;
    };
    void resume_timers() {
        if (!tp_) return;
        if (!tp_->open_timers.empty()) tp_->open_timers.back()->resume();
        tp_ = nullptr;
    }
    static constexpr int MAXR = 8;
    hipStream_t s_;
    int64_t *buf_;
    Read r_[MAXR];
    int n_ = 0, used_ = 0;
    gmagnus_plan_s *tp_ = nullptr;  // plan whose timed scopes this read paused
    int64_t local_[READ_SLOTS];     // pageable staging (plans that must not allocate)
};

int64_t read_scalar(const int64_t *dev, hipStream_t s) {
    int64_t v = 0;
    HostReads r(s);
    r.add(dev, 1, &v);
    r.wait();
    return v;
}

gmagnus_matrix_t typed_desc(const gmagnus_csr_t *m) {
    gmagnus_matrix_t t{};
    if (m) t = gmagnus_matrix_t{m->n_rows, m->n_cols, m->nnz, m->row_ptr, m->col_idx, m->val, GMAGNUS_INDEX_INT32,
                                GMAGNUS_VALUE_FP64};
    return t;
}

Csr to_csr(const gmagnus_matrix_t *m) {
    Csr c{m->n_rows, m->n_cols, m->nnz, m->row_ptr, m->col_idx, m->val};
    c.ci64 = m->index_type == GMAGNUS_INDEX_INT64;
    c.v32 = m->value_type == GMAGNUS_VALUE_FP32;
    return c;
}

// is_b: the right operand, whose column count (C's) may reach 2^35 with
// int64 indices; every other dimension stays below 2^31.
void check_csr_desc(const gmagnus_matrix_t *m, const char *name, bool is_b) {
    GM_REQUIRE(m != nullptr, GMAGNUS_ERROR_INVALID_VALUE, std::string(name) + " is NULL");
    GM_REQUIRE(m->index_type == GMAGNUS_INDEX_INT32 || m->index_type == GMAGNUS_INDEX_INT64,
               GMAGNUS_ERROR_INVALID_VALUE, std::string(name) + ": unknown index type");
    GM_REQUIRE(m->value_type == GMAGNUS_VALUE_FP64 || m->value_type == GMAGNUS_VALUE_FP32,
               GMAGNUS_ERROR_INVALID_VALUE, std::string(name) + ": unknown value type");
    GM_REQUIRE(m->n_rows >= 0 && m->n_cols >= 0 && m->nnz >= 0, GMAGNUS_ERROR_INVALID_VALUE,
               std::string(name) + ": negative size");
    const bool wide = is_b && m->index_type == GMAGNUS_INDEX_INT64;
    GM_REQUIRE(m->n_rows < ((int64_t)1 << 31) && (wide ? m->n_cols <= max_columns(8) : m->n_cols < ((int64_t)1 << 31)),
               GMAGNUS_ERROR_UNSUPPORTED,
               std::string(name) + (wide ? ": rows must be below 2^31 and columns at most 2^35"
                                         : ": dimensions must be below 2^31"));
    GM_REQUIRE(m->row_ptr != nullptr, GMAGNUS_ERROR_INVALID_VALUE, std::string(name) + ": row_ptr is NULL");
    GM_REQUIRE(m->nnz == 0 || (m->col_idx && m->val), GMAGNUS_ERROR_INVALID_VALUE,
               std::string(name) + ": col_idx/val is NULL");
}

void check_pair(const gmagnus_matrix_t *A, const gmagnus_matrix_t *B) {
    check_csr_desc(A, "A", false);
    check_csr_desc(B, "B", true);
    GM_REQUIRE(A->n_cols == B->n_rows, GMAGNUS_ERROR_INVALID_VALUE, "A.n_cols must equal B.n_rows");
    GM_REQUIRE(A->index_type == B->index_type && A->value_type == B->value_type, GMAGNUS_ERROR_INVALID_VALUE,
               "A and B must have the same index and value types");
}

int64_t index_bytes(int32_t t) { return t == GMAGNUS_INDEX_INT64 ? 8 : 4; }
int64_t value_bytes(int32_t t) { return t == GMAGNUS_VALUE_FP32 ? 4 : 8; }

int64_t lds_bytes_of(const gmagnus_options_t &o) {
    if (o.lds_bytes > 0) return o.lds_bytes;
    int dev = 0, v = 0;
    GM_HIP(hipGetDevice(&dev));
    GM_HIP(hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
    return v;
}

// Reads bin boundaries of a partition into host memory.
void read_bins(const int64_t *dev, int nb, int64_t *host, hipStream_t s) {
    HostReads r(s);
    r.add(dev, nb + 1, host);
    r.wait();
}

// Chooses the multisplit tile (elements) and rows per tile for a level.
void choose_tile(LevelGeom &g, int64_t tau) {
    for (int i = 0; i < multisplit_tile_count(); ++i) {
        const int64_t te = multisplit_tile_elems(i);
        const int64_t rows = (te - 1 + tau - 1) / tau + 1;  // input rows hold more than tau elements
        const int R = (int)ceil_pow2(rows);
        const int keys = R * g.n_chunks;
        if (R <= multisplit_max_rows() && keys <= multisplit_max_keys() &&
            (g.next_chunks == 0 || multisplit_next_fits(keys, g.next_chunks))) {
            g.group_elems = te;
            g.group_rows = R;
            return;
        }
    }
    throw Error{GMAGNUS_ERROR_UNSUPPORTED, "tau too small for the multisplit tile sizes"};
}

__global__ void k_affine(int64_t *p, int64_t n, int64_t a) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = i * a;
}

// Greedy row panels from the row products' prefix sums pre[0..n]: from row
// r a panel ends at the last e with pre[e] - pre[r] <= max_products (one row
// at least). One work group; each search step tests SPLIT_BLOCK evenly
// spaced rows of the remaining range at once (the sums are nondecreasing),
// so a panel takes about log_256(n) steps. out[0] = the panel count (-1 when
// max_panels do not reach row n); out[1 + i] = bound i.
constexpr int SPLIT_BLOCK = 256;

// *out = the longest row of a CSR row-pointer array (out zeroed before).
// One atomic per work group at most, and none when the maximum already
// stored is as large: every wave's atomic on the one word serialised at the
// L2 (16384 of them took 0.19 ms for 2^22 rows).
// out[0] += products of the rows of class LIGHT_HEAVY, out[1] += their A
// entries (out zeroed before): the two sizes the heavy path allocates by,
// read together with the row bins instead of in round trips of their own.
constexpr int HT_BLOCK = 256, HT_GRID = 1024;
__global__ __launch_bounds__(HT_BLOCK) void k_heavy_totals(const uint8_t *cls, const int64_t *ip, const int64_t *rp,
                                                           int64_t n, unsigned long long *out) {
    __shared__ int64_t sm[2][HT_BLOCK / GM_WAVE];
    int64_t prod = 0, ent = 0;
    for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < n; r += (int64_t)gridDim.x * blockDim.x)
        if (cls[r] == LIGHT_HEAVY) {
            prod += ip[r];
            ent += rp[r + 1] - rp[r];
        }
#pragma unroll
    for (int d = GM_WAVE / 2; d >= 1; d >>= 1) {
        prod += __shfl_xor(prod, d, GM_WAVE);
        ent += __shfl_xor(ent, d, GM_WAVE);
    }
    if ((threadIdx.x & (GM_WAVE - 1)) == 0) {
        sm[0][threadIdx.x / GM_WAVE] = prod;
        sm[1][threadIdx.x / GM_WAVE] = ent;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < HT_BLOCK / GM_WAVE; ++w) {
            prod += sm[0][w];
            ent += sm[1][w];
        }
        if (prod) atomicAdd(&out[0], (unsigned long long)prod);
        if (ent) atomicAdd(&out[1], (unsigned long long)ent);
    }
}

constexpr int MAXLEN_BLOCK = 256, MAXLEN_GRID = 1024;
__global__ __launch_bounds__(MAXLEN_BLOCK) void k_max_row_len(const int64_t *rp, int64_t n_rows,
                                                             unsigned long long *out) {
    __shared__ int64_t wmax[MAXLEN_BLOCK / GM_WAVE];
    int64_t m = 0;
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n_rows; k += (int64_t)gridDim.x * blockDim.x) {
        const int64_t len = rp[k + 1] - rp[k];
        m = len > m ? len : m;
    }
#pragma unroll
    for (int d = GM_WAVE / 2; d >= 1; d >>= 1) {
        const int64_t o = __shfl_xor(m, d, GM_WAVE);
        m = o > m ? o : m;
    }
    if ((threadIdx.x & (GM_WAVE - 1)) == 0) wmax[threadIdx.x / GM_WAVE] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 1; w < MAXLEN_BLOCK / GM_WAVE; ++w) m = wmax[w] > m ? wmax[w] : m;
        if (m > 0 && (unsigned long long)m > __hip_atomic_load(out, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
            atomicMax(out, (unsigned long long)m);
    }
}

__global__ __launch_bounds__(SPLIT_BLOCK) void k_split_panels(const int64_t *pre, int64_t n, int64_t max_products,
                                                              int64_t max_panels, int64_t *out) {
    __shared__ int best;
    const int t = threadIdx.x;
    int64_t r = 0, cnt = 0;
    if (t == 0) out[1] = 0;
    while (r < n && cnt < max_panels) {
        // saturated: a limit near INT64_MAX means "no limit"
        const int64_t target = max_products > INT64_MAX - pre[r] ? INT64_MAX : pre[r] + max_products;
        int64_t lo = r + 1, hi = n, e = r;  // the answer is the last e in [lo, hi] with pre[e] <= target, else r
        while (lo <= hi) {
            const int64_t span = hi - lo + 1;
            const bool ok = pre[lo + span * t / SPLIT_BLOCK] <= target;
            if (t == 0) best = -1;
            __syncthreads();
            if (ok) atomicMax(&best, t);
            __syncthreads();
            const int b = best;
            __syncthreads();
            if (b < 0) break;  // pre[lo] is past the target
            e = lo + span * b / SPLIT_BLOCK;
            const int64_t next = b + 1 < SPLIT_BLOCK ? lo + span * (b + 1) / SPLIT_BLOCK : hi + 1;
            lo = e + 1;
            hi = next - 1;
        }
        if (e <= r) e = r + 1;
        ++cnt;
        if (t == 0) out[1 + cnt] = e;
        r = e;
    }
    if (t == 0) out[0] = r < n ? -1 : cnt;
}

__global__ void k_copy_i64(int64_t *dst, const int64_t *src, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        dst[i] = src[i];
}

void copy_i64(int64_t *dst, const int64_t *src, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_copy_i64, dim3(grid_for(n, 256, 65536)), dim3(256), 0, s, dst, src, n);
    GM_CHECK_LAUNCH();
}

// *dst = src[*at]: a value whose index is itself on the device, fetched
// there so that both come back in one host read
__global__ void k_pick_i64(const int64_t *src, const int64_t *at, int64_t *dst) { *dst = src[*at]; }

void pick_i64(const int64_t *src, const int64_t *at, int64_t *dst, hipStream_t s) {
    hipLaunchKernelGGL(k_pick_i64, dim3(1), dim3(1), 0, s, src, at, dst);
    GM_CHECK_LAUNCH();
}

// ----------------------------------------------------------- plan phases
void do_plan(gmagnus_plan_s *p, const gmagnus_matrix_t *A, const gmagnus_matrix_t *B, const gmagnus_options_t *opts,
             hipStream_t stream) {
    check_pair(A, B);
    if (opts) {
        GM_REQUIRE(opts->struct_size == sizeof(gmagnus_options_t), GMAGNUS_ERROR_INVALID_VALUE,
                   "options.struct_size mismatch");
        GM_REQUIRE((opts->alloc == nullptr) == (opts->free == nullptr), GMAGNUS_ERROR_INVALID_VALUE,
                   "alloc and free callbacks must be given together");
        p->opts = *opts;
    } else {
        gmagnus_options_init(&p->opts);
    }
    const gmagnus_options_t &o = p->opts;
    p->A = to_csr(A);
    p->B = to_csr(B);
    p->r0 = o.row_begin;
    p->r1 = o.row_end > 0 ? o.row_end : A->n_rows;
    GM_REQUIRE(p->r0 >= 0 && p->r0 <= p->r1 && p->r1 <= A->n_rows, GMAGNUS_ERROR_INVALID_VALUE, "bad row panel");
    p->n = p->r1 - p->r0;
    p->stream = stream;
    p->timing = (o.flags & GMAGNUS_FLAG_TIMING) != 0;
    if ((o.flags & GMAGNUS_FLAG_CONCURRENT_STREAMS) == 0 || (o.flags & GMAGNUS_FLAG_SERIAL_STREAMS)) {
        p->s_heavy = p->s_light = stream;
    } else {
        GM_HIP(hipStreamCreateWithFlags(&p->s_heavy, hipStreamNonBlocking));
        GM_HIP(hipStreamCreateWithFlags(&p->s_light, hipStreamNonBlocking));
        p->own_streams = true;
    }
    p->csize = index_bytes(A->index_type);
    p->vsize = value_bytes(A->value_type);
    p->info.index_type = A->index_type;
    p->info.value_type = A->value_type;
    compute_params(std::max<int64_t>(B->n_cols, 1), lds_bytes_of(o), p->csize, p->vsize, &o, &p->params);
    p->ws.reset(new Workspace(&o, stream));
    Workspace &ws = *p->ws;
    p->err = ws.alloc<int32_t>(1);
    fill<int32_t>(p->err, 0, 1, stream);

    if (o.validate) {
        int32_t *flag = ws.alloc<int32_t>(2);
        validate_csr(p->A, flag, stream);
        validate_csr(p->B, flag + 1, stream);
        int32_t f[2];
        GM_HIP(hipMemcpyAsync(f, flag, sizeof(f), hipMemcpyDeviceToHost, stream));
        GM_HIP(hipStreamSynchronize(stream));
        GM_REQUIRE(f[0] == 0, GMAGNUS_ERROR_INVALID_CSR, "A is not canonical CSR (flags " + std::to_string(f[0]) + ")");
        GM_REQUIRE(f[1] == 0, GMAGNUS_ERROR_INVALID_CSR, "B is not canonical CSR (flags " + std::to_string(f[1]) + ")");
    }
    const int64_t n = p->n;
    p->info.n_rows = n;
    p->info.params = p->params;
    p->info.row_tau = std::min(p->params.tau, light_row_limit());
    if (n == 0) return;

    int64_t rp2[2] = {0, 0};
    {
        HostReads r(stream);
        r.add(A->row_ptr + p->r0, 1, &rp2[0]);
        r.add(A->row_ptr + p->r1, 1, &rp2[1]);
        r.wait();
    }
    const int64_t panel_nnz = rp2[1] - rp2[0];

    Timed t(p, GMAGNUS_K_SETUP, stream);
    p->ip = ws.alloc<int64_t>(n);
    p->minc = ws.alloc_bytes(p->csize * n);
    p->maxc = ws.alloc_bytes(p->csize * n);
    {
        // many more A entries than B rows: summarize B's rows once (length, first
        // and last column), one random read per A entry instead of three
        void *binfo = panel_nnz >= 4 * p->B.n_rows ? ws.alloc_bytes(brow_info_bytes(p->B)) : nullptr;
        row_products(p->A, p->B, p->r0, p->r1, panel_nnz, p->ip, p->minc, p->maxc, stream, binfo);
        ws.free(binfo);
    }
    const bool window = (o.flags & GMAGNUS_FLAG_NO_WINDOW) == 0;
    uint8_t *cls = ws.alloc<uint8_t>(n);
    light_classes_sym(p->ip, p->minc, p->maxc, p->B.ci64, n, p->info.row_tau, window, cls, stream);
    p->perm = ws.alloc<int64_t>(n);
    int64_t *bins = ws.alloc<int64_t>(LIGHT_NBINS + 1);
    int64_t *scratch = ws.alloc<int64_t>(std::max(partition_scratch_elems(n, LIGHT_NBINS), scan_scratch_elems(n)));
    partition_u8(cls, n, LIGHT_NBINS, p->perm, nullptr, bins, scratch, stream);
    // products of all rows and of the heavy rows (C-hat row pointers)
    int64_t *ip_scan = ws.alloc<int64_t>(n + 1);
    scan_i64(p->ip, n, ip_scan, scratch, stream);
    int64_t *heavy_tot = ws.alloc<int64_t>(2);
    fill<int64_t>(heavy_tot, 0, 2, stream);
    hipLaunchKernelGGL(k_heavy_totals, dim3(grid_for(n, HT_BLOCK, HT_GRID)), dim3(HT_BLOCK), 0, stream, cls, p->ip,
                       p->A.rp + p->r0, n, (unsigned long long *)heavy_tot);
    GM_CHECK_LAUNCH();
    {
        int64_t tot[2] = {0, 0};
        HostReads r(stream);
        r.add(bins, LIGHT_NBINS + 1, p->bins_sym);
        r.add(ip_scan + n, 1, &p->products_total);
        r.add(heavy_tot, 2, tot);
        r.wait();
        p->products_heavy = tot[0];
        p->nnz_heavy = tot[1];
    }
    p->n_heavy = p->bins_sym[LIGHT_HEAVY + 1] - p->bins_sym[LIGHT_HEAVY];
    p->heavy_rows = p->perm + p->bins_sym[LIGHT_HEAVY];
    p->chat_ptr = ws.alloc<int64_t>(p->n_heavy + 1);
    scan_gather_i64(p->ip, p->heavy_rows, p->n_heavy, p->chat_ptr, scratch, stream);
    ws.free(heavy_tot);
    ws.free(ip_scan);
    ws.free(scratch);
    ws.free(cls);
    p->info.n_heavy_rows = p->n_heavy;
    p->info.n_light_rows = p->bins_sym[LIGHT_NBINS] - p->bins_sym[LIGHT_W0];
    p->info.products_total = p->products_total;
    p->info.products_heavy = p->products_heavy;
}

void add_bytes(gmagnus_plan_s *p, int cls, double bytes) { p->info.kernel_bytes[cls] += bytes; }

}  // namespace

namespace gm {
// Which expansion the heavy rows take (gmagnus_expansion_path). Without a
// multisplit level, with 64 or more first-level chunks, or when the paper's
// order is asked for, C-hat is written row by row (Algorithm 4); otherwise the first level is split during the
// expansion: in chunk-major row order when the offsets inside a (chunk, row)
// region fit 32 bits, else in slice order. A hierarchy of exactly two levels
// runs both levels inside the row-order expansion when its keys fit the work
// group's LDS and B's entries can be indexed in 32 bits (the fine boundaries).
int32_t expansion_path(const gmagnus_params_t &P, int64_t n_heavy, int64_t products_heavy, int64_t b_nnz,
                       int32_t flags) {
    if (n_heavy <= 0) return GMAGNUS_PATH_NONE;
    const bool paper_hist = (flags & GMAGNUS_FLAG_PAPER_HISTOGRAM) != 0;
    // the fused first-level split handles up to 63 chunks (one lane per chunk boundary)
    const bool fused = P.n_levels > 0 && P.v_chunks[0] < GM_WAVE && !paper_hist &&
                       (flags & GMAGNUS_FLAG_PAPER_EXPANSION) == 0;
    if (!fused) return GMAGNUS_PATH_PAPER;
    const bool rows_order = (flags & GMAGNUS_FLAG_SLICE_SPLIT) == 0 && products_heavy < ((int64_t)1 << 32) &&
                            n_heavy < ((int64_t)1 << 31);
    if (!rows_order) return GMAGNUS_PATH_SLICE_SPLIT;
    const bool two = P.n_levels == 2 && (flags & GMAGNUS_FLAG_LEVEL_BY_LEVEL) == 0 && b_nnz < ((int64_t)1 << 31) &&
                     rows2_fits(P.tau, P.v_chunks[1], P.v_chunks[0] * P.v_chunks[1]);
    return two ? GMAGNUS_PATH_ROWS_TWO_LEVEL : GMAGNUS_PATH_ROWS;
}
}  // namespace gm

namespace {

// Heavy path of the symbolic phase: masked CSC, expansion, multisplit
// levels, final-chunk symbolic, fragment offsets. Runs on p->s_heavy.
void heavy_symbolic(gmagnus_plan_s *p) {
    Workspace &ws = *p->ws;
    const hipStream_t s = p->s_heavy;
    const int64_t nh = p->n_heavy;
    const gmagnus_params_t &P = p->params;
    const int64_t H = p->products_heavy;
    const int c_bits = ilog2(ceil_pow2(std::max<int64_t>(p->B.n_cols, 1)));
    p->n_slots = P.n_levels > 0 ? P.chunks_required : 1;
    p->n_slots_log2 = ilog2(p->n_slots);
    p->slot_width_log2 = c_bits - p->n_slots_log2;
    // With a kept pattern nothing is freed (every buffer a recorded step
    // reads stays valid) and each value-producing step is recorded; the
    // steps reset the cursors they consume, so a replay repeats them exactly.
    const bool keep = (p->opts.flags & GMAGNUS_FLAG_KEEP_PATTERN) != 0;
    ws.hold(keep);
    struct Unhold {
        Workspace &w;
        ~Unhold() { w.hold(false); }
    } unhold{ws};
    auto values_step = [&](std::function<void(const Csr &, const Csr &, hipStream_t)> f) {
        f(p->A, p->B, s);
        if (keep) p->replay.push_back(std::move(f));
    };
    const int64_t *heavy_rows = p->heavy_rows;
    const int64_t r0 = p->r0;

    const bool paper_hist = (p->opts.flags & GMAGNUS_FLAG_PAPER_HISTOGRAM) != 0;
    const int32_t path = expansion_path(P, nh, H, p->B.nnz, p->opts.flags);
    p->info.expansion_path = path;
    GM_REQUIRE(path != GMAGNUS_PATH_PAPER || p->B.n_cols < ((int64_t)1 << 31), GMAGNUS_ERROR_UNSUPPORTED,
               "C-hat row by row holds whole columns: with 2^31 or more columns of C the first level must be split "
               "during the expansion (no paper-order flags, at most 63 first-level chunks)");
    const int64_t VS = p->vsize;   // bytes of a value
    const double CS = (double)p->csize;  // bytes of a column index of A, B and C (internal columns take 4 or 2)
    // split at the first level while expanding, unless the paper's order is asked for
    const bool fused = path != GMAGNUS_PATH_PAPER;
    // the fused split in chunk-major row order (32-bit offsets inside a row's chunk), else in slice order
    const bool rows_order = path == GMAGNUS_PATH_ROWS || path == GMAGNUS_PATH_ROWS_TWO_LEVEL;
    // a hierarchy of exactly two levels in one pass: the expansion splits its
    // heavy regions again and writes the final chunks directly
    const bool two_level = path == GMAGNUS_PATH_ROWS_TWO_LEVEL;
    int64_t *counts0 = nullptr;  // level-0 counts when computed from the structure
    int32_t *sbnd = nullptr;     // per-slice level-0 chunk boundaries (kept for the fused expansion)
    RowEntries ent;              // chunk-major row order: entries, their chunk offsets, the row pointers of A~
    uint2 *pb = nullptr;         // chunk-major offsets of the entries' chunk parts (region, B row)
    int64_t *a_heavy_keep = nullptr;

    // ---- masked CSR -> CSC of the heavy rows and slice offsets
    SliceArrays sl;
    int64_t *row_len, *a_heavy_ptr, *scratch;
    int64_t nnz_heavy_all = 0, blen_total = 0;
    {
        Timed t(p, GMAGNUS_K_CSC, s);
        row_len = ws.alloc<int64_t>(nh);
        a_heavy_ptr = ws.alloc<int64_t>(nh + 1);
        const int64_t n_k = p->A.n_cols;
        scratch = ws.alloc<int64_t>(std::max({scan_scratch_elems(std::max(nh, n_k)), partition_scratch_elems(n_k, 2),
                                              (int64_t)16}));
        gather_row_len(p->A.rp, p->heavy_rows, nh, p->r0, row_len, s);
        scan_i64(row_len, nh, a_heavy_ptr, scratch, s);
        nnz_heavy_all = p->nnz_heavy;  // summed over the same rows at plan time (checked below)
        int64_t *colcnt = ws.alloc<int64_t>(n_k);
        csc_count(p->A, p->B, p->heavy_rows, nh, p->r0, a_heavy_ptr, nnz_heavy_all, colcnt, s);
        uint8_t *kcls = ws.alloc<uint8_t>(n_k);
        slice_flags(p->B, colcnt, n_k, kcls, s);
        int64_t *kperm = ws.alloc<int64_t>(n_k);
        int64_t *kb = ws.alloc<int64_t>(3);
        partition_u8(kcls, n_k, 2, kperm, nullptr, kb, scratch, s);
        int64_t kbh[3];
        read_bins(kb, 2, kbh, s);
        sl.n_slices = kbh[1];
        sl.slice_k = ws.alloc<int32_t>(sl.n_slices);
        int64_t *cnt_s = ws.alloc<int64_t>(sl.n_slices);
        int64_t *ip_s = ws.alloc<int64_t>(sl.n_slices);
        int32_t *k_to_slice = ws.alloc<int32_t>(p->B.n_rows);
        slice_build(p->B, colcnt, kperm, sl.n_slices, sl.slice_k, cnt_s, ip_s, k_to_slice, s);
        sl.col_ptr = ws.alloc<int64_t>(sl.n_slices + 1);
        sl.slice_off = ws.alloc<int64_t>(sl.n_slices + 1);
        int64_t *sc2 = ws.alloc<int64_t>(scan_scratch_elems(sl.n_slices));
        scan_i64(cnt_s, sl.n_slices, sl.col_ptr, sc2, s);
        scan_i64(ip_s, sl.n_slices, sl.slice_off, sc2, s);
        // B~: the B rows of the slices, each read once at least (compulsory bytes)
        int64_t *blen_scan = ws.alloc<int64_t>(sl.n_slices + 1);
        slice_lengths(p->B, sl.slice_k, sl.n_slices, cnt_s, s);
        scan_i64(cnt_s, sl.n_slices, blen_scan, sc2, s);
        int64_t tot[4];
        {
            HostReads r(s);
            r.add(sl.col_ptr + sl.n_slices, 1, &tot[0]);
            r.add(sl.slice_off + sl.n_slices, 1, &tot[1]);
            r.add(blen_scan + sl.n_slices, 1, &tot[2]);
            r.add(a_heavy_ptr + nh, 1, &tot[3]);
            r.wait();
        }
        ws.free(blen_scan);
        sl.nnz = tot[0];
        blen_total = tot[2];
        GM_REQUIRE(tot[1] == H, GMAGNUS_ERROR_HIP, "slice products disagree with the row products");
        GM_REQUIRE(tot[3] == nnz_heavy_all, GMAGNUS_ERROR_HIP, "heavy rows' entries disagree with the plan's count");
        int64_t *cursor = nullptr;
        if (!rows_order) {
            cursor = ws.alloc<int64_t>(std::max<int64_t>(sl.n_slices, 1));
            sl.row_h = ws.alloc<int32_t>(sl.nnz);
            sl.a_val = ws.alloc_bytes(VS * sl.nnz);
            values_step([=](const Csr &A, const Csr &B, hipStream_t st) {
                fill<int64_t>(cursor, 0, sl.n_slices, st);
                csc_fill(A, B, heavy_rows, nh, r0, a_heavy_ptr, nnz_heavy_all, k_to_slice, sl.col_ptr, cursor,
                         sl.row_h, sl.a_val, st);
            });
        } else {
            ent.k = ws.alloc<int32_t>(nnz_heavy_all);
            ent.s = ws.alloc<int32_t>(nnz_heavy_all);
            ent.h = ws.alloc<int32_t>(nnz_heavy_all);
            ent.b0 = ws.alloc<int64_t>(nnz_heavy_all);
            ent.a = ws.alloc_bytes(VS * nnz_heavy_all);
            values_step([=](const Csr &A, const Csr &B, hipStream_t st) {
                heavy_entries(A, B, heavy_rows, nh, r0, a_heavy_ptr, nnz_heavy_all, k_to_slice, ent, st);
            });
        }
        if (P.n_levels > 0 && !paper_hist) {
            // level-0 (row, chunk) counts from the structure of A~ and B
            Timed t2(p, GMAGNUS_K_HISTOGRAM, s);
            const int nc0 = P.v_chunks[0];
            const int shift0 = c_bits - ilog2(nc0);
            sbnd = ws.alloc<int32_t>(sl.n_slices * (nc0 + 1));
            counts0 = ws.alloc<int64_t>(nh * nc0);
            slice_chunk_bounds(p->B, sl, nc0, shift0, sbnd, s);
            struct_hist(p->A, p->heavy_rows, nh, p->r0, a_heavy_ptr, nnz_heavy_all, k_to_slice, sbnd, nc0, rows_order,
                        counts0, s);
            if (rows_order) {
                // every entry's offset inside its (chunk, row) region
                const int64_t nw = entry_offset_waves(nnz_heavy_all);
                int64_t *agg = ws.alloc<int64_t>(nw * nc0), *carry = ws.alloc<int64_t>(nw * nc0);
                int32_t *wfirst = ws.alloc<int32_t>(nw), *wlast = ws.alloc<int32_t>(nw);
                pb = ws.alloc<uint2>(nnz_heavy_all * nc0);
                entry_offsets(ent, nnz_heavy_all, sbnd, nc0, agg, wfirst, wlast, carry, pb, s);
                ws.free(agg);
                ws.free(carry);
                ws.free(wfirst);
                ws.free(wlast);
                add_bytes(p, GMAGNUS_K_HISTOGRAM, 8.0 * nnz_heavy_all + 8.0 * nnz_heavy_all * nc0);
            }
            if (!fused) {
                ws.free(sbnd);
                sbnd = nullptr;
            }
            p->info.kernel_launches[GMAGNUS_K_HISTOGRAM] += 1;
            add_bytes(p, GMAGNUS_K_HISTOGRAM, (CS + 8.0) * nnz_heavy_all + 4.0 * sl.n_slices * (nc0 + 1) + 8.0 * nh * nc0);
        }
        ws.free(cursor);
        ws.free(colcnt);
        ws.free(kcls);
        ws.free(kperm);
        ws.free(kb);
        ws.free(cnt_s);
        ws.free(ip_s);
        ws.free(k_to_slice);
        ws.free(sc2);
        ws.free(row_len);
        if (rows_order)
            a_heavy_keep = a_heavy_ptr;  // region records need the row pointers of A~
        else
            ws.free(a_heavy_ptr);
        ws.free(scratch);
        add_bytes(p, GMAGNUS_K_CSC, (CS + VS) * nnz_heavy_all + (4.0 + VS) * sl.nnz + 8.0 * (p->A.n_cols + sl.n_slices));
    }
    p->info.n_slices = sl.n_slices;
    p->info.nnz_a_heavy = sl.nnz;

    // ---- outer-product expansion into buffer 0 (C-hat row by row, or
    // already split into the first level's chunks when fused)
    int32_t *col_buf[2] = {ws.alloc<int32_t>(H), nullptr};
    void *val_buf[2] = {ws.alloc_bytes(VS * H), nullptr};
    int64_t *exp_tiles =
        ws.alloc<int64_t>(std::max<int64_t>(rows_order ? rows_tile_words(H) : expand_tile_words(H), 1));
    if (!rows_order) {
        Timed t(p, GMAGNUS_K_CSC, s);
        expand_tiles(p->B, sl, H, exp_tiles, s);
    }
    auto free_slices = [&]() {
        ws.free(exp_tiles);
        ws.free(sl.col_ptr);
        ws.free(sl.slice_off);
        ws.free(sl.slice_k);
        ws.free(sl.row_h);
        ws.free(sl.a_val);
        ws.free(ent.k);
        ws.free(ent.s);
        ws.free(ent.h);
        ws.free(ent.b0);
        ws.free(ent.a);
        ws.free(pb);
        ws.free(a_heavy_keep);
        if (sbnd) ws.free(sbnd);
        sbnd = nullptr;
    };
    if (!fused) {
        int64_t *cursor = ws.alloc<int64_t>(nh);
        {
            Timed t(p, GMAGNUS_K_EXPAND, s);
            const int64_t *chat_ptr = p->chat_ptr;
            int32_t *oc = col_buf[0];
            void *ov = val_buf[0];
            values_step([=](const Csr &, const Csr &B, hipStream_t st) {
                copy_i64(cursor, chat_ptr, nh, st);
                expand(B, sl, H, exp_tiles, cursor, oc, ov, st);
            });
        }
        ws.free(cursor);
        p->info.kernel_launches[GMAGNUS_K_EXPAND] += 1;
        add_bytes(p, GMAGNUS_K_EXPAND, (4.0 + VS) * H + (4.0 + VS) * sl.nnz + (CS + VS) * blen_total + 8.0 * nh);
        free_slices();
    }

    // ---- hierarchical multisplit
    int64_t *origin_in = ws.alloc<int64_t>(nh);
    hipLaunchKernelGGL(k_affine, dim3(grid_for(nh, 256, 65536)), dim3(256), 0, s, origin_in, nh, p->n_slots);
    GM_CHECK_LAUNCH();
    const int64_t *in_ptr = p->chat_ptr;
    int64_t n_in = nh, elems = H;
    int cur = 0;
    int m_in_log2 = c_bits;
    int64_t *counts = nullptr;
    p->leaves.clear();
    if (P.n_levels == 0) {
        LeafLevel lv;
        lv.set = LeafSet{p->chat_ptr, col_buf[0], val_buf[0], origin_in, 0, nh};
        lv.set.v32 = p->B.v32;
        lv.width = (int64_t)1 << c_bits;
        lv.elems = H;
        p->leaves.push_back(lv);
    }
    int64_t slots_per_chunk = p->n_slots;
    LeafLevel two_done{};  // the second level's final chunks when both levels run in one pass
    for (int lvl = 0; lvl < P.n_levels; ++lvl) {
        const int nc = P.v_chunks[lvl];
        const bool last = lvl == P.n_levels - 1;
        LevelGeom g{};
        g.n_in = n_in;
        g.elems = elems;
        g.n_chunks = nc;
        g.shift = m_in_log2 - ilog2(nc);
        g.next_chunks = last ? 0 : P.v_chunks[lvl + 1];
        g.next_shift = last ? 0 : g.shift - ilog2(g.next_chunks);
        choose_tile(g, P.tau);
        p->info.level_rows_in[lvl] = n_in;
        p->info.level_elems_in[lvl] = elems;
        slots_per_chunk /= nc;

        const int64_t n_tiles = (elems + g.group_elems - 1) / g.group_elems;
        int64_t *tile_row = ws.alloc<int64_t>(n_tiles);
        const int64_t n_out = n_in * nc;
        int64_t *sc = ws.alloc<int64_t>(std::max(partition_scratch_elems(n_out, 2), scan_scratch_elems(n_out)));
        int64_t *x_map = ws.alloc<int64_t>(n_out);
        int64_t *perm2 = ws.alloc<int64_t>(n_out);
        int64_t *cb = ws.alloc<int64_t>(4);  // class bounds, then the heavy chunks' element count
        int64_t *out_cnt = ws.alloc<int64_t>(n_out);
        int64_t *origin_out = ws.alloc<int64_t>(n_out);
        int64_t *out_ptr = ws.alloc<int64_t>(n_out + 1);
        uint8_t *ccls = ws.alloc<uint8_t>(n_out);
        if (!(fused && lvl == 0)) tile_rows(g, in_ptr, tile_row, s);
        if (lvl == 0 && counts0) {
            counts = counts0;
        } else if (!counts) {
            // the paper's histogram kernel: one pass over the level's input
            // columns (C-hat at the first level; after a fused first split,
            // the chunks that stay heavy)
            Timed t(p, GMAGNUS_K_HISTOGRAM, s);
            counts = ws.alloc<int64_t>(n_out);
            int64_t *h_rows = ws.alloc<int64_t>(std::max<int64_t>(histogram_tiles(g, P.tau), 1));
            histogram(g, P.tau, in_ptr, col_buf[cur], h_rows, counts, s);
            ws.free(h_rows);
            p->info.kernel_launches[GMAGNUS_K_HISTOGRAM] += 1;
            add_bytes(p, GMAGNUS_K_HISTOGRAM, 4.0 * elems + 8.0 * (n_in + 1) + 8.0 * n_out);
        }
        int64_t cbh[4];
        {
            Timed t(p, GMAGNUS_K_SETUP, s);
            chunk_classes(counts, n_out, P.tau, last, ccls, s);
            partition_u8(ccls, n_out, 2, perm2, x_map, cb, sc, s);
            chunk_reorder(counts, x_map, n_out, nc, origin_in, slots_per_chunk, (rows_order && lvl == 0) ? nh : 0,
                          out_cnt, origin_out, s);
            scan_i64(out_cnt, n_out, out_ptr, sc, s);
            pick_i64(out_ptr, cb + 1, cb + 3, s);  // out_ptr[nh_out]: the heavy chunks hold the first places
            read_bins(cb, 3, cbh, s);
        }
        const int64_t nh_out = cbh[1];
        p->info.level_heavy_out[lvl] = nh_out;
        const bool split_in_expand = fused && lvl == 0;
        int64_t *next_counts = nullptr;
        const bool next_fused = split_in_expand ? rows_order && !two_level && rows_next_fits(g.next_chunks)
                                                : multisplit_next_fits(g.group_rows * nc, g.next_chunks);
        if (!last && nh_out > 0 && next_fused) {
            // the multisplit (or the chunk-major expansion) takes the next level's histogram on the way
            next_counts = ws.alloc<int64_t>(nh_out * g.next_chunks);  // zeroed by the step that fills it
        }
        const int nxt = split_in_expand ? 0 : 1 - cur;
        if (!col_buf[nxt]) {
            col_buf[nxt] = ws.alloc<int32_t>(H);
            val_buf[nxt] = ws.alloc_bytes(VS * H);
        }
        if (split_in_expand && rows_order) {
            // chunk-major regions: chunk, first entry and entry count of each, segment bases
            int32_t *reg_c = ws.alloc<int32_t>(n_out);
            int64_t *reg_efirst = ws.alloc<int64_t>(n_out), *reg_ne = ws.alloc<int64_t>(n_out);
            int64_t *seg_base = ws.alloc<int64_t>(n_out + 1);
            {
                Timed t(p, GMAGNUS_K_SETUP, s);
                region_records(perm2, n_out, nh, a_heavy_keep, reg_c, reg_efirst, reg_ne, s);
                scan_i64(reg_ne, n_out, seg_base, sc, s);
            }
            if (two_level && nh_out > 0) {
                // second level laid out from the structure, then one pass writes both
                const int nc1 = P.v_chunks[1];
                const int nf = nc * nc1;
                const int shift1 = g.shift - ilog2(nc1);
                const int64_t n_out1 = nh_out * nc1;
                const int64_t slots1 = slots_per_chunk / nc1;
                int64_t *counts1 = ws.alloc<int64_t>(n_out1);
                {
                    Timed t(p, GMAGNUS_K_HISTOGRAM, s);
                    int32_t *bndf = ws.alloc<int32_t>(fine_bounds_words(sl.n_slices, nf));
                    int64_t *F = ws.alloc<int64_t>(nh * nf);
                    fine_bounds(p->B, sl.slice_k, sl.n_slices, nf, shift1, sbnd, nc, bndf, s);
                    fine_counts(p->B, ent, nnz_heavy_all, bndf, nf, shift1, nh, F, s);
                    level1_counts(perm2, nh_out, nh, F, nf, nc1, counts1, s);
                    ws.free(bndf);
                    ws.free(F);
                    p->info.kernel_launches[GMAGNUS_K_HISTOGRAM] += 1;
                    // B rows of the slices; fine boundaries written and read once per
                    // entry; per-row fine counts; the heavy regions' counts
                    add_bytes(p, GMAGNUS_K_HISTOGRAM, CS * blen_total + 4.0 * (nf + 1) * sl.n_slices +
                                                          (8.0 + 4.0 * (nf + 1)) * nnz_heavy_all + 8.0 * nh * nf +
                                                          16.0 * n_out1);
                }
                uint8_t *ccls1 = ws.alloc<uint8_t>(n_out1);
                int64_t *sc1 = ws.alloc<int64_t>(std::max(partition_scratch_elems(n_out1, 2), scan_scratch_elems(n_out1)));
                int64_t *perm1 = ws.alloc<int64_t>(n_out1), *x_map1 = ws.alloc<int64_t>(n_out1);
                int64_t *cb1 = ws.alloc<int64_t>(3);
                int64_t *out_cnt1 = ws.alloc<int64_t>(n_out1);
                int64_t *origin_out1 = ws.alloc<int64_t>(n_out1);
                int64_t *out_ptr1 = ws.alloc<int64_t>(n_out1 + 1);
                int64_t *cursor1 = ws.alloc<int64_t>(n_out1);
                int64_t elems1 = 0;
                {
                    Timed t(p, GMAGNUS_K_SETUP, s);
                    chunk_classes(counts1, n_out1, P.tau, true, ccls1, s);
                    partition_u8(ccls1, n_out1, 2, perm1, x_map1, cb1, sc1, s);
                    chunk_reorder(counts1, x_map1, n_out1, nc1, origin_out, slots1, 0, out_cnt1, origin_out1, s);
                    scan_i64(out_cnt1, n_out1, out_ptr1, sc1, s);
                    elems1 = cbh[3];
                }
                // sized like the first level's buffers, so panels reuse the same blocks
                col_buf[1] = ws.alloc<int32_t>(H);
                val_buf[1] = ws.alloc_bytes(VS * H);
                {
                    Timed t(p, GMAGNUS_K_EXPAND, s);
                    int32_t *oc0 = col_buf[0], *oc1 = col_buf[1];
                    void *ov0 = val_buf[0], *ov1 = val_buf[1];
                    const int shift0 = g.shift;
                    const int64_t tau = P.tau;
                    int32_t *err = p->err;
                    values_step([=](const Csr &, const Csr &B, hipStream_t st) {
                        // the second level's cursors start at its regions' offsets
                        gather_i64(out_ptr1, x_map1, n_out1, cursor1, st);
                        expand_rows2(B, ent, pb, nnz_heavy_all, out_ptr, seg_base, reg_c, reg_efirst, reg_ne, n_out,
                                     nh_out, H, nc, shift0, nc1, shift1, tau, cursor1, elems1, err, exp_tiles, oc0,
                                     ov0, (uint16_t *)oc1, ov1, st);
                    });
                }
                p->info.kernel_launches[GMAGNUS_K_EXPAND] += 1;
                // products (the final chunks' columns in 16 bits), entries (B row start,
                // value), their chunk offsets (region, B row), B rows, row records
                add_bytes(p, GMAGNUS_K_EXPAND, (4.0 + VS) * H - 2.0 * elems1 + (8.0 + VS) * nnz_heavy_all +
                                                   8.0 * nnz_heavy_all * nc + (CS + VS) * blen_total + 24.0 * n_out +
                                                   8.0 * n_out1);
                p->info.level_rows_in[1] = nh_out;
                p->info.level_elems_in[1] = elems1;
                p->info.level_heavy_out[1] = 0;
                two_done.set = LeafSet{out_ptr1, nullptr, val_buf[1], origin_out1, 0, n_out1, (const uint16_t *)col_buf[1]};
                two_done.set.v32 = p->B.v32;
                two_done.width = (int64_t)1 << shift1;
                two_done.elems = elems1;
                ws.free(counts1);
                ws.free(ccls1);
                ws.free(sc1);
                ws.free(perm1);
                ws.free(x_map1);
                ws.free(cb1);
                ws.free(out_cnt1);
                ws.free(cursor1);
            } else {
                Timed t(p, GMAGNUS_K_EXPAND, s);
                const int nn = last ? 0 : g.next_chunks, nshift = g.next_shift, shift0 = g.shift;
                int32_t *oc = col_buf[nxt];
                void *ov = val_buf[nxt];
                values_step([=](const Csr &, const Csr &B, hipStream_t st) {
                    if (next_counts) fill<int64_t>(next_counts, 0, nh_out * nn, st);
                    expand_rows(B, ent, pb, nnz_heavy_all, out_ptr, seg_base, reg_c, reg_efirst, reg_ne, n_out,
                                nh_out, H, nc, shift0, nn, nshift, next_counts, exp_tiles, oc, ov, st);
                });
                p->info.kernel_launches[GMAGNUS_K_EXPAND] += 1;
                add_bytes(p, GMAGNUS_K_EXPAND,
                          (4.0 + VS) * H + (8.0 + VS) * nnz_heavy_all + 8.0 * nnz_heavy_all * nc +
                              (CS + VS) * blen_total + 24.0 * n_out);
            }
            ws.free(reg_c);
            ws.free(reg_efirst);
            ws.free(reg_ne);
            ws.free(seg_base);
            free_slices();
        } else if (split_in_expand) {
            // cursor of output row (h, c), indexed h * nc + c
            int64_t *cursor = ws.alloc<int64_t>(n_out);
            {
                Timed t(p, GMAGNUS_K_EXPAND, s);
                const int shift0 = g.shift;
                int32_t *oc = col_buf[nxt];
                void *ov = val_buf[nxt];
                values_step([=](const Csr &, const Csr &B, hipStream_t st) {
                    gather_i64(out_ptr, x_map, n_out, cursor, st);
                    expand_split(B, sl, H, exp_tiles, sbnd, nc, shift0, cursor, oc, ov, st);
                });
            }
            ws.free(cursor);
            p->info.kernel_launches[GMAGNUS_K_EXPAND] += 1;
            add_bytes(p, GMAGNUS_K_EXPAND, (4.0 + VS) * H + (4.0 + VS) * sl.nnz + (CS + VS) * blen_total + 8.0 * n_out);
            free_slices();
        } else {
            int64_t *cursor = ws.alloc<int64_t>(n_out);
            {
                Timed t(p, GMAGNUS_K_MULTISPLIT, s);
                const int32_t *ic = col_buf[cur];
                const void *iv = val_buf[cur];
                int32_t *oc = col_buf[nxt];
                void *ov = val_buf[nxt];
                const int nn = g.next_chunks;
                const bool v32 = p->B.v32;
                values_step([=](const Csr &, const Csr &, hipStream_t st) {
                    copy_i64(cursor, out_ptr, n_out, st);
                    if (next_counts) fill<int64_t>(next_counts, 0, nh_out * nn, st);
                    multisplit(g, in_ptr, tile_row, ic, iv, v32, x_map, cursor, oc, ov, nh_out, next_counts, st);
                });
            }
            ws.free(cursor);
            p->info.kernel_launches[GMAGNUS_K_MULTISPLIT] += 1;
            add_bytes(p, GMAGNUS_K_MULTISPLIT, 2.0 * (4.0 + VS) * elems + 8.0 * (n_in + 1) + 8.0 * n_out);
        }
        p->info.levels_run = lvl + 1;
        LeafLevel lv;
        lv.set = LeafSet{out_ptr, col_buf[nxt], val_buf[nxt], origin_out, last ? 0 : nh_out, n_out};
        lv.set.v32 = p->B.v32;
        lv.width = (int64_t)1 << g.shift;
        p->leaves.push_back(lv);
        if (two_done.set.ptr) {
            p->leaves.push_back(two_done);
            p->info.levels_run = lvl + 2;
        }
        ws.free(tile_row);
        ws.free(sc);
        ws.free(x_map);
        ws.free(perm2);
        ws.free(cb);
        ws.free(out_cnt);
        ws.free(ccls);
        ws.free(counts);
        counts = next_counts;
        if (last || nh_out == 0 || two_done.set.ptr) break;
        in_ptr = out_ptr;
        n_in = nh_out;
        elems = cbh[3];
        origin_in = origin_out;
        m_in_log2 = g.shift;
        cur = nxt;
    }
    if (counts) ws.free(counts);

    // ---- final chunks: symbolic
    p->slot = ws.alloc<int64_t>(nh * p->n_slots);
    fill<int64_t>(p->slot, 0, nh * p->n_slots, s);
    // Every level's classes first, then one host read of all their bins and
    // element ranges; every level's symbolic launches and numeric classes,
    // then one read of all numeric bins (two round trips, not two per level).
    struct LeafTmp {
        int64_t *sc = nullptr, *bins = nullptr;
        uint8_t *lc = nullptr;
        int64_t e0 = 0, e1 = 0;
    };
    std::vector<LeafTmp> tmp(p->leaves.size());
    for (size_t i = 0; i < p->leaves.size(); ++i) {
        LeafLevel &lv = p->leaves[i];
        const int64_t nl = lv.set.hi - lv.set.lo;
        if (nl <= 0) continue;
        LeafTmp &tl = tmp[i];
        lv.leaf_nnz = ws.alloc<int64_t>(nl);
        lv.items_sym = ws.alloc<int64_t>(nl);
        lv.items_num = ws.alloc<int64_t>(nl);
        tl.sc = ws.alloc<int64_t>(partition_scratch_elems(nl, LEAF_NBINS));
        tl.bins = ws.alloc<int64_t>(LEAF_NBINS + 1);
        tl.lc = ws.alloc<uint8_t>(nl);
        Timed t(p, GMAGNUS_K_SETUP, s);
        fill<int64_t>(lv.leaf_nnz, 0, nl, s);
        leaf_classes_sym(lv.set, P.tau, lv.width, tl.lc, s);
        partition_u8(tl.lc, nl, LEAF_NBINS, lv.items_sym, nullptr, tl.bins, tl.sc, s);
    }
    {
        HostReads r(s);
        for (size_t i = 0; i < p->leaves.size(); ++i) {
            LeafLevel &lv = p->leaves[i];
            if (lv.set.hi - lv.set.lo <= 0) continue;
            if (!r.room(LEAF_NBINS + 3, 3)) r.wait();
            r.add(tmp[i].bins, LEAF_NBINS + 1, lv.bins_sym);
            r.add(lv.set.ptr + lv.set.lo, 1, &tmp[i].e0);
            r.add(lv.set.ptr + lv.set.hi, 1, &tmp[i].e1);
        }
        r.wait();
    }
    for (size_t i = 0; i < p->leaves.size(); ++i) {
        LeafLevel &lv = p->leaves[i];
        const int64_t nl = lv.set.hi - lv.set.lo;
        if (nl <= 0) continue;
        LeafTmp &tl = tmp[i];
        lv.elems = tl.e1 - tl.e0;
        {
            LeafTask *tasks = ws.alloc<LeafTask>(nl);
            leaf_tasks_sym(lv.set, lv.items_sym, nl, tasks, s);
            Timed t(p, GMAGNUS_K_CHUNK_SYM, s);
            for (int b = LEAF_H0; b < LEAF_NBINS; ++b) {
                if (b == LEAF_DENSE_BIG) continue;  // launched together with LEAF_DENSE, first
                const int64_t b0 = b == LEAF_DENSE ? lv.bins_sym[LEAF_DENSE_BIG] : lv.bins_sym[b];
                const int64_t cnt = lv.bins_sym[b + 1] - b0;
                leaf_symbolic(lv.set, b, tasks + b0, cnt, lv.width, tl.e1, lv.leaf_nnz, p->slot, s);
                if (cnt) p->info.kernel_launches[GMAGNUS_K_CHUNK_SYM] += 1;
                if (b == LEAF_DENSE) p->info.n_leaves_dense += cnt;
                else if (b == LEAF_RANK || b == LEAF_RANK_L || b == LEAF_RANK_XL || b == LEAF_RANK_T)
                    p->info.n_leaves_rank += cnt;
                else p->info.n_leaves_hash += cnt;
            }
            add_bytes(p, GMAGNUS_K_CHUNK_SYM, (lv.set.col16 ? 2.0 : 4.0) * lv.elems + 16.0 * nl);
            ws.free(tasks);
        }
        // numeric bins now, so the numeric phase needs no host round trip
        Timed t(p, GMAGNUS_K_SETUP, s);
        leaf_classes_num(lv.set, lv.leaf_nnz, P.tau, lv.width, tl.lc, s);
        partition_u8(tl.lc, nl, LEAF_NBINS, lv.items_num, nullptr, tl.bins, tl.sc, s);
    }
    {
        HostReads r(s);
        for (size_t i = 0; i < p->leaves.size(); ++i) {
            LeafLevel &lv = p->leaves[i];
            if (lv.set.hi - lv.set.lo <= 0) continue;
            if (!r.room(LEAF_NBINS + 1, 1)) r.wait();
            r.add(tmp[i].bins, LEAF_NBINS + 1, lv.bins_num);
        }
        r.wait();
    }
    for (LeafTmp &tl : tmp) {
        ws.free(tl.sc);
        ws.free(tl.bins);
        ws.free(tl.lc);
    }
    {
        Timed t(p, GMAGNUS_K_ROWPTR, s);
        slot_scan(p->slot, nh, p->n_slots, p->heavy_rows, p->row_nnz, s);
        add_bytes(p, GMAGNUS_K_ROWPTR, 16.0 * nh * p->n_slots);
    }
    // the other buffer (if only level 0 wrote into it, or never used) stays until numeric
}

// (*keep: a workspace block the light stream's kernels still use, freed by the
// caller after the streams join)
void light_symbolic_all(gmagnus_plan_s *p, void **keep) {
    const hipStream_t s = p->s_light;
    Timed t(p, GMAGNUS_K_LIGHT_SYM, s);
    double ips = 0;
    for (int b = LIGHT_W0; b < LIGHT_NBINS; ++b) {
        const int64_t cnt = p->bins_sym[b + 1] - p->bins_sym[b];
        if (b == LIGHT_W0 && cnt > 0 && cnt >= p->B.n_rows / 8) {
            // many narrow rows: summarize B's rows once, then one mask per A entry
            void *masks = p->ws->alloc_bytes(brow_mask_bytes(p->B));
            light_symbolic_narrow(p->A, p->B, p->r0, p->perm + p->bins_sym[b], cnt, p->minc, masks, p->row_nnz, s);
            *keep = masks;
        } else {
            light_symbolic(p->A, p->B, p->r0, b, p->perm + p->bins_sym[b], cnt, p->minc, p->maxc, p->row_nnz, s);
        }
        if (cnt) p->info.kernel_launches[GMAGNUS_K_LIGHT_SYM] += 1;
    }
    ips = (double)(p->products_total - p->products_heavy);
    add_bytes(p, GMAGNUS_K_LIGHT_SYM, (double)p->csize * ips);
}

void do_symbolic(gmagnus_plan_s *p, int64_t *c_row_ptr, int64_t *c_nnz) {
    GM_REQUIRE(c_row_ptr != nullptr && c_nnz != nullptr, GMAGNUS_ERROR_INVALID_VALUE, "NULL output");
    GM_REQUIRE(!p->symbolic_done, GMAGNUS_ERROR_NOT_READY, "symbolic already ran for this plan");
    Workspace &ws = *p->ws;
    const int64_t n = p->n;
    if (n == 0) {
        fill<int64_t>(c_row_ptr, 0, 1, p->stream);
        GM_HIP(hipStreamSynchronize(p->stream));
        *c_nnz = 0;
        p->symbolic_done = true;
        return;
    }
    p->row_nnz = ws.alloc<int64_t>(n);
    fill<int64_t>(p->row_nnz, 0, n, p->stream);
    hipEvent_t fork, jh, jl;
    GM_HIP(hipEventCreateWithFlags(&fork, hipEventDisableTiming));
    GM_HIP(hipEventCreateWithFlags(&jh, hipEventDisableTiming));
    GM_HIP(hipEventCreateWithFlags(&jl, hipEventDisableTiming));
    struct EvGuard {
        hipEvent_t a, b, c;
        ~EvGuard() {
            (void)hipEventDestroy(a);
            (void)hipEventDestroy(b);
            (void)hipEventDestroy(c);
        }
    } guard{fork, jh, jl};
    GM_HIP(hipEventRecord(fork, p->stream));
    if (p->s_light != p->stream) GM_HIP(hipStreamWaitEvent(p->s_light, fork, 0));
    if (p->s_heavy != p->stream) GM_HIP(hipStreamWaitEvent(p->s_heavy, fork, 0));
    // light work is enqueued first so it overlaps the heavy path's host round trips
    void *light_keep = nullptr;
    light_symbolic_all(p, &light_keep);
    if (p->n_heavy > 0) heavy_symbolic(p);
    GM_HIP(hipEventRecord(jl, p->s_light));
    GM_HIP(hipEventRecord(jh, p->s_heavy));
    GM_HIP(hipStreamWaitEvent(p->stream, jl, 0));
    GM_HIP(hipStreamWaitEvent(p->stream, jh, 0));
    ws.free(light_keep);
    // C's row pointers, then the light rows' numeric bins; nnz(C) and the
    // bins come back in one host round trip
    int64_t *hs = nullptr, *sc = nullptr;
    {
        Timed t(p, GMAGNUS_K_ROWPTR, p->stream);
        sc = ws.alloc<int64_t>(scan_scratch_elems(n));
        scan_i64(p->row_nnz, n, c_row_ptr, sc, p->stream);
        if (p->n_heavy > 0) {
            hs = ws.alloc<int64_t>(p->n_heavy + 1);
            scan_gather_i64(p->row_nnz, p->heavy_rows, p->n_heavy, hs, sc, p->stream);  // sc: after the first scan
        }
        add_bytes(p, GMAGNUS_K_ROWPTR, 16.0 * n);
    }
    uint8_t *cls = ws.alloc<uint8_t>(n);
    int64_t *bins = ws.alloc<int64_t>(LIGHT_NBINS + 1);
    int64_t *psc = ws.alloc<int64_t>(partition_scratch_elems(n, LIGHT_NBINS));
    {
        Timed t(p, GMAGNUS_K_SETUP, p->stream);
        const bool window = (p->opts.flags & GMAGNUS_FLAG_NO_WINDOW) == 0;
        p->perm_num = ws.alloc<int64_t>(n);
        light_classes_num(p->ip, p->row_nnz, p->minc, p->maxc, p->B.ci64, n, p->info.row_tau, window, cls,
                          p->stream);
        partition_u8(cls, n, LIGHT_NBINS, p->perm_num, nullptr, bins, psc, p->stream);
    }
    {
        HostReads r(p->stream);
        r.add(c_row_ptr + n, 1, &p->c_nnz);
        if (hs) r.add(hs + p->n_heavy, 1, &p->info.c_nnz_heavy);
        r.add(bins, LIGHT_NBINS + 1, p->bins_num);
        r.wait();
    }
    ws.free(hs);
    ws.free(sc);
    ws.free(cls);
    ws.free(bins);
    ws.free(psc);
    *c_nnz = p->c_nnz;
    p->info.c_nnz = p->c_nnz;
    p->symbolic_done = true;
}

void do_numeric(gmagnus_plan_s *p, const int64_t *c_row_ptr, void *c_col, void *c_val) {
    GM_REQUIRE(p->symbolic_done, GMAGNUS_ERROR_NOT_READY, "numeric called before symbolic");
    GM_REQUIRE(c_row_ptr != nullptr, GMAGNUS_ERROR_INVALID_VALUE, "NULL c_row_ptr");
    GM_REQUIRE(p->c_nnz == 0 || (c_col && c_val), GMAGNUS_ERROR_INVALID_VALUE, "NULL C output arrays");
    if (p->n == 0 || p->c_nnz == 0) return;
    hipEvent_t fork, jh, jl;
    GM_HIP(hipEventCreateWithFlags(&fork, hipEventDisableTiming));
    GM_HIP(hipEventCreateWithFlags(&jh, hipEventDisableTiming));
    GM_HIP(hipEventCreateWithFlags(&jl, hipEventDisableTiming));
    struct EvGuard {
        hipEvent_t a, b, c;
        ~EvGuard() {
            (void)hipEventDestroy(a);
            (void)hipEventDestroy(b);
            (void)hipEventDestroy(c);
        }
    } guard{fork, jh, jl};
    GM_HIP(hipEventRecord(fork, p->stream));
    if (p->s_light != p->stream) GM_HIP(hipStreamWaitEvent(p->s_light, fork, 0));
    if (p->s_heavy != p->stream) GM_HIP(hipStreamWaitEvent(p->s_heavy, fork, 0));
    {
        const hipStream_t s = p->s_heavy;
        Timed t(p, GMAGNUS_K_CHUNK_NUM, s);
        for (auto &lv : p->leaves) {
            const int64_t nl = lv.set.hi - lv.set.lo;
            if (nl <= 0) continue;
            LeafTask *tasks = p->ws->alloc<LeafTask>(nl);
            int32_t *counter = p->ws->alloc<int32_t>(1);
            leaf_tasks_num(lv.set, lv.items_num, nl, lv.leaf_nnz, p->n_slots_log2, p->heavy_rows, c_row_ptr, p->slot,
                           p->slot_width_log2, tasks, s);
            for (int b = LEAF_H0; b < LEAF_NBINS; ++b) {
                if (b == LEAF_DENSE_BIG) continue;  // launched together with LEAF_DENSE, first
                const int64_t b0 = b == LEAF_DENSE ? lv.bins_num[LEAF_DENSE_BIG] : lv.bins_num[b];
                const int64_t cnt = lv.bins_num[b + 1] - b0;
                leaf_numeric(lv.set, b, tasks + b0, cnt, lv.width, c_col, p->B.ci64, p->slot_width_log2, c_val,
                             p->err, counter, s);
                if (cnt) p->info.kernel_launches[GMAGNUS_K_CHUNK_NUM] += 1;
            }
            p->ws->free(tasks);
            p->ws->free(counter);
            add_bytes(p, GMAGNUS_K_CHUNK_NUM, ((lv.set.col16 ? 2.0 : 4.0) + p->vsize) * lv.elems);
        }
    }
    {
        const hipStream_t s = p->s_light;
        Timed t(p, GMAGNUS_K_LIGHT_NUM, s);
        for (int b = LIGHT_W0; b < LIGHT_NBINS; ++b) {
            const int64_t cnt = p->bins_num[b + 1] - p->bins_num[b];
            light_numeric(p->A, p->B, p->r0, b, p->perm_num + p->bins_num[b], cnt, p->minc, p->maxc, c_row_ptr, c_col,
                          c_val, p->err, s);
            if (cnt) p->info.kernel_launches[GMAGNUS_K_LIGHT_NUM] += 1;
        }
        add_bytes(p, GMAGNUS_K_LIGHT_NUM, (double)(p->csize + p->vsize) * (double)(p->products_total - p->products_heavy));
    }
    GM_HIP(hipEventRecord(jl, p->s_light));
    GM_HIP(hipEventRecord(jh, p->s_heavy));
    GM_HIP(hipStreamWaitEvent(p->stream, jl, 0));
    GM_HIP(hipStreamWaitEvent(p->stream, jh, 0));
    // output bytes of C, split by the rows they belong to
    const double cb = (double)(p->csize + p->vsize);  // bytes of an entry of C
    add_bytes(p, GMAGNUS_K_CHUNK_NUM, cb * (double)p->info.c_nnz_heavy);
    add_bytes(p, GMAGNUS_K_LIGHT_NUM, cb * (double)(p->c_nnz - p->info.c_nnz_heavy));
}

// New values on the kept patterns: the light rows read A and B directly in
// the numeric phase; the heavy rows' recorded steps rewrite the expansion and
// multisplit buffers that the final chunks' numeric kernels read.
void do_update_values(gmagnus_plan_s *p, const void *a_val, const void *b_val) {
    GM_REQUIRE((p->opts.flags & GMAGNUS_FLAG_KEEP_PATTERN) != 0, GMAGNUS_ERROR_INVALID_VALUE,
               "plan made without GMAGNUS_FLAG_KEEP_PATTERN");
    GM_REQUIRE(p->symbolic_done, GMAGNUS_ERROR_NOT_READY, "values updated before symbolic");
    GM_REQUIRE((a_val || p->A.nnz == 0) && (b_val || p->B.nnz == 0), GMAGNUS_ERROR_INVALID_VALUE, "NULL values");
    p->A.v = a_val;
    p->B.v = b_val;
    if (p->replay.empty()) return;
    hipEvent_t fork, join;
    GM_HIP(hipEventCreateWithFlags(&fork, hipEventDisableTiming));
    GM_HIP(hipEventCreateWithFlags(&join, hipEventDisableTiming));
    struct EvGuard {
        hipEvent_t a, b;
        ~EvGuard() {
            (void)hipEventDestroy(a);
            (void)hipEventDestroy(b);
        }
    } guard{fork, join};
    const hipStream_t s = p->s_heavy;
    GM_HIP(hipEventRecord(fork, p->stream));
    if (s != p->stream) GM_HIP(hipStreamWaitEvent(s, fork, 0));
    {
        Timed t(p, GMAGNUS_K_EXPAND, s);
        for (auto &f : p->replay) f(p->A, p->B, s);
    }
    GM_HIP(hipEventRecord(join, s));
    if (s != p->stream) GM_HIP(hipStreamWaitEvent(p->stream, join, 0));
}

template <class F>
gmagnus_status_t guarded(F &&f) {
    try {
        f();
        return GMAGNUS_SUCCESS;
    } catch (const Error &e) {
        set_last_error(e.msg);
        return e.status;
    } catch (const std::bad_alloc &) {
        set_last_error("host allocation failed");
        return GMAGNUS_ERROR_OUT_OF_MEMORY;
    } catch (...) {
        set_last_error("unexpected exception");
        return GMAGNUS_ERROR_HIP;
    }
}

}  // namespace

namespace gm {
gmagnus_status_t make_plan(gmagnus_plan_t *out, const gmagnus_matrix_t *A, const gmagnus_matrix_t *B,
                           const gmagnus_options_t *opts, void *hip_stream, bool no_alloc) {
    if (!out) {
        set_last_error("NULL plan output");
        return GMAGNUS_ERROR_INVALID_VALUE;
    }
    *out = nullptr;
    gmagnus_plan_s *p = nullptr;
    gmagnus_status_t st = guarded([&] {
        p = new gmagnus_plan_s();
        p->no_alloc = no_alloc;
        TimedPlanScope tps(p);
        if (no_alloc)
            GM_REQUIRE(opts && opts->alloc && opts->free, GMAGNUS_ERROR_INVALID_VALUE,
                       "a plan that must not allocate needs workspace callbacks");
        do_plan(p, A, B, opts, (hipStream_t)hip_stream);
    });
    if (st != GMAGNUS_SUCCESS) {
        delete p;
        return st;
    }
    *out = p;
    return st;
}
}  // namespace gm

// =================================================================== C ABI
extern "C" {

void gmagnus_options_init(gmagnus_options_t *opts) {
    if (!opts) return;
    std::memset(opts, 0, sizeof(*opts));
    opts->struct_size = sizeof(gmagnus_options_t);
}

gmagnus_status_t gmagnus_get_params_typed(int64_t c_m, int64_t lds_bytes, int32_t index_type, int32_t value_type,
                                          const gmagnus_options_t *opts, gmagnus_params_t *out) {
    return guarded([&] {
        GM_REQUIRE(out != nullptr, GMAGNUS_ERROR_INVALID_VALUE, "NULL output");
        GM_REQUIRE(!opts || opts->struct_size == sizeof(gmagnus_options_t), GMAGNUS_ERROR_INVALID_VALUE,
                   "options.struct_size mismatch");
        GM_REQUIRE(index_type == GMAGNUS_INDEX_INT32 || index_type == GMAGNUS_INDEX_INT64, GMAGNUS_ERROR_INVALID_VALUE,
                   "unknown index type");
        GM_REQUIRE(value_type == GMAGNUS_VALUE_FP64 || value_type == GMAGNUS_VALUE_FP32, GMAGNUS_ERROR_INVALID_VALUE,
                   "unknown value type");
        compute_params(c_m, lds_bytes, index_bytes(index_type), value_bytes(value_type), opts, out);
    });
}

gmagnus_status_t gmagnus_get_params(int64_t c_m, int64_t lds_bytes, const gmagnus_options_t *opts,
                                    gmagnus_params_t *out) {
    return gmagnus_get_params_typed(c_m, lds_bytes, GMAGNUS_INDEX_INT32, GMAGNUS_VALUE_FP64, opts, out);
}

int32_t gmagnus_expansion_path(const gmagnus_params_t *params, int64_t n_heavy, int64_t products_heavy,
                               int64_t b_nnz, int32_t flags) {
    if (!params) return GMAGNUS_PATH_NONE;
    return expansion_path(*params, n_heavy, products_heavy, b_nnz, flags);
}

gmagnus_status_t gmagnus_plan_typed(gmagnus_plan_t *out, const gmagnus_matrix_t *A, const gmagnus_matrix_t *B,
                                    const gmagnus_options_t *opts, void *hip_stream) {
    return gm::make_plan(out, A, B, opts, hip_stream, false);
}

gmagnus_status_t gmagnus_plan(gmagnus_plan_t *out, const gmagnus_csr_t *A, const gmagnus_csr_t *B,
                              const gmagnus_options_t *opts, void *hip_stream) {
    const gmagnus_matrix_t a = typed_desc(A), b = typed_desc(B);
    return gm::make_plan(out, A ? &a : nullptr, B ? &b : nullptr, opts, hip_stream, false);
}

gmagnus_status_t gmagnus_spgemm_symbolic(gmagnus_plan_t plan, int64_t *c_row_ptr, int64_t *c_nnz) {
    if (!plan) {
        set_last_error("NULL plan");
        return GMAGNUS_ERROR_INVALID_VALUE;
    }
    return guarded([&] {
        TimedPlanScope tps(plan);
        do_symbolic(plan, c_row_ptr, c_nnz);
    });
}

gmagnus_status_t gmagnus_spgemm_numeric_typed(gmagnus_plan_t plan, const int64_t *c_row_ptr, void *c_col_idx,
                                              void *c_val) {
    if (!plan) {
        set_last_error("NULL plan");
        return GMAGNUS_ERROR_INVALID_VALUE;
    }
    return guarded([&] {
        TimedPlanScope tps(plan);
        do_numeric(plan, c_row_ptr, c_col_idx, c_val);
    });
}

gmagnus_status_t gmagnus_spgemm_numeric(gmagnus_plan_t plan, const int64_t *c_row_ptr, int32_t *c_col_idx,
                                        double *c_val) {
    if (plan && (plan->B.ci64 || plan->B.v32)) {
        set_last_error("the plan's matrices have int64 columns or fp32 values: use gmagnus_spgemm_numeric_typed");
        return GMAGNUS_ERROR_INVALID_VALUE;
    }
    return gmagnus_spgemm_numeric_typed(plan, c_row_ptr, c_col_idx, c_val);
}

gmagnus_status_t gmagnus_update_values_typed(gmagnus_plan_t plan, const void *a_val, const void *b_val) {
    if (!plan) {
        set_last_error("NULL plan");
        return GMAGNUS_ERROR_INVALID_VALUE;
    }
    return guarded([&] {
        TimedPlanScope tps(plan);
        do_update_values(plan, a_val, b_val);
    });
}

gmagnus_status_t gmagnus_update_values(gmagnus_plan_t plan, const double *a_val, const double *b_val) {
    if (plan && plan->B.v32) {
        set_last_error("the plan's values are fp32: use gmagnus_update_values_typed");
        return GMAGNUS_ERROR_INVALID_VALUE;
    }
    return gmagnus_update_values_typed(plan, a_val, b_val);
}

gmagnus_status_t gmagnus_plan_info(gmagnus_plan_t plan, gmagnus_plan_info_t *out) {
    if (!plan || !out) {
        set_last_error("NULL plan or output");
        return GMAGNUS_ERROR_INVALID_VALUE;
    }
    return guarded([&] {
        if (plan->timing || plan->symbolic_done) {
            GM_HIP(hipStreamSynchronize(plan->stream));
            if (plan->s_heavy != plan->stream) GM_HIP(hipStreamSynchronize(plan->s_heavy));
            if (plan->s_light != plan->stream) GM_HIP(hipStreamSynchronize(plan->s_light));
        }
        if (plan->timing) {
            for (auto &t : plan->timers) {
                float ms = 0;
                GM_HIP(hipEventElapsedTime(&ms, t.a, t.b));
                plan->info.kernel_ms[t.cls] += ms;
                (void)hipEventDestroy(t.a);
                (void)hipEventDestroy(t.b);
            }
            plan->timers.clear();
        }
        if (plan->err) {
            int32_t f = 0;
            GM_HIP(hipMemcpy(&f, plan->err, sizeof(f), hipMemcpyDeviceToHost));
            plan->info.check_flags = f;
        }
        if (plan->ws) plan->info.workspace_peak_bytes = (int64_t)plan->ws->peak_bytes();
        *out = plan->info;
    });
}

void gmagnus_plan_destroy(gmagnus_plan_t plan) { delete plan; }

gmagnus_status_t gmagnus_row_products(const gmagnus_csr_t *A, const gmagnus_csr_t *B, int64_t *ip, void *hip_stream) {
    const gmagnus_matrix_t a = typed_desc(A), b = typed_desc(B);
    return gmagnus_row_products_typed(A ? &a : nullptr, B ? &b : nullptr, ip, hip_stream);
}

gmagnus_status_t gmagnus_row_products_typed(const gmagnus_matrix_t *A, const gmagnus_matrix_t *B, int64_t *ip,
                                            void *hip_stream) {
    return guarded([&] {
        check_pair(A, B);
        GM_REQUIRE(ip != nullptr || A->n_rows == 0, GMAGNUS_ERROR_INVALID_VALUE, "NULL ip");
        if (A->n_rows == 0) return;
        hipStream_t s = (hipStream_t)hip_stream;
        row_products(to_csr(A), to_csr(B), 0, A->n_rows, A->nnz, ip, nullptr, nullptr, s);
        GM_HIP(hipStreamSynchronize(s));
    });
}

gmagnus_status_t gmagnus_split_panels(const gmagnus_csr_t *A, const gmagnus_csr_t *B, int64_t max_products,
                                      int64_t *bounds, int64_t max_panels, int64_t *n_panels, void *hip_stream) {
    const gmagnus_matrix_t a = typed_desc(A), b = typed_desc(B);
    return gmagnus_split_panels_typed(A ? &a : nullptr, B ? &b : nullptr, max_products, bounds, max_panels, n_panels,
                                      hip_stream);
}

gmagnus_status_t gmagnus_split_panels_typed(const gmagnus_matrix_t *A, const gmagnus_matrix_t *B,
                                            int64_t max_products, int64_t *bounds, int64_t max_panels,
                                            int64_t *n_panels, void *hip_stream) {
    return guarded([&] {
        check_pair(A, B);
        GM_REQUIRE(bounds && n_panels && max_panels >= 1 && max_products >= 1, GMAGNUS_ERROR_INVALID_VALUE,
                   "bad panel arguments");
        const int64_t n = A->n_rows;
        hipStream_t s = (hipStream_t)hip_stream;
        bounds[0] = 0;
        *n_panels = 0;
        if (n == 0) return;
        Workspace ws(nullptr, s);
        {
            // no row can have more products than its A entries times B's longest
            // row: when nnz(A) times that stays within the limit, the whole
            // matrix is one panel and the row products need not be formed
            int64_t *mx = ws.alloc<int64_t>(1);
            fill<int64_t>(mx, 0, 1, s);
            hipLaunchKernelGGL(k_max_row_len, dim3(grid_for(B->n_rows, MAXLEN_BLOCK, MAXLEN_GRID)), dim3(MAXLEN_BLOCK),
                               0, s, B->row_ptr, B->n_rows, (unsigned long long *)mx);
            GM_CHECK_LAUNCH();
            const int64_t maxlen = read_scalar(mx, s);
            if (maxlen == 0 || A->nnz <= max_products / maxlen) {
                bounds[1] = n;
                *n_panels = 1;
                return;
            }
        }
        int64_t *ip = ws.alloc<int64_t>(n), *sc = ws.alloc<int64_t>(n + 1);
        int64_t *scratch = ws.alloc<int64_t>(scan_scratch_elems(n));
        int64_t *out = ws.alloc<int64_t>(max_panels + 2);
        row_products(to_csr(A), to_csr(B), 0, n, A->nnz, ip, nullptr, nullptr, s);
        scan_i64(ip, n, sc, scratch, s);
        hipLaunchKernelGGL(k_split_panels, dim3(1), dim3(SPLIT_BLOCK), 0, s, sc, n, max_products, max_panels, out);
        GM_CHECK_LAUNCH();
        // the count and the first bounds in one read; more panels than that in a second
        const int64_t first = std::min<int64_t>(max_panels + 2, READ_SLOTS);
        std::vector<int64_t> head(first);
        {
            HostReads r(s);
            r.add(out, (int)first, head.data());
            r.wait();
        }
        const int64_t cnt = head[0];
        GM_REQUIRE(cnt >= 1, GMAGNUS_ERROR_INVALID_VALUE, "more panels needed than max_panels");
        const int64_t have = std::min<int64_t>(cnt + 1, first - 1);
        std::copy(head.begin() + 1, head.begin() + 1 + have, bounds);
        if (cnt + 1 > have) {
            GM_HIP(hipMemcpyAsync(bounds + have, out + 1 + have, sizeof(int64_t) * (cnt + 1 - have),
                                  hipMemcpyDeviceToHost, s));
            GM_HIP(hipStreamSynchronize(s));
        }
        *n_panels = cnt;
    });
}

void gmagnus_release_cache(void) { cache_release(); }

const char *gmagnus_last_error(void) { return g_last_error.c_str(); }

const char *gmagnus_status_string(gmagnus_status_t status) {
    switch (status) {
    case GMAGNUS_SUCCESS: return "GMAGNUS_SUCCESS";
    case GMAGNUS_ERROR_INVALID_VALUE: return "GMAGNUS_ERROR_INVALID_VALUE";
    case GMAGNUS_ERROR_INVALID_CSR: return "GMAGNUS_ERROR_INVALID_CSR";
    case GMAGNUS_ERROR_OUT_OF_MEMORY: return "GMAGNUS_ERROR_OUT_OF_MEMORY";
    case GMAGNUS_ERROR_NOT_READY: return "GMAGNUS_ERROR_NOT_READY";
    case GMAGNUS_ERROR_HIP: return "GMAGNUS_ERROR_HIP";
    case GMAGNUS_ERROR_UNSUPPORTED: return "GMAGNUS_ERROR_UNSUPPORTED";
    }
    return "GMAGNUS_ERROR_UNKNOWN";
}

}  // extern "C"
