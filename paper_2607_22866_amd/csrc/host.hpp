// Host-side infrastructure: status propagation, the device workspace
// allocator, and the launch wrappers every kernel translation unit exports.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/gmagnus.h"
#include "common.hpp"

namespace gm {

// Error carried from the point of failure to the C ABI.
struct Error {
    gmagnus_status_t status;
    std::string msg;
};

void set_last_error(const std::string &msg);

#define GM_HIP(expr)                                                                                   \
    do {                                                                                               \
        hipError_t e_ = (expr);                                                                        \
        if (e_ != hipSuccess)                                                                          \
            throw ::gm::Error{GMAGNUS_ERROR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)};   \
    } while (0)

#define GM_CHECK_LAUNCH() GM_HIP(hipGetLastError())

#define GM_REQUIRE(cond, status, msg)                         \
    do {                                                      \
        if (!(cond)) throw ::gm::Error{(status), (msg)};      \
    } while (0)

// Device memory for one plan. Blocks come from the user's callbacks or from
// the library's process-wide caching allocator. free() keeps a block on the
// plan's own free list (reused by later allocations of the same plan, which
// are ordered after the freeing work by the plan's stream joins); every block
// goes back to the user or the shared cache only on destruction, after the
// plan's streams have been synchronised.
class Workspace {
  public:
    Workspace(const gmagnus_options_t *opts, hipStream_t stream) : stream_(stream) {
        if (opts && opts->alloc && opts->free) {
            ualloc_ = opts->alloc;
            ufree_ = opts->free;
            uctx_ = opts->alloc_ctx;
        }
        if (opts) limit_ = (size_t)(opts->workspace_limit_bytes > 0 ? opts->workspace_limit_bytes : 0);
    }
    ~Workspace() { release_all(); }
    Workspace(const Workspace &) = delete;
    Workspace &operator=(const Workspace &) = delete;

    void *alloc_bytes(size_t bytes);
    template <typename T>
    T *alloc(int64_t n) {
        return static_cast<T *>(alloc_bytes(sizeof(T) * (size_t)(n > 0 ? n : 1)));
    }
    // While held, free() keeps blocks in use (a plan that must keep every
    // buffer its recorded launches read).
    void free(void *p);
    void hold(bool h) { hold_ = h; }
    void release_all();
    size_t bytes_in_use() const { return in_use_; }
    size_t bytes_owned() const { return owned_; }
    size_t peak_bytes() const { return peak_; }

  private:
    struct Block {
        void *p;
        size_t bytes;
    };
    hipStream_t stream_;
    void *(*ualloc_)(size_t, void *, void *) = nullptr;
    void (*ufree_)(void *, void *, void *) = nullptr;
    void *uctx_ = nullptr;
    std::vector<Block> blocks_;  // owned, in use
    std::vector<Block> spare_;   // owned, freed by the plan
    size_t in_use_ = 0;
    size_t owned_ = 0;           // bytes of blocks_ and spare_
    size_t peak_ = 0;            // largest owned_
    size_t limit_ = 0;           // bound on owned_ (0: none)
    void give_back(const Block &b);
    bool hold_ = false;
};

void cache_release();

// Builds a plan (gmagnus_plan); with no_alloc the plan's workspace comes only
// from opts' callbacks and its host reads use pageable memory.
gmagnus_status_t make_plan(gmagnus_plan_t *out, const gmagnus_matrix_t *A, const gmagnus_matrix_t *B,
                           const gmagnus_options_t *opts, void *hip_stream, bool no_alloc);

// Raises a kernel's dynamic LDS limit to `bytes` on the current device, once
// per (device, kernel); thread-safe.
void allow_dynamic_lds(const void *kernel, int bytes);

// ----------------------------------------------------------------- prims.hip
// Exclusive scan of n int64 values; out has n+1 entries (out[n] = total).
// `scratch` must hold scan_scratch_elems(n) int64.
int64_t scan_scratch_elems(int64_t n);
void scan_i64(const int64_t *in, int64_t n, int64_t *out, int64_t *scratch, hipStream_t s);
// Exclusive scan of the int64 values in[idx[i]] (gather), n entries.
void scan_gather_i64(const int64_t *in, const int64_t *idx, int64_t n, int64_t *out, int64_t *scratch,
                     hipStream_t s);

// Stable partition of items 0..n-1 into `nc` classes given by cls[i] (int8).
// perm[pos] = i in class-major, index-stable order; inv[i] = pos when inv is
// not null; class_start (device, nc+1) receives the class boundaries.
int64_t partition_scratch_elems(int64_t n, int nc);
void partition_u8(const uint8_t *cls, int64_t n, int nc, int64_t *perm, int64_t *inv, int64_t *class_start,
                  int64_t *scratch, hipStream_t s);

template <typename T>
void fill(T *p, T v, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_fill<T>, dim3(grid_for(n, 256, 16384)), dim3(256), 0, s, p, v, n);
    GM_CHECK_LAUNCH();
}

// ----------------------------------------------------------------- setup.hip
// Fills ip/minc/maxc for rows [r0, r1) of A (local index r - r0); with minc
// and maxc null only ip (no reads of B's columns). minc / maxc hold B's
// column type (int32 or int64). binfo (brow_info_bytes(B) of workspace, or
// null): a per-B-row summary is built there first and read instead of B's
// row pointers and columns (worth it when the panel has many more A entries
// than B has rows).
int64_t brow_info_bytes(const Csr &B);
void row_products(const Csr &A, const Csr &B, int64_t r0, int64_t r1, int64_t panel_nnz, int64_t *ip, void *minc,
                  void *maxc, hipStream_t s, void *binfo = nullptr);
// Checks canonical CSR; sets *flag (device int32) to nonzero on violation.
void validate_csr(const Csr &M, int32_t *flag, hipStream_t s);


// Masked CSR->CSC of the heavy rows (Algorithm 3, MaskedCsr2Csc).
struct SliceArrays {
    int64_t n_slices = 0;
    int64_t nnz = 0;              // heavy A entries kept (nonempty B row)
    int64_t *col_ptr = nullptr;   // n_slices + 1
    int64_t *slice_off = nullptr; // n_slices + 1 (products)
    int32_t *slice_k = nullptr;   // n_slices: column of A / row of B
    int32_t *row_h = nullptr;     // nnz: heavy-local row index
    void *a_val = nullptr;        // nnz values of A's type
};
void csc_count(const Csr &A, const Csr &B, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
               const int64_t *a_heavy_ptr, int64_t nnz_heavy_all, int64_t *colcnt, hipStream_t s);
void slice_flags(const Csr &B, const int64_t *colcnt, int64_t n_k, uint8_t *cls, hipStream_t s);
void slice_build(const Csr &B, const int64_t *colcnt, const int64_t *slice_perm, int64_t n_slices,
                 int32_t *slice_k, int64_t *cnt_out, int64_t *ip_out, int32_t *k_to_slice, hipStream_t s);
void csc_fill(const Csr &A, const Csr &B, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
              const int64_t *a_heavy_ptr, int64_t nnz_heavy_all, const int32_t *k_to_slice,
              const int64_t *col_ptr, int64_t *fill_cursor, int32_t *row_h, void *a_val, hipStream_t s);
// len[s] = nnz(B[slice_k[s], :]).
void slice_lengths(const Csr &B, const int32_t *slice_k, int64_t n, int64_t *len, hipStream_t s);
// Level-0 histogram from the structure: per-slice chunk boundaries in its B
// row (n_slices * (nc + 1) offsets), then per heavy row the sum of its A~
// entries' chunk sizes (counts: n_heavy * nc).
void slice_chunk_bounds(const Csr &B, const SliceArrays &sl, int nc, int shift, int32_t *bnd, hipStream_t s);
// (cmajor: counts[c * n_heavy + h] instead of counts[h * nc + c])
void struct_hist(const Csr &A, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0, const int64_t *a_heavy_ptr,
                 int64_t nnz_heavy_all, const int32_t *k_to_slice, const int32_t *bnd, int nc, bool cmajor,
                 int64_t *counts, hipStream_t s);
void gather_row_len(const int64_t *row_ptr, const int64_t *rows, int64_t n, int64_t r0, int64_t *out, hipStream_t s);
void gather_i64(const int64_t *src, const int64_t *idx, int64_t n, int64_t *out, hipStream_t s);

// ---------------------------------------------------------------- expand.hip
// Outer-product expansion (Algorithm 4) of every slice into C-hat:
// expand_tiles() locates every tile's first slice and A~ entry (into
// expand_tile_words(total) int64), expand() writes the products.
int64_t expand_tile_words(int64_t total);
void expand_tiles(const Csr &B, const SliceArrays &sl, int64_t total, int64_t *info_words, hipStream_t s);
void expand(const Csr &B, const SliceArrays &sl, int64_t total, const int64_t *info_words, int64_t *chat_cursor,
            int32_t *chat_col, void *chat_val, hipStream_t s);
// Expansion fused with the first level's split into nc chunks of 2^shift
// columns: bnd are the slices' chunk boundaries (slice_chunk_bounds), cursor
// the next free position of output row (h, c) at h * nc + c; columns are
// written chunk-local.
void expand_split(const Csr &B, const SliceArrays &sl, int64_t total, const int64_t *info_words, const int32_t *bnd,
                  int nc, int shift, int64_t *cursor, int32_t *out_col, void *out_val, hipStream_t s);

// ------------------------------------------------------------- rowsplit.hip
// The heavy rows' A entries in row order: B row, its slice (-1 for an empty
// B row), heavy row, start of the B row, value.
struct RowEntries {
    int32_t *k = nullptr;
    int32_t *s = nullptr;
    int32_t *h = nullptr;
    int64_t *b0 = nullptr;
    void *a = nullptr;  // A's value type
};
void heavy_entries(const Csr &A, const Csr &B, const int64_t *heavy_rows, int64_t n_heavy, int64_t r0,
                   const int64_t *a_heavy_ptr, int64_t nnz_heavy_all, const int32_t *k_to_slice, const RowEntries &ent,
                   hipStream_t s);
// pb[c * n_ent + e] = (offset of entry e's chunk-c part inside region (c, row
// of e), offset of that part in e's B row); chunk-major (segmented scan;
// scratch: agg and carry n_waves * nc, wfirst/wlast n_waves).
int64_t entry_offset_waves(int64_t n_ent);
void entry_offsets(const RowEntries &ent, int64_t n_ent, const int32_t *bnd, int nc, int64_t *agg, int32_t *wfirst,
                   int32_t *wlast, int64_t *carry, uint2 *pb, hipStream_t s);
// Region r of the chunk-major level-0 output (perm: position -> c * n_heavy + h).
void region_records(const int64_t *perm, int64_t n_out, int64_t n_heavy, const int64_t *a_heavy_ptr, int32_t *reg_c,
                    int64_t *reg_efirst, int64_t *reg_ne, hipStream_t s);
int64_t rows_tile_words(int64_t total);
bool rows_next_fits(int next_nc);
// Chunk-major row-order expansion with the level-0 split: writes the level-0
// output (chunk-local columns) and, when next_counts is given, the next
// level's counts of the heavy regions.
void expand_rows(const Csr &B, const RowEntries &ent, const uint2 *pb, int64_t n_ent, const int64_t *out_ptr,
                 const int64_t *seg_base, const int32_t *reg_c, const int64_t *reg_efirst, const int64_t *reg_ne,
                 int64_t n_out, int64_t n_heavy_out, int64_t total, int nc, int shift, int next_nc, int next_shift,
                 int64_t *next_counts, int64_t *tile_words, int32_t *out_col, void *out_val, hipStream_t s);

// Two levels in one pass (the hierarchy has exactly two levels): the
// expansion splits the products of the first level's heavy regions by the
// second level's chunk and writes them straight into the final chunks.
// fine_bounds: per slice, offsets of the first column >= f << fshift in its
// B row for the nf + 1 fine boundaries (fine_bounds_words entries);
// fine_counts: F[h * nf + f], products of heavy row h in fine chunk f;
// level1_counts: counts of the second level's rows r * nc1 + c1 for the
// first level's heavy regions (perm: region -> c * n_heavy + h).
int64_t fine_bounds_words(int64_t n_slices, int nf);
void fine_bounds(const Csr &B, const int32_t *slice_k, int64_t n_slices, int nf, int fshift, const int32_t *sbnd,
                 int nc, int32_t *bndf, hipStream_t s);
void fine_counts(const Csr &B, const RowEntries &ent, int64_t n_ent, const int32_t *bndf, int nf, int fshift,
                 int64_t n_heavy, int64_t *F, hipStream_t s);
void level1_counts(const int64_t *perm, int64_t n_regions, int64_t n_heavy, const int64_t *F, int nf, int nc1,
                   int64_t *counts1, hipStream_t s);
// whether the fused second level's keys fit the work group
bool rows2_fits(int64_t tau, int nc1, int nf);
// cursor1: next free place of second-level row r * nc1 + c1 (starts at its
// row pointer); light regions are written to out_*0 at their first-level place;
// the final chunks' columns (at most 2^16 wide) are stored in 16 bits.
void expand_rows2(const Csr &B, const RowEntries &ent, const uint2 *pb, int64_t n_ent,
                  const int64_t *out_ptr, const int64_t *seg_base, const int32_t *reg_c, const int64_t *reg_efirst,
                  const int64_t *reg_ne, int64_t n_out, int64_t n_heavy_out, int64_t total, int nc, int shift,
                  int nc1, int shift1, int64_t tau, int64_t *cursor1, int64_t n_out1_elems, int32_t *err,
                  int64_t *tile_words, int32_t *out_col0, void *out_val0, uint16_t *out_col1, void *out_val1,
                  hipStream_t s);

// ------------------------------------------------------------ multisplit.hip
struct LevelGeom {
    int64_t n_in;        // input rows
    int64_t elems;       // input elements
    int n_chunks;        // chunks per input row (power of two)
    int shift;           // log2 of the output chunk width
    int next_chunks;     // chunks per row at the next level (0 when last)
    int next_shift;      // log2 of the next level's chunk width
    int64_t group_elems; // elements per work group (tile)
    int group_rows;      // rows a tile may touch (power of two, bounded via tau)
};
// Tile sizes the multisplit kernel is built for, largest first.
int multisplit_tile_count();
int64_t multisplit_tile_elems(int i);
int multisplit_max_keys();
int multisplit_max_rows();
bool multisplit_next_fits(int keys, int next_chunks);
void tile_rows(const LevelGeom &g, const int64_t *in_ptr, int64_t *tile_row, hipStream_t s);
// Level histogram (n_in * n_chunks counts); tile_row is scratch of
// histogram_tiles() entries.
int64_t histogram_tiles(const LevelGeom &g, int64_t tau);
void histogram(const LevelGeom &g, int64_t tau, const int64_t *in_ptr, const int32_t *in_col, int64_t *tile_row,
               int64_t *counts, hipStream_t s);
void chunk_classes(const int64_t *counts, int64_t n, int64_t tau, bool last, uint8_t *cls, hipStream_t s);
// out_cnt[inv[i]] = counts[i]; origin_out[inv[i]] = origin_in[h] + c * stride with (h, c) =
// (i / n_chunks, i % n_chunks), or (i % cmajor_rows, i / cmajor_rows) when cmajor_rows > 0.
void chunk_reorder(const int64_t *counts, const int64_t *inv, int64_t n, int n_chunks, const int64_t *origin_in,
                   int64_t stride, int64_t cmajor_rows, int64_t *out_cnt, int64_t *origin_out, hipStream_t s);
void multisplit(const LevelGeom &g, const int64_t *in_ptr, const int64_t *tile_row, const int32_t *in_col,
                const void *in_val, bool v32, const int64_t *x_map, int64_t *cursor, int32_t *out_col, void *out_val,
                int64_t n_heavy_out, int64_t *next_counts, hipStream_t s);

// ------------------------------------------------------------ accumulate.hip
// Final chunks ("leaves"): chunk rows [lo, hi) of some level's output.
struct LeafSet {
    const int64_t *ptr;    // chunk row pointers of that level's output
    const int32_t *col;    // chunk-local columns (or col16)
    const void *val;       // values: fp32 when v32, else fp64
    const int64_t *origin; // slot id h * n_slots + slot, per chunk row
    int64_t lo, hi;
    const uint16_t *col16 = nullptr;  // chunk-local columns stored in 16 bits (final chunks of at most 2^16 columns)
    bool v32 = false;
};
enum LeafBin : uint8_t {
    LEAF_EMPTY = 0, LEAF_H0, LEAF_H1, LEAF_H2, LEAF_H3, LEAF_DENSE_BIG, LEAF_DENSE, LEAF_RANK, LEAF_RANK_L, LEAF_RANK_XL,
    LEAF_RANK_T, LEAF_NBINS
};
enum LightBin : uint8_t {
    LIGHT_EMPTY = 0, LIGHT_HEAVY, LIGHT_W0, LIGHT_W1, LIGHT_W2, LIGHT_H0, LIGHT_H1, LIGHT_H2, LIGHT_H3, LIGHT_H4, LIGHT_H5, LIGHT_H6, LIGHT_NBINS
};
// Largest tau the light accumulators can hold.
int64_t tau_limit();
// light/heavy row threshold: min(tau, light_row_limit())
int64_t light_row_limit();
// (minc / maxc of B's column type: int64 when ci64; a row whose column span
// does not fit 31 bits is sent to the heavy path)
void light_classes_sym(const int64_t *ip, const void *minc, const void *maxc, bool ci64, int64_t n, int64_t tau,
                       bool window, uint8_t *cls, hipStream_t s);
void light_classes_num(const int64_t *ip, const int64_t *row_nnz, const void *minc, const void *maxc, bool ci64,
                       int64_t n, int64_t tau, bool window, uint8_t *cls, hipStream_t s);
void leaf_classes_sym(const LeafSet &L, int64_t tau, int64_t width, uint8_t *cls, hipStream_t s);
void leaf_classes_num(const LeafSet &L, const int64_t *leaf_nnz, int64_t tau, int64_t width, uint8_t *cls,
                      hipStream_t s);
// Launch record of one leaf, built in bin-partition order: element range
// [s, e); symbolic: t = slot id, a = leaf index; numeric: t = first C
// position, a = nnz written, b = the slot within the row (its first column is
// b << slot width).
struct LeafTask {
    int64_t s, e, t;
    int32_t a, b;
};
void leaf_tasks_sym(const LeafSet &L, const int64_t *items, int64_t n, LeafTask *tasks, hipStream_t s);
void leaf_tasks_num(const LeafSet &L, const int64_t *items, int64_t n, const int64_t *leaf_nnz, int n_slots_log2,
                    const int64_t *heavy_rows, const int64_t *c_row_ptr, const int64_t *slot_off,
                    int slot_width_log2, LeafTask *tasks, hipStream_t s);
// LEAF_DENSE_BIG holds the dense leaves of at least DENSE_BIG_LEN elements; it
// sits just before LEAF_DENSE so one launch covers both bins with the big
// leaves first (they start early instead of finishing last).
constexpr int64_t DENSE_BIG_LEN = 32768;
// Leaf symbolic: leaf_nnz[leaf] and slot_cnt[slot] for the n tasks of a bin.
// (e_end: end of the level's elements in the column array; column loads stay below it)
void leaf_symbolic(const LeafSet &L, int bin, const LeafTask *tasks, int64_t n, int64_t width, int64_t e_end,
                   int64_t *leaf_nnz, int64_t *slot_cnt, hipStream_t s);
// Leaf numeric: writes C at each task's position.
// counter: one device int32 the dense bin uses to hand out chunks.
// (c_col of C's column type: int64 when ci64; c_val of the leaf set's value type)
void leaf_numeric(const LeafSet &L, int bin, const LeafTask *tasks, int64_t n, int64_t width, void *c_col, bool ci64,
                  int slot_width_log2, void *c_val, int32_t *err, int32_t *counter, hipStream_t s);
// Light rows (local index r): symbolic count into row_nnz[r]; numeric into C.
// (minc / maxc of B's column type; C's columns and values of A's and B's types)
// Symbolic of the narrowest window bin (rows spanning at most 64 columns)
// from per-B-row column masks; masks: brow_mask_bytes(B) of workspace.
int64_t brow_mask_bytes(const Csr &B);
void light_symbolic_narrow(const Csr &A, const Csr &B, int64_t r0, const int64_t *items, int64_t n,
                           const void *minc, void *masks, int64_t *row_nnz, hipStream_t s);
void light_symbolic(const Csr &A, const Csr &B, int64_t r0, int bin, const int64_t *items, int64_t n,
                    const void *minc, const void *maxc, int64_t *row_nnz, hipStream_t s);
void light_numeric(const Csr &A, const Csr &B, int64_t r0, int bin, const int64_t *items, int64_t n,
                   const void *minc, const void *maxc, const int64_t *c_row_ptr, void *c_col, void *c_val,
                   int32_t *err, hipStream_t s);
// Per heavy row h: in-place exclusive scan of slot[h*n_slots .. +n_slots),
// row total into row_nnz[heavy_rows[h]].
void slot_scan(int64_t *slot, int64_t n_heavy, int64_t n_slots, const int64_t *heavy_rows, int64_t *row_nnz,
               hipStream_t s);

}  // namespace gm
