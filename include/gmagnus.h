/*
 * gmagnus.h -- C ABI of an MI355X (gfx950) SpGEMM, C = A * B on CSR, built on
 * the heavy-row method of "gMAGNUS: Fast SpGEMM on GPUs for Irregular Matrices
 * via Hierarchical Multisplit".
 *
 * What is computed (Section II-B, Eq. gustav): row i of C is the sum over the
 * nonzeros A[i,k] of A[i,k] * B[k,:]. The pattern of C holds every (i, j)
 * reached by at least one product A[i,k]*B[k,j], including entries whose sum
 * is exactly zero. Output rows have strictly increasing columns.
 *
 * How (Algorithm 3): rows whose product count exceeds a local-memory
 * threshold tau are "heavy". Heavy rows are expanded by an outer product into
 * an intermediate matrix (Section III-B, Algorithm 4), split into column
 * chunks by a hierarchical multisplit (Section III-C, Algorithm 5) until every
 * chunk's column range fits a dense accumulator in LDS, and accumulated chunk
 * by chunk; light rows and light chunks use an LDS hash or dense-window
 * accumulator (Section III-E). Parameters follow Section III-D.
 *
 * Conventions shared by every entry point
 *   - All matrix arrays are DEVICE pointers (hipMalloc'ed or torch tensors on
 *     the current device). Sizes and scalars are host values.
 *   - Index types: int64 row pointers; int32 column indices and fp64 values
 *     through gmagnus_csr_t, or int32 / int64 column indices and fp64 / fp32
 *     values through gmagnus_matrix_t and the *_typed entry points (C takes
 *     the types of A and B, which must agree).
 *   - Input CSR must be canonical: row_ptr[0] = 0, non-decreasing,
 *     row_ptr[n_rows] = nnz, columns in [0, n_cols) and strictly increasing
 *     within each row. options.validate = 1 checks this on the device.
 *   - All work is ordered on the HIP stream given to gmagnus_plan (NULL = the
 *     null stream). Calls that return sizes to the host synchronise it.
 *   - Errors are reported by status code; no entry point aborts or throws.
 *     gmagnus_last_error() returns a message for the calling thread's last
 *     failure.
 *   - A plan is not thread-safe. Different plans on different streams may be
 *     used concurrently.
 */
#ifndef GMAGNUS_H
#define GMAGNUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GMAGNUS_SUCCESS = 0,
    GMAGNUS_ERROR_INVALID_VALUE = 1, /* bad argument: NULL pointer, shape mismatch, bad option */
    GMAGNUS_ERROR_INVALID_CSR = 2,   /* validate = 1 found a non-canonical input */
    GMAGNUS_ERROR_OUT_OF_MEMORY = 3, /* device workspace could not be allocated */
    GMAGNUS_ERROR_NOT_READY = 4,     /* call order violated (numeric before symbolic) */
    GMAGNUS_ERROR_HIP = 5,           /* a HIP runtime call or kernel launch failed */
    GMAGNUS_ERROR_UNSUPPORTED = 6    /* size beyond the library's limits (e.g. > 2^31-1 columns) */
} gmagnus_status_t;

/* A CSR matrix in device memory (Section II-A notation: rowPtr, col, val). */
typedef struct {
    int64_t n_rows;
    int64_t n_cols;
    int64_t nnz;
    const int64_t *row_ptr; /* device, n_rows + 1 */
    const int32_t *col_idx; /* device, nnz */
    const double *val;      /* device, nnz */
} gmagnus_csr_t;

/* Column-index and value types (the s_col and s_val of Section III-D). */
typedef enum { GMAGNUS_INDEX_INT32 = 0, GMAGNUS_INDEX_INT64 = 1 } gmagnus_index_type_t;
typedef enum { GMAGNUS_VALUE_FP64 = 0, GMAGNUS_VALUE_FP32 = 1 } gmagnus_value_type_t;

/* A CSR matrix in device memory with its types named. With int64 column
 * indices B (and C) may have up to 2^35 columns; every other dimension,
 * A's columns included, stays below 2^31. */
typedef struct {
    int64_t n_rows;
    int64_t n_cols;
    int64_t nnz;
    const int64_t *row_ptr; /* device, n_rows + 1 */
    const void *col_idx;    /* device, nnz int32_t or int64_t (index_type) */
    const void *val;        /* device, nnz double or float (value_type) */
    int32_t index_type;     /* gmagnus_index_type_t */
    int32_t value_type;     /* gmagnus_value_type_t */
} gmagnus_matrix_t;

/* Options. Zero fields mean "derive" (Section III-D); initialise with
 * gmagnus_options_init. The overrides exist so tests can force any number of
 * multisplit levels on small inputs; C does not depend on them. */
typedef struct {
    size_t struct_size;          /* sizeof(gmagnus_options_t) */
    int64_t row_begin, row_end;  /* row panel of A (and C); row_end = 0 means n_rows */
    int64_t lds_bytes;           /* s_LM; 0 = the device's LDS per workgroup (160 KB) */
    int64_t tau;                 /* heavy threshold; 0 = derived; clamped to the light-path capacity */
    int32_t dense_width_log2;    /* log2 W of the dense accumulator; 0 = derived (13 for 160 KB) */
    int32_t chunks_max_log2;     /* log2 of the per-level chunk limit; 0 = derived (5 for 160 KB) */
    int32_t validate;            /* 1 = check canonical CSR of A and B on the device */
    int32_t flags;               /* GMAGNUS_FLAG_* bits */
    /* Optional workspace allocator (device memory). NULL = the library's own
     * caching allocator. free() receives exactly the pointers alloc() returned. */
    void *(*alloc)(size_t bytes, void *stream, void *ctx);
    void (*free)(void *ptr, void *stream, void *ctx);
    void *alloc_ctx;
    /* Bound on the device workspace one plan holds at any time, in bytes
     * (0 = none). A plan that would need more fails with
     * GMAGNUS_ERROR_OUT_OF_MEMORY and releases what it holds. */
    int64_t workspace_limit_bytes;
} gmagnus_options_t;

#define GMAGNUS_FLAG_TIMING 1u         /* record per-phase device times (HIP events) into the plan info */
#define GMAGNUS_FLAG_SERIAL_STREAMS 2u /* run heavy and light work on one stream (the default; kept so callers
                                          that ask for it explicitly keep working) */
#define GMAGNUS_FLAG_NO_WINDOW 4u      /* never use the dense-window accumulator for light rows */
#define GMAGNUS_FLAG_PAPER_HISTOGRAM 8u /* level-0 histogram by a pass over C-hat's columns (the paper's
                                           kernel) instead of from the structure of A and B;
                                           implies GMAGNUS_FLAG_PAPER_EXPANSION */
#define GMAGNUS_FLAG_PAPER_EXPANSION 16u /* write C-hat row by row, then split it at the first level (the
                                            paper's order), instead of splitting during the expansion */
#define GMAGNUS_FLAG_SLICE_SPLIT 32u /* split during the expansion in the paper's slice order (runs written at
                                        atomic cursors) instead of the chunk-major row order */
#define GMAGNUS_FLAG_CONCURRENT_STREAMS 128u /* run the heavy rows and the light rows on two streams joined
                                               with events (Algorithm 3's two queues) instead of one after the
                                               other; measured slower on R-MAT scale 22, where the light rows'
                                               kernels take CU slots from the bandwidth-bound heavy kernels */
#define GMAGNUS_FLAG_LEVEL_BY_LEVEL 64u /* with two multisplit levels, write the first level's heavy chunks out
                                           and split them in a pass of their own, instead of splitting them again
                                           inside the expansion and writing the final chunks directly */
#define GMAGNUS_FLAG_KEEP_PATTERN 256u /* keep the heavy path's structural buffers after symbolic so that
                                          gmagnus_update_values can recompute C for new values of A and B
                                          on the same patterns (costs the memory of those buffers) */

#define GMAGNUS_MAX_LEVELS 8

/* Parameters chosen by the planner (Section III-D, GetMagnusParams). */
typedef struct {
    int64_t tau;             /* heavy threshold on product counts (rows and chunks) */
    int64_t dense_width;     /* W: column width of a final chunk (dense accumulator) */
    int64_t chunks_required; /* ceil_pow2(C.m) / W, at least 1 */
    int64_t chunks_max;      /* chunks one multisplit level may create */
    int64_t min_group_elems; /* elements per multisplit work group (lower bound) */
    int64_t group_rows;      /* rows one multisplit work group can touch */
    int32_t n_levels;        /* multisplit levels (0 when C.m <= W) */
    int32_t v_chunks[GMAGNUS_MAX_LEVELS]; /* chunks per row at each level */
} gmagnus_params_t;

/* Kernel classes timed under GMAGNUS_FLAG_TIMING. */
enum {
    GMAGNUS_K_SETUP = 0,       /* row products, binning, partitions, scans */
    GMAGNUS_K_CSC = 1,         /* masked CSR->CSC of heavy rows and slice offsets */
    GMAGNUS_K_EXPAND = 2,      /* outer-product expansion into C-hat */
    GMAGNUS_K_HISTOGRAM = 3,   /* level-0 chunk histogram */
    GMAGNUS_K_MULTISPLIT = 4,  /* multisplit levels (with fused next-level histogram) */
    GMAGNUS_K_CHUNK_SYM = 5,   /* symbolic of final chunks */
    GMAGNUS_K_CHUNK_NUM = 6,   /* numeric of final chunks (writes C) */
    GMAGNUS_K_LIGHT_SYM = 7,   /* symbolic of light rows */
    GMAGNUS_K_LIGHT_NUM = 8,   /* numeric of light rows (writes C) */
    GMAGNUS_K_ROWPTR = 9,      /* fragment offsets and the C row-pointer scan */
    GMAGNUS_K_COUNT = 10
};

/* Counts and timings of one plan (one row panel). */
typedef struct {
    gmagnus_params_t params;
    int64_t n_rows;                /* rows in the panel */
    int64_t n_heavy_rows;          /* rows with more than row_tau products */
    int64_t n_light_rows;          /* rows with 1..row_tau products */
    int64_t products_total;        /* sum of products over the panel's rows */
    int64_t products_heavy;        /* products of heavy rows = nnz of C-hat */
    int64_t n_slices;              /* outer-product slices (columns of the masked A) */
    int64_t nnz_a_heavy;           /* nonzeros of A in heavy rows with a nonempty B row */
    int64_t level_rows_in[GMAGNUS_MAX_LEVELS];     /* input rows of each multisplit level */
    int64_t level_elems_in[GMAGNUS_MAX_LEVELS];    /* input elements of each level */
    int64_t level_heavy_out[GMAGNUS_MAX_LEVELS];   /* heavy chunks produced by each level */
    int32_t levels_run;            /* levels actually executed (early exit when no heavy chunk) */
    int64_t n_leaves_dense;        /* final chunks accumulated densely */
    int64_t n_leaves_hash;         /* final chunks accumulated with the hash map */
    int64_t n_leaves_rank;         /* final chunks accumulated with the bitmap-rank accumulator */
    int64_t c_nnz;                 /* nonzeros of the panel of C (after symbolic) */
    int64_t c_nnz_heavy;           /* of which in heavy rows */
    int32_t check_flags;           /* nonzero: a kernel's output count disagreed with symbolic (a bug) */
    int32_t expansion_path;        /* GMAGNUS_PATH_* the heavy rows took */
    int64_t workspace_peak_bytes;  /* largest device workspace the plan has held */
    int32_t index_type;            /* gmagnus_index_type_t of A, B and C */
    int32_t value_type;            /* gmagnus_value_type_t of A, B and C */
    /* Under GMAGNUS_FLAG_TIMING: summed device milliseconds, launches and
     * algorithmic (compulsory) HBM bytes per kernel class. */
    double kernel_ms[GMAGNUS_K_COUNT];
    int64_t kernel_launches[GMAGNUS_K_COUNT];
    double kernel_bytes[GMAGNUS_K_COUNT];
    /* Light/heavy row threshold: min(tau, 3456). Rows of 3457..tau products
     * take the heavy path (their chunks are all light); chunks are classified
     * by tau itself. */
    int64_t row_tau;
} gmagnus_plan_info_t;

/* Expansion orders of the heavy rows (Section III-B), as chosen by
 * gmagnus_expansion_path and reported in gmagnus_plan_info_t. */
enum {
    GMAGNUS_PATH_NONE = 0,           /* no heavy rows */
    GMAGNUS_PATH_PAPER = 1,          /* C-hat written row by row (Algorithm 4), then split level by level */
    GMAGNUS_PATH_SLICE_SPLIT = 2,    /* first level split during a slice-order expansion (atomic cursors) */
    GMAGNUS_PATH_ROWS = 3,           /* first level split during a chunk-major row-order expansion */
    GMAGNUS_PATH_ROWS_TWO_LEVEL = 4  /* both levels of a two-level hierarchy split during the row-order expansion */
};

typedef struct gmagnus_plan_s *gmagnus_plan_t;

/* Fills *opts with defaults (all derive; whole matrix). */
void gmagnus_options_init(gmagnus_options_t *opts);

/* Host-only parameter selection (Section III-D) for a product with c_m
 * columns and s_LM = lds_bytes; the option overrides (tau, dense_width_log2,
 * chunks_max_log2) apply when opts is not NULL. No device is touched.
 * Errors: INVALID_VALUE for c_m < 1, lds_bytes < 1024 or inconsistent overrides. */
gmagnus_status_t gmagnus_get_params(int64_t c_m, int64_t lds_bytes, const gmagnus_options_t *opts,
                                    gmagnus_params_t *out);

/* Host-only parameter selection for the given column-index and value types
 * (Section III-D: tau from s_col + s_val, W from s_val, the multisplit group
 * and chunk limits from both). The library caps tau at the light-row
 * accumulators' capacity (6912 products) and W at 8192 columns (its dense
 * accumulator and narrow bitmap shapes); fp32 values derive tau = 10240 and
 * W = 16384 at 160 KB and are capped. Errors as gmagnus_get_params, plus
 * INVALID_VALUE for an unknown type and c_m beyond the index type's range. */
gmagnus_status_t gmagnus_get_params_typed(int64_t c_m, int64_t lds_bytes, int32_t index_type, int32_t value_type,
                                          const gmagnus_options_t *opts, gmagnus_params_t *out);

/* Host-only: the expansion order a plan with these parameters takes for a
 * panel with n_heavy heavy rows holding products_heavy products, with B
 * holding b_nnz entries and the given GMAGNUS_FLAG_* bits. No device is
 * touched. NULL params gives GMAGNUS_PATH_NONE. */
int32_t gmagnus_expansion_path(const gmagnus_params_t *params, int64_t n_heavy, int64_t products_heavy,
                               int64_t b_nnz, int32_t flags);

/* Setup phase of Algorithm 3 for rows [row_begin, row_end) of C = A*B:
 * parameter selection, per-row product counts (InterOffsets) and the
 * light/heavy split (ThreshPartition). A and B are borrowed: they must stay
 * valid and unchanged until gmagnus_plan_destroy. Synchronises the stream.
 * Errors: INVALID_VALUE (NULL, A.n_cols != B.n_rows, bad panel), UNSUPPORTED
 * (n_cols >= 2^31), INVALID_CSR (validate), OUT_OF_MEMORY, HIP. */
gmagnus_status_t gmagnus_plan(gmagnus_plan_t *out, const gmagnus_csr_t *A, const gmagnus_csr_t *B,
                              const gmagnus_options_t *opts, void *hip_stream);

/* gmagnus_plan for typed matrices (Section III-D's type sizes): A and B must
 * have the same index and value types, which C takes. Errors as gmagnus_plan,
 * plus INVALID_VALUE for unknown or mismatched types, UNSUPPORTED beyond the
 * limits of gmagnus_matrix_t. */
gmagnus_status_t gmagnus_plan_typed(gmagnus_plan_t *out, const gmagnus_matrix_t *A, const gmagnus_matrix_t *B,
                                    const gmagnus_options_t *opts, void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops or harnesses that forbid allocation): the same plan
 * as gmagnus_plan, with its whole device workspace carved from a static
 * device array of GMAGNUS_STATIC_WORKSPACE_MIB MiB that each device holds
 * from the first call on it until the process ends. Neither this call nor
 * symbolic / numeric / update_values on the plan calls hipMalloc, hipFree or
 * any other allocating routine of HIP (host reads use pageable memory);
 * A, B and C stay the caller's. Plans made this way on one device take
 * disjoint blocks of the array, so they may coexist, but together they are
 * bounded by its size; blocks go back when the plan is destroyed, and hold
 * whatever the last plan wrote (nothing relies on their contents).
 * opts must not set alloc / free; workspace_limit_bytes is capped at the
 * array's size. Errors: as gmagnus_plan; UNSUPPORTED when the panel has more
 * rows than the array could hold the setup work of (about 3.2 million rows
 * for 128 MiB); OUT_OF_MEMORY from this call or a later phase when the
 * array cannot hold the next block the plan needs (the plan then fails
 * cleanly and gives its blocks back). */
#define GMAGNUS_STATIC_WORKSPACE_MIB 128
gmagnus_status_t gmagnus_plan_static(gmagnus_plan_t *out, const gmagnus_csr_t *A, const gmagnus_csr_t *B,
                                     const gmagnus_options_t *opts, void *hip_stream);

/* Symbolic phase: runs the heavy-row expansion and hierarchical multisplit
 * (Algorithm 3, outer product and reorder), counts the distinct columns of
 * every light row and final chunk, and writes the panel's row pointers:
 * c_row_ptr (device, panel_rows + 1, starting at 0) and *c_nnz (host).
 * Synchronises the stream (C.nnz is needed on the host to size C).
 * Errors: INVALID_VALUE (NULL), OUT_OF_MEMORY, HIP. */
gmagnus_status_t gmagnus_spgemm_symbolic(gmagnus_plan_t plan, int64_t *c_row_ptr, int64_t *c_nnz);

/* Numeric phase: accumulates every light row and final chunk and writes
 * c_col_idx / c_val (device, c_nnz entries each) at the offsets given by
 * c_row_ptr (the array symbolic filled; it must be unchanged). Columns come
 * out strictly increasing within each row. Asynchronous on the plan's stream.
 * Errors: INVALID_VALUE (NULL), NOT_READY (symbolic has not run), HIP. */
gmagnus_status_t gmagnus_spgemm_numeric(gmagnus_plan_t plan, const int64_t *c_row_ptr, int32_t *c_col_idx,
                                        double *c_val);

/* gmagnus_spgemm_numeric for any plan: c_col_idx and c_val have the plan's
 * index and value types (int32 / int64, double / float). gmagnus_spgemm_numeric
 * itself accepts only plans of int32 columns and fp64 values
 * (INVALID_VALUE otherwise). */
gmagnus_status_t gmagnus_spgemm_numeric_typed(gmagnus_plan_t plan, const int64_t *c_row_ptr, void *c_col_idx,
                                              void *c_val);

/* Pattern reuse: the symbolic phase depends on the nonzero patterns of A and
 * B only (Section II-A: it fixes C.rowPtr and C.nnz; the numeric phase fills
 * the values), so repeated products on fixed patterns with changing values
 * (algebraic multigrid's Galerkin products, Section I) need the symbolic
 * work once. This call replaces the values of A and B the plan reads with
 * a_val (A.nnz doubles, in A's CSR order) and b_val (B.nnz doubles, in B's
 * CSR order), device pointers the caller keeps alive and unchanged until the
 * plan's next numeric phase has finished (they may be the arrays given at
 * gmagnus_plan, and a_val may equal b_val when A and B are one matrix). It
 * redoes only the value-producing passes of the heavy rows (the outer-product
 * expansion and the multisplit levels, on the layout symbolic computed);
 * gmagnus_spgemm_numeric then writes C for the new values into the structure
 * symbolic produced, with the same c_row_ptr. Asynchronous on the plan's
 * stream. Requires GMAGNUS_FLAG_KEEP_PATTERN at gmagnus_plan.
 * Errors: INVALID_VALUE (NULL values with nonzeros present, or the plan was
 * made without GMAGNUS_FLAG_KEEP_PATTERN), NOT_READY (symbolic has not run),
 * HIP. */
gmagnus_status_t gmagnus_update_values(gmagnus_plan_t plan, const double *a_val, const double *b_val);

/* gmagnus_update_values for any plan: a_val and b_val hold the plan's value
 * type (gmagnus_update_values itself requires fp64 values). */
gmagnus_status_t gmagnus_update_values_typed(gmagnus_plan_t plan, const void *a_val, const void *b_val);

/* Copies the plan's parameters, counts and (with GMAGNUS_FLAG_TIMING) kernel
 * timings. Synchronises the stream when timings are requested. */
gmagnus_status_t gmagnus_plan_info(gmagnus_plan_t plan, gmagnus_plan_info_t *out);

/* Releases the plan's workspace (after synchronising its stream). NULL is a no-op. */
void gmagnus_plan_destroy(gmagnus_plan_t plan);

/* Product counts per row (InterOffsets, Algorithm 3): ip[i] = sum over the
 * nonzeros A[i,k] of nnz(B[k,:]) for i in [0, A.n_rows); ip is a device array
 * of A.n_rows int64. Asynchronous on hip_stream.
 * Errors: INVALID_VALUE, UNSUPPORTED, HIP. */
gmagnus_status_t gmagnus_row_products(const gmagnus_csr_t *A, const gmagnus_csr_t *B, int64_t *ip,
                                      void *hip_stream);

/* gmagnus_row_products for typed matrices (only A's columns and B's row
 * pointers are read). */
gmagnus_status_t gmagnus_row_products_typed(const gmagnus_matrix_t *A, const gmagnus_matrix_t *B, int64_t *ip,
                                            void *hip_stream);

/* Splits the rows of A into consecutive panels whose product counts stay at
 * or below max_products each (a row above the limit gets a panel of its own)
 * so that C can be produced panel by panel when it does not fit in memory.
 * bounds (host, max_panels + 1 entries) receives row boundaries
 * 0 = b[0] < b[1] < ... < b[n] = A.n_rows; *n_panels receives n.
 * Synchronises the stream. Errors: INVALID_VALUE (also when more than
 * max_panels panels are needed), OUT_OF_MEMORY, HIP. */
gmagnus_status_t gmagnus_split_panels(const gmagnus_csr_t *A, const gmagnus_csr_t *B, int64_t max_products,
                                      int64_t *bounds, int64_t max_panels, int64_t *n_panels, void *hip_stream);

/* gmagnus_split_panels for typed matrices. */
gmagnus_status_t gmagnus_split_panels_typed(const gmagnus_matrix_t *A, const gmagnus_matrix_t *B, int64_t max_products,
                                            int64_t *bounds, int64_t max_panels, int64_t *n_panels, void *hip_stream);

/* Streaming bandwidth probe (the measured peak of the speed-of-light
 * comparison, Section IV-C): runs one kernel of the given kind over `bytes`
 * bytes (16-byte elements, grid-stride loop over `grid` work groups of 256
 * threads; grid <= 0 picks one), once to warm up and then `reps` times, and
 * returns the mean time of one run in *ms (host). Kinds:
 *   READ, READ_NT   read src (ordinary / nontemporal loads); dst is a sink of
 *                   at least 8 bytes that is written only if the loaded values
 *                   sum to -1
 *   WRITE, WRITE_NT write dst (ordinary / nontemporal stores)
 *   COPY            copy src to dst (bytes read plus bytes written moved)
 *   GATHER          read 4 GiB as random 128-byte lines of the first `bytes`
 *                   bytes of src (a power of two, 4 KiB .. 128 GiB; grid is
 *                   ignored): the rate of line gathers from a working set of
 *                   that size, i.e. what the caches in front of HBM serve;
 *                   dst is a sink as for READ
 * src and dst are device pointers, 16-byte aligned, of `bytes` bytes (dst: 8
 * bytes for the read kinds). Synchronises the stream.
 * Errors: INVALID_VALUE (kind, sizes, alignment, NULL), HIP. */
enum {
    GMAGNUS_PROBE_READ = 0,
    GMAGNUS_PROBE_READ_NT = 1,
    GMAGNUS_PROBE_WRITE = 2,
    GMAGNUS_PROBE_WRITE_NT = 3,
    GMAGNUS_PROBE_COPY = 4,
    GMAGNUS_PROBE_GATHER = 5
};
gmagnus_status_t gmagnus_bandwidth_probe(int32_t kind, void *dst, const void *src, int64_t bytes, int32_t grid,
                                         int32_t reps, void *hip_stream, double *ms);

/* Frees device blocks cached by the library's allocator (no plan may be alive). */
void gmagnus_release_cache(void);

/* Message for the calling thread's most recent failure ("" if none). */
const char *gmagnus_last_error(void);

/* Static name of a status code. */
const char *gmagnus_status_string(gmagnus_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* GMAGNUS_H */
