/*
 * Seeded synthetic sparse-matrix generators (CSR, int64 row pointers,
 * int32 column indices sorted and unique within a row, fp64 values).
 *
 * This file holds input generation only: it contains none of the SpGEMM
 * arithmetic. Both the CPU oracle side and the GPU side draw their inputs
 * from it, so the two compare on identical matrices.
 *
 * Random numbers come from a counter-based generator (SplitMix64 finaliser
 * applied to key + (counter+1)*golden-gamma), so every draw depends only on
 * (seed, stream, counter) and never on the thread count or schedule.
 *
 * Workload families (the shapes of the paper's evaluation, Section IV-A):
 *   - R-MAT: recursive quadrant draws, most significant bit first, with
 *     probabilities (a, b, c, d); duplicate edges are summed.
 *   - Banded: row i holds columns max(0, i-h) .. min(n-1, i+h).
 *   - Erdos-Renyi: exactly d distinct columns per row, uniform without
 *     replacement (Floyd's sampling).
 *   - Uniform random CSR with a given density (small test matrices).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* Key for an independent stream: seed and stream id folded through the mixer. */
static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
    return mix64(mix64(seed + GOLDEN) ^ (stream * 0xD1B54A32D192ED03ULL));
}

static inline uint64_t draw(uint64_t key, uint64_t ctr) { return mix64(key + (ctr + 1) * GOLDEN); }

/* U[0,1) with 53 random bits. */
static inline double unif01(uint64_t x) { return (double)(x >> 11) * 0x1.0p-53; }

/* Uniform integer in [0, range) via a 128-bit multiply-high (bias < 2^-40 here). */
static inline uint64_t below(uint64_t x, uint64_t range) {
    return (uint64_t)(((unsigned __int128)x * range) >> 64);
}

enum { VAL_U01 = 0, VAL_PM1 = 1, VAL_INT3 = 2, VAL_ONES = 3 };

static inline double make_value(int mode, uint64_t x) {
    switch (mode) {
    case VAL_U01: return unif01(x);
    case VAL_PM1: return 2.0 * unif01(x) - 1.0;
    case VAL_INT3: return (double)((int64_t)below(x, 7) - 3); /* {-3..3} */
    default: return 1.0;
    }
}

typedef struct {
    int64_t n_rows, n_cols, nnz;
    int64_t *row_ptr;
    int32_t *col;
    double *val;
} gm_gen_csr;

void gm_gen_free(gm_gen_csr *m) {
    if (!m) return;
    free(m->row_ptr);
    free(m->col);
    free(m->val);
    free(m);
}

int64_t gm_gen_nnz(const gm_gen_csr *m) { return m->nnz; }

/* Copies the generated CSR into caller buffers (n_rows+1, nnz, nnz). */
void gm_gen_copy(const gm_gen_csr *m, int64_t *row_ptr, int32_t *col, double *val) {
    memcpy(row_ptr, m->row_ptr, (size_t)(m->n_rows + 1) * sizeof(int64_t));
    memcpy(col, m->col, (size_t)m->nnz * sizeof(int32_t));
    memcpy(val, m->val, (size_t)m->nnz * sizeof(double));
}

static int cmp_u64(const void *a, const void *b) {
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return (x > y) - (x < y);
}

/* Builds canonical CSR from an edge list (row, col, val per edge index e):
 * rows bucketed, each row sorted by (col, e), duplicates summed in e order. */
static gm_gen_csr *from_edges(int64_t n_rows, int64_t n_cols, int64_t n_edges, const int32_t *er,
                              const int32_t *ec, const double *ev) {
    gm_gen_csr *m = (gm_gen_csr *)calloc(1, sizeof(gm_gen_csr));
    int64_t *cnt = (int64_t *)calloc((size_t)n_rows + 1, sizeof(int64_t));
    uint64_t *keys = (uint64_t *)malloc((size_t)(n_edges > 0 ? n_edges : 1) * sizeof(uint64_t));
    int64_t *cur = (int64_t *)malloc(((size_t)n_rows + 1) * sizeof(int64_t));
    int64_t *uniq = (int64_t *)calloc((size_t)n_rows + 1, sizeof(int64_t));
    if (!m || !cnt || !keys || !cur || !uniq) goto fail;

#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n_edges; ++e) __atomic_fetch_add(&cnt[er[e] + 1], 1, __ATOMIC_RELAXED);
    for (int64_t i = 0; i < n_rows; ++i) cnt[i + 1] += cnt[i];
    memcpy(cur, cnt, ((size_t)n_rows + 1) * sizeof(int64_t));
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < n_edges; ++e) {
        int64_t p = __atomic_fetch_add(&cur[er[e]], 1, __ATOMIC_RELAXED);
        keys[p] = ((uint64_t)(uint32_t)ec[e] << 32) | (uint64_t)e;
    }
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t i = 0; i < n_rows; ++i) {
        int64_t b = cnt[i], len = cnt[i + 1] - cnt[i];
        if (len > 1) qsort(keys + b, (size_t)len, sizeof(uint64_t), cmp_u64);
        int64_t u = 0;
        for (int64_t p = b; p < b + len; ++p)
            if (p == b || (keys[p] >> 32) != (keys[p - 1] >> 32)) ++u;
        uniq[i + 1] = u;
    }
    for (int64_t i = 0; i < n_rows; ++i) uniq[i + 1] += uniq[i];
    m->n_rows = n_rows;
    m->n_cols = n_cols;
    m->nnz = uniq[n_rows];
    m->row_ptr = uniq;
    uniq = NULL;
    m->col = (int32_t *)malloc((size_t)(m->nnz > 0 ? m->nnz : 1) * sizeof(int32_t));
    m->val = (double *)malloc((size_t)(m->nnz > 0 ? m->nnz : 1) * sizeof(double));
    if (!m->col || !m->val) goto fail;
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t i = 0; i < n_rows; ++i) {
        int64_t q = m->row_ptr[i] - 1;
        for (int64_t p = cnt[i]; p < cnt[i + 1]; ++p) {
            uint32_t c = (uint32_t)(keys[p] >> 32);
            double v = ev[keys[p] & 0xFFFFFFFFULL];
            if (p == cnt[i] || c != (uint32_t)(keys[p - 1] >> 32)) {
                ++q;
                m->col[q] = (int32_t)c;
                m->val[q] = v;
            } else {
                m->val[q] += v;
            }
        }
    }
    free(cnt);
    free(keys);
    free(cur);
    return m;
fail:
    free(cnt);
    free(keys);
    free(cur);
    free(uniq);
    gm_gen_free(m);
    return NULL;
}

/* R-MAT with 2^scale rows/cols and edge_factor * 2^scale edge draws. Each of
 * the scale levels of an edge draws one uniform and picks a quadrant:
 * [0,a) -> (0,0), [a,a+b) -> (0,1), [a+b,a+b+c) -> (1,0), else (1,1).
 * Self-loops are kept; duplicate (row, col) draws are summed. */
gm_gen_csr *gm_gen_rmat(int32_t scale, int64_t edge_factor, double a, double b, double c,
                        uint64_t seed, int32_t value_mode) {
    if (scale < 1 || scale > 30 || edge_factor < 1) return NULL;
    int64_t n = (int64_t)1 << scale;
    int64_t E = edge_factor * n;
    if (E >= ((int64_t)1 << 32)) return NULL;
    int32_t *er = (int32_t *)malloc((size_t)E * sizeof(int32_t));
    int32_t *ec = (int32_t *)malloc((size_t)E * sizeof(int32_t));
    double *ev = (double *)malloc((size_t)E * sizeof(double));
    if (!er || !ec || !ev) {
        free(er); free(ec); free(ev);
        return NULL;
    }
    const uint64_t kq = stream_key(seed, 1), kv = stream_key(seed, 2);
    const double ab = a + b, abc = a + b + c;
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < E; ++e) {
        uint32_t r = 0, q = 0;
        for (int32_t l = 0; l < scale; ++l) {
            double u = unif01(draw(kq, (uint64_t)e * (uint64_t)scale + (uint64_t)l));
            uint32_t rb = (u >= ab), cb = (u >= a && u < ab) || (u >= abc);
            r = (r << 1) | rb;
            q = (q << 1) | cb;
        }
        er[e] = (int32_t)r;
        ec[e] = (int32_t)q;
        ev[e] = make_value(value_mode, draw(kv, (uint64_t)e));
    }
    gm_gen_csr *m = from_edges(n, n, E, er, ec, ev);
    free(er);
    free(ec);
    free(ev);
    return m;
}

/* Banded n x n matrix, row i holding columns max(0,i-h)..min(n-1,i+h). */
gm_gen_csr *gm_gen_banded(int64_t n, int32_t half, uint64_t seed, int32_t value_mode) {
    if (n < 1 || half < 0 || n >= ((int64_t)1 << 31)) return NULL;
    gm_gen_csr *m = (gm_gen_csr *)calloc(1, sizeof(gm_gen_csr));
    if (!m) return NULL;
    m->n_rows = m->n_cols = n;
    m->row_ptr = (int64_t *)malloc(((size_t)n + 1) * sizeof(int64_t));
    if (!m->row_ptr) { gm_gen_free(m); return NULL; }
    m->row_ptr[0] = 0;
    for (int64_t i = 0; i < n; ++i) {
        int64_t lo = i - half < 0 ? 0 : i - half, hi = i + half > n - 1 ? n - 1 : i + half;
        m->row_ptr[i + 1] = m->row_ptr[i] + (hi - lo + 1);
    }
    m->nnz = m->row_ptr[n];
    m->col = (int32_t *)malloc((size_t)m->nnz * sizeof(int32_t));
    m->val = (double *)malloc((size_t)m->nnz * sizeof(double));
    if (!m->col || !m->val) { gm_gen_free(m); return NULL; }
    const uint64_t kv = stream_key(seed, 3);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        int64_t lo = i - half < 0 ? 0 : i - half;
        for (int64_t p = m->row_ptr[i]; p < m->row_ptr[i + 1]; ++p) {
            m->col[p] = (int32_t)(lo + (p - m->row_ptr[i]));
            m->val[p] = make_value(value_mode, draw(kv, (uint64_t)p));
        }
    }
    return m;
}

static int cmp_i32(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* n_rows x n_cols with exactly d distinct uniform columns per row (Floyd). */
gm_gen_csr *gm_gen_erdos_renyi(int64_t n_rows, int64_t n_cols, int32_t d, uint64_t seed,
                               int32_t value_mode) {
    if (n_rows < 0 || n_cols < 1 || d < 0 || d > n_cols || n_cols >= ((int64_t)1 << 31)) return NULL;
    gm_gen_csr *m = (gm_gen_csr *)calloc(1, sizeof(gm_gen_csr));
    if (!m) return NULL;
    m->n_rows = n_rows;
    m->n_cols = n_cols;
    m->nnz = n_rows * d;
    m->row_ptr = (int64_t *)malloc(((size_t)n_rows + 1) * sizeof(int64_t));
    m->col = (int32_t *)malloc((size_t)(m->nnz > 0 ? m->nnz : 1) * sizeof(int32_t));
    m->val = (double *)malloc((size_t)(m->nnz > 0 ? m->nnz : 1) * sizeof(double));
    if (!m->row_ptr || !m->col || !m->val) { gm_gen_free(m); return NULL; }
    for (int64_t i = 0; i <= n_rows; ++i) m->row_ptr[i] = i * d;
    const uint64_t kc = stream_key(seed, 4), kv = stream_key(seed, 5);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_rows; ++i) {
        int32_t *cols = m->col + i * d;
        int32_t k = 0;
        for (int64_t j = n_cols - d; j < n_cols; ++j) {
            int64_t t = (int64_t)below(draw(kc, (uint64_t)i * (uint64_t)d + (uint64_t)k), (uint64_t)j + 1);
            int dup = 0;
            for (int32_t q = 0; q < k; ++q)
                if (cols[q] == (int32_t)t) { dup = 1; break; }
            cols[k++] = dup ? (int32_t)j : (int32_t)t;
        }
        qsort(cols, (size_t)d, sizeof(int32_t), cmp_i32);
        for (int32_t q = 0; q < d; ++q)
            m->val[i * d + q] = make_value(value_mode, draw(kv, (uint64_t)(i * d + q)));
    }
    return m;
}

/* Each entry present independently with probability `density`. */
gm_gen_csr *gm_gen_uniform(int64_t n_rows, int64_t n_cols, double density, uint64_t seed,
                           int32_t value_mode) {
    if (n_rows < 0 || n_cols < 1 || n_cols >= ((int64_t)1 << 31)) return NULL;
    gm_gen_csr *m = (gm_gen_csr *)calloc(1, sizeof(gm_gen_csr));
    if (!m) return NULL;
    m->n_rows = n_rows;
    m->n_cols = n_cols;
    m->row_ptr = (int64_t *)calloc(((size_t)n_rows + 1), sizeof(int64_t));
    if (!m->row_ptr) { gm_gen_free(m); return NULL; }
    const uint64_t kp = stream_key(seed, 6), kv = stream_key(seed, 7);
    for (int64_t i = 0; i < n_rows; ++i) {
        int64_t c = 0;
        for (int64_t j = 0; j < n_cols; ++j)
            if (unif01(draw(kp, (uint64_t)(i * n_cols + j))) < density) ++c;
        m->row_ptr[i + 1] = m->row_ptr[i] + c;
    }
    m->nnz = m->row_ptr[n_rows];
    m->col = (int32_t *)malloc((size_t)(m->nnz > 0 ? m->nnz : 1) * sizeof(int32_t));
    m->val = (double *)malloc((size_t)(m->nnz > 0 ? m->nnz : 1) * sizeof(double));
    if (!m->col || !m->val) { gm_gen_free(m); return NULL; }
    for (int64_t i = 0; i < n_rows; ++i) {
        int64_t p = m->row_ptr[i];
        for (int64_t j = 0; j < n_cols; ++j)
            if (unif01(draw(kp, (uint64_t)(i * n_cols + j))) < density) {
                m->col[p] = (int32_t)j;
                m->val[p] = make_value(value_mode, draw(kv, (uint64_t)p));
                ++p;
            }
    }
    return m;
}

int gm_gen_threads(void) { return omp_get_max_threads(); }
