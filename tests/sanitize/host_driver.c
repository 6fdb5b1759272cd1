/*
 * Host-side driver for a sanitizer build (AddressSanitizer + UndefinedBehavior
 * Sanitizer) of the input generators (workloads/gen.c) and the CPU oracle
 * (oracle/spgemm_oracle.c): generates small matrices of every family, runs
 * every oracle entry point on them and checks that the results agree with
 * each other (row products, distinct counts by sorting and by marking, the
 * filled rows). Exit status 0 when all checks pass; the sanitizers abort on
 * the first memory or undefined-behaviour error.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct {
    int64_t n_rows, n_cols, nnz;
    int64_t *row_ptr;
    int32_t *col;
    double *val;
} gm_gen_csr;
gm_gen_csr *gm_gen_rmat(int32_t scale, int64_t edge_factor, double a, double b, double c, uint64_t seed,
                        int32_t value_mode);
gm_gen_csr *gm_gen_banded(int64_t n, int32_t half, uint64_t seed, int32_t value_mode);
gm_gen_csr *gm_gen_erdos_renyi(int64_t n_rows, int64_t n_cols, int32_t d, uint64_t seed, int32_t value_mode);
gm_gen_csr *gm_gen_uniform(int64_t n_rows, int64_t n_cols, double density, uint64_t seed, int32_t value_mode);
void gm_gen_free(gm_gen_csr *m);

typedef struct {
    int64_t n_rows, n_cols;
    const int64_t *row_ptr;
    const int64_t *col;
    const double *val;
} oracle_csr;
void oracle_row_products(const oracle_csr *A, const oracle_csr *B, int64_t *ip);
int oracle_count_rows(const oracle_csr *A, const oracle_csr *B, const int64_t *rows, int64_t n_list, int64_t *counts);
int oracle_fill_rows(const oracle_csr *A, const oracle_csr *B, const int64_t *rows, int64_t n_list,
                     const int64_t *offsets, int64_t *col, double *val, double *bound, int64_t *terms);
int oracle_row_counts(const oracle_csr *A, const oracle_csr *B, int64_t row_begin, int64_t row_end,
                      int64_t *counts);

static int failures = 0;
#define CHECK(cond, ...)                              \
    do {                                              \
        if (!(cond)) {                                \
            fprintf(stderr, "check failed: " __VA_ARGS__); \
            fprintf(stderr, "\n");                    \
            ++failures;                               \
        }                                             \
    } while (0)

/* C = M * M through every oracle entry point; returns 0 on agreement. */
static void run(const char *name, gm_gen_csr *m) {
    if (!m) {
        fprintf(stderr, "%s: generator failed\n", name);
        ++failures;
        return;
    }
    int64_t *col64 = (int64_t *)malloc((size_t)(m->nnz > 0 ? m->nnz : 1) * sizeof(int64_t));
    for (int64_t e = 0; e < m->nnz; ++e) col64[e] = m->col[e];
    oracle_csr A = {m->n_rows, m->n_cols, m->row_ptr, col64, m->val};
    const int64_t n = m->n_rows;
    int64_t *ip = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t *rows = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t *cnt_sort = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t *cnt_mark = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t *off = (int64_t *)malloc((size_t)(n + 1) * sizeof(int64_t));
    for (int64_t i = 0; i < n; ++i) rows[i] = i;
    oracle_row_products(&A, &A, ip);
    CHECK(oracle_count_rows(&A, &A, rows, n, cnt_sort) == 0, "%s: count_rows", name);
    CHECK(oracle_row_counts(&A, &A, 0, n, cnt_mark) == 0, "%s: row_counts", name);
    off[0] = 0;
    for (int64_t i = 0; i < n; ++i) {
        CHECK(cnt_sort[i] == cnt_mark[i], "%s: row %lld counts %lld vs %lld", name, (long long)i,
              (long long)cnt_sort[i], (long long)cnt_mark[i]);
        CHECK(cnt_sort[i] <= ip[i], "%s: row %lld has more entries than products", name, (long long)i);
        off[i + 1] = off[i] + cnt_sort[i];
    }
    const int64_t nnz = off[n];
    int64_t *c = (int64_t *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(int64_t));
    double *v = (double *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(double));
    double *b = (double *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(double));
    int64_t *t = (int64_t *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(int64_t));
    CHECK(oracle_fill_rows(&A, &A, rows, n, off, c, v, b, t) == 0, "%s: fill_rows", name);
    for (int64_t i = 0; i < n; ++i) {
        int64_t terms = 0;
        for (int64_t p = off[i]; p < off[i + 1]; ++p) {
            CHECK(p == off[i] || c[p] > c[p - 1], "%s: row %lld columns not increasing", name, (long long)i);
            CHECK(c[p] >= 0 && c[p] < m->n_cols, "%s: column out of range", name);
            CHECK(b[p] >= 0.0 && t[p] >= 1, "%s: bound or term count", name);
            terms += t[p];
        }
        CHECK(terms == ip[i], "%s: row %lld terms %lld vs products %lld", name, (long long)i, (long long)terms,
              (long long)ip[i]);
    }
    /* a sub-range of rows through the marking counter */
    if (n > 2) {
        int64_t *part = (int64_t *)malloc((size_t)n * sizeof(int64_t));
        CHECK(oracle_row_counts(&A, &A, 1, n - 1, part) == 0, "%s: row_counts range", name);
        for (int64_t i = 1; i < n - 1; ++i) CHECK(part[i - 1] == cnt_mark[i], "%s: range count", name);
        free(part);
    }
    printf("%s: n=%lld nnz(A)=%lld nnz(C)=%lld ok\n", name, (long long)n, (long long)m->nnz, (long long)nnz);
    free(c);
    free(v);
    free(b);
    free(t);
    free(off);
    free(cnt_mark);
    free(cnt_sort);
    free(rows);
    free(ip);
    free(col64);
    gm_gen_free(m);
}

int main(void) {
    run("rmat10", gm_gen_rmat(10, 8, 0.57, 0.19, 0.19, 1, 0));
    run("rmat9_int", gm_gen_rmat(9, 16, 0.60, 0.17, 0.17, 2, 2));
    run("banded", gm_gen_banded(3000, 13, 3, 1));
    run("banded_tiny", gm_gen_banded(5, 13, 4, 3));
    run("er", gm_gen_erdos_renyi(2000, 2000, 16, 5, 1));
    run("uniform", gm_gen_uniform(300, 300, 0.02, 6, 1));
    run("empty", gm_gen_uniform(7, 7, 0.0, 7, 1));
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    return 0;
}
