/*
 * CPU ORACLE for the numeric SpGEMM C = A*B on CSR inputs.
 *
 * Test infrastructure only: the test suite, the smoke check and the CPU
 * baseline leg of the benchmark call this. The GPU library never links or
 * calls it, and it shares no code with the GPU library.
 *
 * What it computes is the plain definition the paper starts from:
 *   C[i,:] = sum_j A[i,j] * B[j,:]                (Section II-B, Eq. gustav)
 * computed row by row as in Gustavson's method (Algorithm 1): every
 * intermediate product A[i,j]*B[j,k] of row i is formed, the products are
 * stably sorted by column, and each run of equal columns is reduced. The
 * sorted, unique columns are the "SortAndWrite" output of Algorithm 1.
 * The symbolic phase (Section II-B) is the run count per row; the numeric
 * phase fills columns and values at the given row offsets.
 *
 * Choices where the paper is silent:
 *   - a column appears in C[i,:] iff some product lands there, even if the
 *     sum is exactly zero (structural entries are kept);
 *   - each run is reduced with Neumaier's compensated summation, so the
 *     oracle's own rounding error is far below the comparison tolerance;
 *   - bound[e] = sum of |A[i,j]*B[j,k]| over the run, the scale of the
 *     per-entry tolerance, and terms[e] = the run's length (the number of
 *     products summed into the entry);
 *   - column indices are 64-bit (32-bit inputs are widened by the caller) and
 *     values fp64: for fp32 inputs, widened exactly, every product is exact
 *     in fp64 (24 + 24 significant bits) and the compensated sum is the
 *     exact result to about one fp64 rounding.
 *
 * Rows are processed in parallel (OpenMP, dynamic schedule); each row is
 * computed by one thread in a fixed order, so results do not depend on the
 * thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <omp.h>

typedef struct {
    int64_t n_rows, n_cols;
    const int64_t *row_ptr;
    const int64_t *col;
    const double *val;
} oracle_csr;

/* Number of intermediate products of row i: sum over A[i,:] of nnz(B[j,:]). */
static int64_t row_products(const oracle_csr *A, const oracle_csr *B, int64_t i) {
    int64_t n = 0;
    for (int64_t p = A->row_ptr[i]; p < A->row_ptr[i + 1]; ++p) {
        int64_t j = A->col[p];
        n += B->row_ptr[j + 1] - B->row_ptr[j];
    }
    return n;
}

void oracle_row_products(const oracle_csr *A, const oracle_csr *B, int64_t *ip) {
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t i = 0; i < A->n_rows; ++i) ip[i] = row_products(A, B, i);
}

/* A product's sort key: its column, then its position q in (j, k) order,
 * so sorting by (col, q) is stable. */
typedef struct {
    int64_t col;
    int64_t q;
} oracle_key;

static int cmp_key(const void *a, const void *b) {
    const oracle_key *x = (const oracle_key *)a, *y = (const oracle_key *)b;
    if (x->col != y->col) return (x->col > y->col) - (x->col < y->col);
    return (x->q > y->q) - (x->q < y->q);
}

/* Forms the products of row i in (j, k) order and sorts them by column
 * (stable); prod[q] is the product at position q. Returns the product count,
 * or -1 on allocation failure. */
static int64_t expand_sorted(const oracle_csr *A, const oracle_csr *B, int64_t i, oracle_key **keys_out,
                             double **prod_out) {
    int64_t n = row_products(A, B, i);
    *keys_out = NULL;
    *prod_out = NULL;
    oracle_key *keys = (oracle_key *)malloc((size_t)(n > 0 ? n : 1) * sizeof(oracle_key));
    double *prod = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    if (!keys || !prod) {
        free(keys);
        free(prod);
        return -1;
    }
    int64_t q = 0;
    for (int64_t p = A->row_ptr[i]; p < A->row_ptr[i + 1]; ++p) {
        int64_t j = A->col[p];
        double a = A->val[p];
        for (int64_t r = B->row_ptr[j]; r < B->row_ptr[j + 1]; ++r) {
            keys[q].col = B->col[r];
            keys[q].q = q;
            prod[q] = a * B->val[r];
            ++q;
        }
    }
    qsort(keys, (size_t)n, sizeof(oracle_key), cmp_key);
    *keys_out = keys;
    *prod_out = prod;
    return n;
}

/* Symbolic: number of distinct columns of C[rows[t], :] into counts[t].
 * Returns 0, or -1 if some row could not be processed. */
int oracle_count_rows(const oracle_csr *A, const oracle_csr *B, const int64_t *rows, int64_t n_list,
                      int64_t *counts) {
    int failed = 0;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n_list; ++t) {
        oracle_key *keys;
        double *prod;
        int64_t n = expand_sorted(A, B, rows[t], &keys, &prod);
        if (n < 0) {
            failed = 1;
            counts[t] = -1;
            continue;
        }
        int64_t runs = 0;
        for (int64_t q = 0; q < n; ++q)
            if (q == 0 || keys[q].col != keys[q - 1].col) ++runs;
        counts[t] = runs;
        free(keys);
        free(prod);
    }
    return failed ? -1 : 0;
}

/* Numeric: row rows[t] is written at positions offsets[t] .. of col, val,
 * bound and terms (terms may be NULL). */
int oracle_fill_rows(const oracle_csr *A, const oracle_csr *B, const int64_t *rows, int64_t n_list,
                     const int64_t *offsets, int64_t *col, double *val, double *bound, int64_t *terms) {
    int failed = 0;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n_list; ++t) {
        oracle_key *keys;
        double *prod;
        int64_t n = expand_sorted(A, B, rows[t], &keys, &prod);
        if (n < 0) {
            failed = 1;
            continue;
        }
        int64_t out = offsets[t] - 1, run = 0;
        double s = 0.0, comp = 0.0, mag = 0.0;
        for (int64_t q = 0; q < n; ++q) {
            const int64_t c = keys[q].col;
            double x = prod[keys[q].q];
            if (q == 0 || c != keys[q - 1].col) {
                if (q > 0) {
                    val[out] = s + comp;
                    bound[out] = mag;
                    if (terms) terms[out] = run;
                }
                ++out;
                col[out] = c;
                s = 0.0;
                comp = 0.0;
                mag = 0.0;
                run = 0;
            }
            /* Neumaier: carry the low-order part lost by s + x. */
            double t2 = s + x;
            if (fabs(s) >= fabs(x))
                comp += (s - t2) + x;
            else
                comp += (x - t2) + s;
            s = t2;
            mag += fabs(x);
            ++run;
        }
        if (n > 0) {
            val[out] = s + comp;
            bound[out] = mag;
            if (terms) terms[out] = run;
        }
        free(keys);
        free(prod);
    }
    return failed ? -1 : 0;
}

/* Symbolic by marking, for whole matrices: counts[i - row_begin] = number of
 * distinct columns of C[i, :] for i in [row_begin, row_end). Each thread
 * keeps one stamp per column of C, the last row that reached that column; a
 * product adds one to its row's count when it is the first to reach its
 * column for that row. This is the distinct-column count of the symbolic
 * phase (Section II-B) without forming or sorting the products, so it
 * finishes whole R-MAT products on a few cores. Returns 0, or -1 when the
 * stamp arrays cannot be allocated. */
int oracle_row_counts(const oracle_csr *A, const oracle_csr *B, int64_t row_begin, int64_t row_end,
                      int64_t *counts) {
    int failed = 0;
    if (row_end - row_begin > ((int64_t)1 << 31) - 2 || B->n_cols > ((int64_t)1 << 31)) return -1;
#pragma omp parallel
    {
        int32_t *stamp = (int32_t *)malloc((size_t)(B->n_cols > 0 ? B->n_cols : 1) * sizeof(int32_t));
        if (!stamp) {
#pragma omp atomic write
            failed = 1;
        } else {
            for (int64_t c = 0; c < B->n_cols; ++c) stamp[c] = -1;
        }
#pragma omp barrier
        if (!failed) {
#pragma omp for schedule(dynamic, 64)
            for (int64_t i = row_begin; i < row_end; ++i) {
                const int32_t mark = (int32_t)(i - row_begin);
                int64_t n = 0;
                for (int64_t p = A->row_ptr[i]; p < A->row_ptr[i + 1]; ++p) {
                    const int64_t j = A->col[p];
                    for (int64_t r = B->row_ptr[j]; r < B->row_ptr[j + 1]; ++r) {
                        const int64_t c = B->col[r];
                        if (stamp[c] != mark) {
                            stamp[c] = mark;
                            ++n;
                        }
                    }
                }
                counts[i - row_begin] = n;
            }
        }
        free(stamp);
    }
    return failed ? -1 : 0;
}

int oracle_threads(void) { return omp_get_max_threads(); }
