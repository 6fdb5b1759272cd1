// Host-side driver for a sanitizer build of the library's host code (its
// planner, path routing and argument validation): every call below stays on
// the host (no device is needed or touched). Exit status 0 when all checks
// pass; AddressSanitizer / UndefinedBehaviorSanitizer abort on an error.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <initializer_list>

#include "../../include/gmagnus.h"

static int failures = 0;
#define CHECK(cond)                                                  \
    do {                                                             \
        if (!(cond)) {                                               \
            std::fprintf(stderr, "check failed line %d: %s\n", __LINE__, #cond); \
            ++failures;                                              \
        }                                                            \
    } while (0)

int main() {
    gmagnus_options_t o;
    gmagnus_options_init(&o);
    CHECK(o.struct_size == sizeof(o));
    gmagnus_params_t p;
    const int64_t lds[] = {1024, 65536, 131072, 163840, 233472};
    const int64_t cms[] = {1, 7, 4096, 8193, 65536, (1 << 22) + 3, (int64_t)1 << 30, ((int64_t)1 << 31) - 1};
    for (int it = 0; it < 2; ++it)
        for (int vt = 0; vt < 2; ++vt)
            for (int64_t s : lds)
                for (int64_t cm : cms) {
                    const gmagnus_status_t st = gmagnus_get_params_typed(cm, s, it, vt, nullptr, &p);
                    // tiny local memories need more multisplit levels than the library runs
                    CHECK(st == GMAGNUS_SUCCESS || (st == GMAGNUS_ERROR_UNSUPPORTED && s < 65536));
                    if (st != GMAGNUS_SUCCESS) continue;
                    CHECK(p.tau >= 1 && p.dense_width >= 32 && p.chunks_required >= 1);
                    int64_t prod = 1;
                    for (int l = 0; l < p.n_levels; ++l) prod *= p.v_chunks[l];
                    CHECK(p.n_levels == 0 ? p.chunks_required == 1 : prod == p.chunks_required);
                    for (int32_t flags : {0, 8, 16, 32, 64})
                        CHECK(gmagnus_expansion_path(&p, 10, 1000, 100, flags) >= GMAGNUS_PATH_PAPER);
                }
    // overrides and their validation
    o.tau = 200;
    o.dense_width_log2 = 6;
    o.chunks_max_log2 = 2;
    CHECK(gmagnus_get_params(4096, 163840, &o, &p) == GMAGNUS_SUCCESS && p.n_levels == 3);
    o.dense_width_log2 = 14;
    CHECK(gmagnus_get_params(4096, 163840, &o, &p) == GMAGNUS_ERROR_INVALID_VALUE);
    CHECK(std::strlen(gmagnus_last_error()) > 0);
    CHECK(gmagnus_get_params(0, 163840, nullptr, &p) == GMAGNUS_ERROR_INVALID_VALUE);
    CHECK(gmagnus_get_params_typed(4096, 163840, 7, 0, nullptr, &p) == GMAGNUS_ERROR_INVALID_VALUE);
    CHECK(gmagnus_get_params_typed(((int64_t)1 << 35) + 1, 163840, 1, 0, nullptr, &p) == GMAGNUS_ERROR_INVALID_VALUE);
    CHECK(gmagnus_expansion_path(nullptr, 1, 1, 1, 0) == GMAGNUS_PATH_NONE);
    // plan argument validation (fails before any device call)
    gmagnus_plan_t plan = nullptr;
    gmagnus_csr_t a{4, 5, 0, (const int64_t *)0x1000, nullptr, nullptr};
    gmagnus_csr_t b{6, 3, 0, (const int64_t *)0x1000, nullptr, nullptr};
    CHECK(gmagnus_plan(&plan, &a, &b, nullptr, nullptr) == GMAGNUS_ERROR_INVALID_VALUE && !plan);
    CHECK(gmagnus_plan(nullptr, &a, &b, nullptr, nullptr) == GMAGNUS_ERROR_INVALID_VALUE);
    gmagnus_matrix_t ta{4, 5, 0, (const int64_t *)0x1000, nullptr, nullptr, 0, 0};
    gmagnus_matrix_t tb{5, 3, 0, (const int64_t *)0x1000, nullptr, nullptr, 1, 0};
    CHECK(gmagnus_plan_typed(&plan, &ta, &tb, nullptr, nullptr) == GMAGNUS_ERROR_INVALID_VALUE && !plan);
    int64_t nnz = 0;
    CHECK(gmagnus_spgemm_symbolic(nullptr, nullptr, &nnz) == GMAGNUS_ERROR_INVALID_VALUE);
    CHECK(gmagnus_spgemm_numeric_typed(nullptr, nullptr, nullptr, nullptr) == GMAGNUS_ERROR_INVALID_VALUE);
    gmagnus_plan_destroy(nullptr);
    for (int s = 0; s <= 7; ++s) CHECK(gmagnus_status_string((gmagnus_status_t)s) != nullptr);
    double ms = 0;
    CHECK(gmagnus_bandwidth_probe(9, nullptr, nullptr, 16, 0, 1, nullptr, &ms) == GMAGNUS_ERROR_INVALID_VALUE);
    if (failures) {
        std::fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    std::printf("library host checks ok\n");
    return 0;
}
