/* Drives every CPU-oracle entry point over special values, ragged and empty
 * sizes and random inputs, for a build under AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_oracle_sanitize.py).  Each buffer
 * is allocated at its exact size, so that a read or write past its end is
 * reported.  Prints "ok" and exits 0 when every call returned and the few
 * checked values hold. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "kbo.h"

#define CHECK(c)                                                     \
    do {                                                             \
        if (!(c)) {                                                  \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                                \
        }                                                            \
    } while (0)

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (uint32_t)(rng >> 16);
}

static void* exact_alloc(size_t bytes) { return malloc(bytes ? bytes : 1); }

/* Random storage of n elements of dtype, with special values mixed in. */
static void* random_tensor(int dtype, uint64_t n) {
    const size_t b = dtype == KBO_F32 ? 4 : 2;
    unsigned char* p = exact_alloc(n * b);
    static const uint32_t sp32[] = {0x00000000u, 0x80000000u, 0x7F800000u, 0xFF800000u, 0x7FC00000u,
                                    0x00000001u, 0x807FFFFFu, 0x7F7FFFFFu};
    static const uint16_t sp16[] = {0x0000u, 0x8000u, 0x7C00u, 0xFC00u, 0x7E00u, 0x0001u, 0x7BFFu, 0x7F80u};
    for (uint64_t i = 0; i < n; ++i) {
        const uint32_t u = next_u32();
        if (dtype == KBO_F32) {
            uint32_t v = (u % 16 == 0) ? sp32[u % 8] : (next_u32() & 0x3FFFFFFFu) | 0x3C000000u;
            memcpy(p + 4 * i, &v, 4);
        } else {
            uint16_t v = (u % 16 == 0) ? sp16[u % 8] : (uint16_t)((next_u32() & 0x3FFFu) | 0x3000u);
            memcpy(p + 2 * i, &v, 2);
        }
    }
    return p;
}

static int screen_cases(void) {
    const int dtypes[3] = {KBO_F32, KBO_F16, KBO_BF16};
    const uint64_t sizes[] = {0, 1, 7, 511, 512, 513, 4097};
    for (int d = 0; d < 3; ++d) {
        for (size_t s = 0; s < sizeof(sizes) / sizeof(sizes[0]); ++s) {
            const uint64_t n = sizes[s];
            void* r = random_tensor(dtypes[d], n);
            void* c = random_tensor(dtypes[d], n);
            for (uint32_t flags = 0; flags < 2; ++flags) {
                kbo_stats st;
                CHECK(kbo_screen(dtypes[d], r, c, n, 1e-3f, 1e-3f, flags, &st) == 0);
                CHECK(st.numel == n && st.mismatches <= n);
                kbo_stats self;
                CHECK(kbo_screen(dtypes[d], r, r, n, 0.f, 0.f, flags, &self) == 0);
                CHECK(self.bitwise_equal == 1);
                /* chunk and merge */
                kbo_partial a, b;
                kbo_partial_init(&a);
                kbo_partial_init(&b);
                CHECK(kbo_screen_range(dtypes[d], r, c, 0, n / 2, 1e-3f, 1e-3f, flags, &a) == 0);
                CHECK(kbo_screen_range(dtypes[d], r, c, n / 2, n, 1e-3f, 1e-3f, flags, &b) == 0);
                kbo_merge(&a, &b);
                kbo_stats m;
                kbo_finalize(&a, &m);
                CHECK(m.mismatches == st.mismatches && m.nan_count == st.nan_count);
                kbo_locate_t loc;
                CHECK(kbo_locate(dtypes[d], r, c, n, 1e-3f, 1e-3f, flags, st.max_abs_err, st.max_rel_err,
                                 &loc) == 0);
                CHECK(loc.first_mismatch < (int64_t)n);
            }
            if (dtypes[d] != KBO_F32) {
                uint8_t* out = exact_alloc(n);
                kbo_match16_n(dtypes[d], c, r, 1e-2f, 1e-2f, 0, out, n);
                free(out);
            }
            free(r);
            free(c);
        }
    }
    return 0;
}

static int map_cases(void) {
    const uint64_t n = 1031;
    float* f = exact_alloc(n * 4);
    uint16_t* h = exact_alloc(n * 2);
    uint32_t* x = exact_alloc(n * 4);
    for (uint64_t i = 0; i < n; ++i) {
        x[i] = next_u32();
        memcpy(&f[i], &x[i], 4);
    }
    kbo_f32_to_f16_n(f, h, n);
    kbo_f16_to_f32_n(h, f, n);
    kbo_f32_to_bf16_n(f, h, n);
    kbo_bf16_to_f32_n(h, f, n);
    kbo_uniform_n(x, -1.f, 1.f, f, n);
    for (uint64_t i = 0; i < n; ++i) CHECK(f[i] >= -1.f && f[i] < 1.f);
    const int dts[4] = {KBO_F32, KBO_F16, KBO_BF16, KBO_U32};
    for (int d = 0; d < 4; ++d) {
        for (int dist = 0; dist < 3; ++dist) {
            const size_t b = dts[d] == KBO_F16 || dts[d] == KBO_BF16 ? 2 : 4;
            void* dst = exact_alloc(n * b);
            const int rc = kbo_gen(dst, dts[d], n, dist, 0.f, 1.f, 7, 3, 1, 5);
            CHECK(rc == 0 || rc == -1);
            free(dst);
        }
    }
    uint32_t in[4] = {1, 2, 3, 4}, key[2] = {5, 6}, out[4];
    kbo_philox4x32_10(in, key, out);
    CHECK(kbo_normal01(0xFFFFFFFFu, 123u, 0) == 0.f);
    free(f);
    free(h);
    free(x);
    return 0;
}

static int rung_cases(void) {
    const int C = 9, S = 3, N = 17;
    double* t = exact_alloc(sizeof(double) * C * S * N);
    for (int i = 0; i < C * S * N; ++i) t[i] = 10.0 + (next_u32() % 1000) / 10.0;
    kbo_row_t* rows = exact_alloc(sizeof(kbo_row_t) * C * S);
    kbo_score_t* sc = exact_alloc(sizeof(kbo_score_t) * C);
    CHECK(kbo_rung_stats(t, C, S, N, 0, 2, 60.0, 0.02, 0.01, rows, sc) == 0);
    CHECK(kbo_rung_stats(t, C, S, N, -1, 0, 0.0, 0.02, 0.01, rows, sc) == 0);
    CHECK(kbo_rung_stats(t, 0, S, N, -1, 0, 0.0, 0.02, 0.01, rows, sc) == -1 ||
          kbo_rung_stats(t, 0, S, N, -1, 0, 0.0, 0.02, 0.01, rows, sc) == 0);
    double* score = exact_alloc(sizeof(double) * C);
    int32_t* valid = exact_alloc(sizeof(int32_t) * C);
    int32_t *rank = exact_alloc(sizeof(int32_t) * C), *order = exact_alloc(sizeof(int32_t) * C),
            *prom = exact_alloc(sizeof(int32_t) * C);
    for (int i = 0; i < C; ++i) {
        score[i] = sc[i].score;
        valid[i] = (i % 4) != 3;
    }
    CHECK(kbo_rung_promote(score, valid, C, 0, 2, 5, rank, order, prom) == 0);
    CHECK(kbo_rung_promote(score, valid, C, -1, 1, 1, rank, order, prom) == 0);
    CHECK(kbo_rung_promote(score, valid, C, 0, 3, 2, rank, order, prom) == -1);
    int32_t entering[3] = {21, 7, 3}, failed[3] = {5, 2, 0}, promoted[3] = {7, 3, 3};
    double fp[3], pp[3];
    CHECK(kbo_rung_survival(entering, failed, promoted, 3, 21, fp, pp) == 0);
    double q[1] = {4.0};
    CHECK(kbo_quantile_sorted(q, 1, 0.99) == 4.0);
    free(t);
    free(rows);
    free(sc);
    free(score);
    free(valid);
    free(rank);
    free(order);
    free(prom);
    return 0;
}

/* The derived inputs: Student-t, softmax rows, index draws, planted changes
 * on every dtype (in place and not), scatters with out-of-range indices. */
static int derived_cases(void) {
    uint32_t w[4] = {0u, 0u, 0xFFFFFFFFu, 0u}; /* a zero chi-square: z0 / 0 */
    (void)kbo_student_t3(w);
    for (uint64_t n = 0; n < 40; n += 13) {
        float* t = exact_alloc(n * 4);
        CHECK(kbo_gen(t, KBO_F32, n, KBO_DIST_STUDENT_T3, 0.0f, 1.0f, 1, 2, 3, 1ull << 40) == 0);
        free(t);
    }
    for (uint64_t cols = 1; cols < 70; cols += 17) {
        float* sm = exact_alloc(3 * cols * 4);
        CHECK(kbo_gen_softmax_rows(sm, 5, 3, cols, 2.0f, 0, 3, 0) == 0);
        free(sm);
    }
    CHECK(kbo_gen_softmax_rows(NULL, 0, 1, 0, 2.0f, 0, 3, 0) == -1);
    uint64_t* idx = exact_alloc(7 * 8);
    CHECK(kbo_gen_indices(idx, 7, 7, 0, 9, 1) == 0);
    CHECK(kbo_gen_indices(idx, 7, 6, 0, 9, 1) == -1);
    for (int dtype = 0; dtype < 3; ++dtype) {
        const uint64_t n = 1029;
        void* src = random_tensor(dtype, n);
        void* dst = exact_alloc(n * (dtype == KBO_F32 ? 4 : 2));
        for (int op = 1; op <= 7; ++op) {
            const int want = (op >= 6 && dtype != KBO_F32) ? -1 : 0;
            CHECK(kbo_perturb(dst, src, dtype, n, op, -0.5f, 0.5f, 0.5f, 0, 4, op, 3) == want);
            CHECK(kbo_perturb(src, src, dtype, n, op, 0.25f, 0.5f, 0.75f, 0, 4, op, 0) == want);
        }
        CHECK(kbo_perturb(dst, src, dtype, n, 8, 0.0f, 0.0f, 0.0f, 0, 0, 0, 0) == -1);
        const uint64_t sidx[3] = {0, n - 1, n};
        CHECK(kbo_scatter(dst, src, dtype, n, sidx, 3, KBO_SCATTER_NAN) == 0);
        CHECK(kbo_scatter(dst, src, dtype, n, sidx, 3, KBO_SCATTER_INF_SIGN_OF_REF) == 0);
        CHECK(kbo_scatter(dst, src, dtype, n, sidx, 3, 3) == -1);
        free(src);
        free(dst);
    }
    free(idx);
    return 0;
}

int main(void) {
    if (screen_cases() || map_cases() || rung_cases() || derived_cases()) return 1;
    printf("ok\n");
    return 0;
}
