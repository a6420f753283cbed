/*
 * kbo_derived.c -- plain CPU oracle for the derived seeded inputs.
 *
 * TEST INFRASTRUCTURE ONLY, like kbo.c: loaded by the test suite, the smoke
 * check and the benchmark's CPU-baseline leg, never by the product path.
 *
 * The screening check of the Verifier runs a candidate on seeded test inputs
 * and compares its output with the reference output (Sections 3.1 and 3.4).
 * These functions build the synthetic outputs the screen is measured on,
 * from the same counter-based stream as kbo_gen (Philox4x32-10, key = seed,
 * counter = (lo32(b), hi32(b), sub, stream_id)):
 *   - Student-t values with 3 degrees of freedom (a heavy-tailed output);
 *   - softmax rows of normal logits (rows that sum to one);
 *   - seeded sets of distinct indices (where NaNs or infinities are planted);
 *   - the planted changes that turn a reference into a candidate (uniform
 *     and normal noise, seeded masks, last-bit flips, signed zeros,
 *     subnormal flushes, special values).
 * Each function applies its definition element by element, in the order the
 * definition states, in binary64 where it says so and in binary32 otherwise
 * (built with -ffp-contract=off: no multiply-add is fused unless written as
 * fmaf).
 *
 * Pins (tests/test_oracle_derived.py, no GPU): the Student-t by closed-form
 * word patterns and by its distribution (the t(3) CDF in closed form, the
 * two-sided 5% point 3.182446); the softmax by scipy's softmax in binary64,
 * shift invariance and the row-sum bound; the index draws by brute force on
 * tiny n and by the word stream itself when n = 2^32; every planted change
 * by the cases that reduce it to kbo_gen's pinned uniform and normal maps,
 * by exact rational arithmetic, and by the frequencies of its masks.
 */
#include "kbo.h"

#include <math.h>
#include <string.h>

#if defined(__x86_64__)
#include <xmmintrin.h>
#endif

/* Gradual underflow and round-to-nearest-even for the duration of a call
 * (subnormal values are part of these definitions). */
static unsigned int fpenv_enter(void) {
#if defined(__x86_64__)
    unsigned int saved = _mm_getcsr();
    _mm_setcsr(saved & ~((1u << 15) | (1u << 6) | (3u << 13)));
    return saved;
#else
    return 0;
#endif
}

static void fpenv_leave(unsigned int saved) {
#if defined(__x86_64__)
    _mm_setcsr(saved);
#else
    (void)saved;
#endif
}

static uint32_t f32_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float bits_f32(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* ---------------------------------------------------------------------------
 * Student-t, 3 degrees of freedom.
 * ------------------------------------------------------------------------- */
double kbo_student_t3_64(const uint32_t w[4]) {
    double z0, z1, z2, z3;
    kbo_box_muller64(w[0], w[1], &z0, &z1);
    kbo_box_muller64(w[2], w[3], &z2, &z3);
    double chi2 = (z1 * z1 + z2 * z2) + z3 * z3; /* chi-square, 3 degrees of freedom */
    return z0 / sqrt(chi2 / 3.0);
}

float kbo_student_t3(const uint32_t w[4]) { return (float)kbo_student_t3_64(w); }

/* ---------------------------------------------------------------------------
 * Softmax rows.
 * ------------------------------------------------------------------------- */
void kbo_softmax_row(const float* x, uint64_t n, float* out) {
    const unsigned int env = fpenv_enter();
    float m = x[0];
    for (uint64_t j = 1; j < n; ++j)
        if (x[j] > m) m = x[j];
    double s = 0.0;
    for (uint64_t j = 0; j < n; ++j) s += exp((double)x[j] - (double)m);
    for (uint64_t j = 0; j < n; ++j) out[j] = (float)(exp((double)x[j] - (double)m) / s);
    fpenv_leave(env);
}

int kbo_gen_softmax_rows(float* dst, uint64_t row0, uint64_t rows, uint64_t cols, float sigma,
                         uint64_t seed, uint32_t stream_id, uint32_t sub) {
    if (cols == 0) return -1;
    for (uint64_t i = 0; i < rows; ++i) {
        float* row = dst + i * cols;
        /* the logits, generated in place, then replaced by the softmax */
        kbo_gen(row, KBO_F32, cols, KBO_DIST_NORMAL, 0.0f, sigma, seed, stream_id, sub, (row0 + i) * cols);
        kbo_softmax_row(row, cols, row);
    }
    return 0;
}

/* ---------------------------------------------------------------------------
 * Distinct index draws.
 * ------------------------------------------------------------------------- */
int kbo_gen_indices(uint64_t* out, uint32_t m, uint64_t n, uint64_t seed, uint32_t stream_id,
                    uint32_t sub) {
    if (n == 0 || (uint64_t)m > n) return -1;
    uint32_t have = 0;
    for (uint64_t j = 0; have < m; ++j) {
        uint32_t w[4];
        kbo_stream_block(seed, stream_id, sub, j, w);
        uint64_t x = (((uint64_t)w[1] << 32) | w[0]) % n;
        int seen = 0;
        for (uint32_t i = 0; i < have; ++i)
            if (out[i] == x) seen = 1;
        if (!seen) out[have++] = x;
    }
    return 0;
}

/* ---------------------------------------------------------------------------
 * Planted changes.
 * ------------------------------------------------------------------------- */
static float widen(int dtype, const void* src, uint64_t j) {
    if (dtype == KBO_F32) return ((const float*)src)[j];
    uint16_t h = ((const uint16_t*)src)[j];
    return dtype == KBO_F16 ? kbo_f16_to_f32(h) : kbo_bf16_to_f32(h);
}

/* An arithmetic result, rounded to the dtype; a NaN result is stored as the
 * dtype's positive quiet NaN (IEEE 754 leaves the sign and payload of a NaN
 * an operation creates to the platform). */
static void store(int dtype, void* dst, uint64_t j, float v) {
    if (isnan(v)) {
        if (dtype == KBO_F32) ((uint32_t*)dst)[j] = 0x7FC00000u;
        else ((uint16_t*)dst)[j] = dtype == KBO_F16 ? 0x7E00u : 0x7FC0u;
        return;
    }
    if (dtype == KBO_F32) ((float*)dst)[j] = v;
    else if (dtype == KBO_F16) ((uint16_t*)dst)[j] = kbo_f32_to_f16(v);
    else ((uint16_t*)dst)[j] = kbo_f32_to_bf16(v);
}

static void copy_elem(int dtype, void* dst, const void* src, uint64_t j) {
    if (dtype == KBO_F32) ((uint32_t*)dst)[j] = ((const uint32_t*)src)[j];
    else ((uint16_t*)dst)[j] = ((const uint16_t*)src)[j];
}

int kbo_perturb(void* dst, const void* src, int dtype, uint64_t n, int op, float a, float b, float p,
                uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset) {
    if (dtype != KBO_F32 && dtype != KBO_F16 && dtype != KBO_BF16) return -1;
    if (op < KBO_PERTURB_ADD_UNIFORM || op > KBO_PERTURB_ZERO_SUBNORMAL_REL) return -1;
    if (op >= KBO_PERTURB_SPECIALS && dtype != KBO_F32) return -1;
    const unsigned int env = fpenv_enter();
    for (uint64_t j = 0; j < n; ++j) {
        const uint64_t g = offset + j;
        uint32_t w[4];
        if (op <= KBO_PERTURB_FLIP_LSB_WHERE) {
            /* one word per element: word g mod 4 of block g / 4 */
            kbo_stream_block(seed, stream_id, sub, g >> 2, w);
            const uint32_t word = w[g & 3u];
            const float x = widen(dtype, src, j);
            if (op == KBO_PERTURB_ADD_UNIFORM) {
                store(dtype, dst, j, x + kbo_uniform(word, a, b));
            } else if (op == KBO_PERTURB_REL_UNIFORM) {
                store(dtype, dst, j, fmaf(x, kbo_uniform(word, a, b), x));
            } else if (op == KBO_PERTURB_ADD_NORMAL) {
                const unsigned k = (unsigned)(g & 3u), pair = k >> 1;
                const float z = kbo_normal01(w[2 * pair], w[2 * pair + 1], (int)(k & 1u));
                store(dtype, dst, j, x + fmaf(z, a, 0.0f));
            } else if (op == KBO_PERTURB_SCALE_WHERE) {
                if (kbo_u01(word) < p) store(dtype, dst, j, x * a);
                else copy_elem(dtype, dst, src, j);
            } else { /* FLIP_LSB_WHERE */
                copy_elem(dtype, dst, src, j);
                if (kbo_u01(word) < p) {
                    if (dtype == KBO_F32) ((uint32_t*)dst)[j] ^= 1u;
                    else ((uint16_t*)dst)[j] ^= 1u;
                }
            }
            continue;
        }
        /* one whole block per element, binary32 only */
        kbo_stream_block(seed, stream_id, sub, g, w);
        const uint32_t bits = ((const uint32_t*)src)[j];
        const float v = kbo_u01(w[0]);
        uint32_t out = bits;
        if (op == KBO_PERTURB_SPECIALS) {
            const uint32_t sign = w[1] & 0x80000000u;
            if (v < a) out = sign | (w[2] & 0x7FFFFFu) | 1u; /* a subnormal */
            else if (v < b) out = sign;                      /* a signed zero */
            else if (v < p) out = sign | 0x7F800000u;        /* an infinity */
        } else { /* ZERO_SUBNORMAL_REL */
            const uint32_t mag = bits & 0x7FFFFFFFu;
            if (v < p) {
                if (mag == 0u) out = bits ^ 0x80000000u;                    /* zero: flip its sign */
                else if (mag < 0x00800000u) out = bits & 0x80000000u;       /* subnormal: flush */
                else if (mag < 0x7F800000u) {                               /* finite normal */
                    const float x = bits_f32(bits);
                    out = f32_bits(fmaf(x, kbo_uniform(w[1], a, b), x));
                }
            }
        }
        ((uint32_t*)dst)[j] = out;
    }
    fpenv_leave(env);
    return 0;
}

int kbo_scatter(void* dst, const void* ref, int dtype, uint64_t n, const uint64_t* idx, uint32_t m,
                int mode) {
    if (dtype != KBO_F32 && dtype != KBO_F16 && dtype != KBO_BF16) return -1;
    if (mode != KBO_SCATTER_NAN && mode != KBO_SCATTER_INF_SIGN_OF_REF) return -1;
    for (uint32_t i = 0; i < m; ++i) {
        const uint64_t k = idx[i];
        if (k >= n) continue;
        if (dtype == KBO_F32) {
            const uint32_t sign = ((const uint32_t*)ref)[k] & 0x80000000u;
            ((uint32_t*)dst)[k] = mode == KBO_SCATTER_NAN ? 0x7FC00000u : (sign | 0x7F800000u);
        } else {
            const uint16_t sign = (uint16_t)(((const uint16_t*)ref)[k] & 0x8000u);
            const uint16_t nan = dtype == KBO_F16 ? 0x7E00u : 0x7FC0u;
            const uint16_t inf = dtype == KBO_F16 ? 0x7C00u : 0x7F80u;
            ((uint16_t*)dst)[k] = mode == KBO_SCATTER_NAN ? nan : (uint16_t)(sign | inf);
        }
    }
    return 0;
}
