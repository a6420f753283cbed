/*
 * kbo.c -- plain CPU oracle for the candidate-screening path.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  Slow on purpose:
 * one element at a time, in the order the definitions below are stated, so
 * that each function can be checked against its definition by eye.
 *
 * Floating point: binary32 arithmetic for the comparison (SSE on x86-64, no
 * x87), binary64 for the squared-error sums, round to nearest even, gradual
 * underflow.  Built with -ffp-contract=off so that no multiply-add is fused
 * unless written as fmaf().  The entry points that compute clear the
 * flush-to-zero and denormals-are-zero bits for their duration, so a host
 * process that set them cannot change the answers.
 *
 * Pins (tests run without a GPU): Philox against the published Random123
 * known-answer vectors and against rocRAND's engine run on the host; the
 * uniform map exhaustively against exact rational arithmetic on samples and
 * by structure over all 2^24 values; the normal map by closed-form points,
 * the Box-Muller radius/angle identities and distribution tests; the
 * conversions exhaustively against numpy and torch; the screen by hand-built
 * cases with known answers, invariants and brute force on tiny inputs.
 */
#include "kbo.h"

#include <math.h>
#include <string.h>

#if defined(__x86_64__)
#include <xmmintrin.h>
#endif

/* ---------------------------------------------------------------------------
 * Floating-point environment guard: gradual underflow is part of the
 * definitions below (subnormal differences and tolerances count).
 * ------------------------------------------------------------------------- */
typedef struct { unsigned int saved; } fpenv_guard;

static fpenv_guard fpenv_enter(void) {
    fpenv_guard g = {0};
#if defined(__x86_64__)
    g.saved = _mm_getcsr();
    /* bit 15 = flush to zero, bit 6 = denormals are zero; rounding bits 13-14
     * cleared = round to nearest even. */
    _mm_setcsr(g.saved & ~((1u << 15) | (1u << 6) | (3u << 13)));
#endif
    return g;
}

static void fpenv_leave(fpenv_guard g) {
#if defined(__x86_64__)
    _mm_setcsr(g.saved);
#else
    (void)g;
#endif
}

static uint32_t f32_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float bits_f32(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* ---------------------------------------------------------------------------
 * Philox4x32-10 (SC'11 paper, Section 4).
 * Round: (hi0, lo0) = M0 * x0 and (hi1, lo1) = M1 * x2 as 64-bit products;
 *        new state = (hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0).
 * Key schedule: (k0, k1) += (W0, W1) mod 2^32 after every round.
 * ------------------------------------------------------------------------- */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u /* golden ratio */
#define PHILOX_W1 0xBB67AE85u /* sqrt(3) - 1 */

void kbo_philox4x32_10(const uint32_t in[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t x0 = in[0], x1 = in[1], x2 = in[2], x3 = in[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

void kbo_stream_block(uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t b,
                      uint32_t out[4]) {
    uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), sub, stream_id};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    kbo_philox4x32_10(ctr, key, out);
}

/* ---------------------------------------------------------------------------
 * Word -> float maps.
 * ------------------------------------------------------------------------- */
float kbo_u01(uint32_t x) {
    /* the top 24 bits scaled by 2^-24: every value is exact in binary32 */
    return (float)(x >> 8) * 0x1p-24f;
}

float kbo_uniform(uint32_t x, float a, float b) {
    float width = b - a; /* binary32, one rounding */
    return fmaf(kbo_u01(x), width, a);
}

/* 2*pi rounded to the nearest binary64. */
#define KBO_TWO_PI 6.283185307179586476925286766559

void kbo_box_muller64(uint32_t xa, uint32_t xb, double* zc, double* zs) {
    double u1 = ((double)xa + 1.0) * 0x1p-32; /* (0, 1], exact */
    double u2 = (double)xb * 0x1p-32;         /* [0, 1), exact */
    double rho = sqrt(-2.0 * log(u1));
    double theta = KBO_TWO_PI * u2;
    *zc = rho * cos(theta);
    *zs = rho * sin(theta);
}

float kbo_normal01(uint32_t xa, uint32_t xb, int odd) {
    double zc, zs;
    kbo_box_muller64(xa, xb, &zc, &zs);
    return (float)(odd ? zs : zc);
}

/* ---------------------------------------------------------------------------
 * IEEE 754 binary32 <-> binary16 / bfloat16, round to nearest, ties to even.
 * ------------------------------------------------------------------------- */

/* m / 2^shift rounded to nearest, ties to even (shift >= 0). */
static uint64_t shift_rne(uint64_t m, int shift) {
    if (shift == 0) return m;
    if (shift >= 64) return 0; /* m < 2^63 here, so m / 2^shift < 1/2 */
    uint64_t q = m >> shift;
    uint64_t rem = m & ((1ull << shift) - 1);
    uint64_t half = 1ull << (shift - 1);
    if (rem > half || (rem == half && (q & 1))) q++;
    return q;
}

uint16_t kbo_f32_to_f16(float f) {
    uint32_t x = f32_bits(f);
    uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
    uint32_t expf_ = (x >> 23) & 0xffu;
    uint32_t man = x & 0x7fffffu;
    if (expf_ == 0xffu) return (uint16_t)(sign | (man ? 0x7e00u : 0x7c00u));
    if (expf_ == 0) return sign; /* |f| < 2^-126, far below half the least binary16 */
    /* |f| = m * 2^(e - 23) with m in [2^23, 2^24) */
    uint64_t m = (1u << 23) | man;
    int e = (int)expf_ - 127;
    uint64_t q;
    uint32_t mag;
    if (e >= -14) {
        /* binary16 normal range: 11 significant bits, ulp = 2^(e - 10) */
        q = shift_rne(m, 13);
        /* encoding ((e + 14) << 10) + q is continuous: q = 2^11 carries into
         * the exponent field */
        uint64_t enc = ((uint64_t)(e + 14) << 10) + q;
        mag = enc >= 0x7c00u ? 0x7c00u : (uint32_t)enc;
    } else {
        /* subnormal target, ulp = 2^-24: q = round(m * 2^(e - 23) / 2^-24) */
        q = shift_rne(m, -e - 1);
        mag = (uint32_t)q; /* q = 2^10 encodes the least normal */
    }
    return (uint16_t)(sign | mag);
}

uint16_t kbo_f32_to_bf16(float f) {
    uint32_t x = f32_bits(f);
    uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
    uint32_t mag = x & 0x7fffffffu;
    if (mag > 0x7f800000u) return (uint16_t)(sign | 0x7fc0u); /* NaN -> quiet NaN */
    /* bfloat16 keeps the binary32 exponent field; the binary32 magnitude
     * encoding is monotone with a uniform step inside each binade, so
     * dropping 16 bits with round-to-nearest-even rounds the value (a carry
     * reaches the next binade, or infinity from the largest finite). */
    return (uint16_t)(sign | (uint16_t)shift_rne(mag, 16));
}

float kbo_f16_to_f32(uint16_t h) {
    uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
    uint32_t e = (h >> 10) & 0x1fu;
    uint32_t man = h & 0x3ffu;
    if (e == 0x1fu) return bits_f32(sign | 0x7f800000u | (man << 13));
    float mag = e == 0 ? ldexpf((float)man, -24)                  /* subnormal */
                       : ldexpf((float)(0x400u | man), (int)e - 25); /* normal */
    return sign ? -mag : mag;
}

float kbo_bf16_to_f32(uint16_t h) { return bits_f32((uint32_t)h << 16); }

/* ---------------------------------------------------------------------------
 * Generator: element g = offset + j comes from word (g mod 4) of block g / 4;
 * a normal takes the word pair of its half-block, the cosine branch for even
 * g and the sine branch for odd g.  A Student-t value takes all of block g.
 * ------------------------------------------------------------------------- */
int kbo_gen(void* dst, int dtype, uint64_t n, int dist, float p0, float p1,
            uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset) {
    if (dist == KBO_DIST_U32 && dtype != KBO_U32) return -1;
    if (dist != KBO_DIST_U32 && dtype == KBO_U32) return -1;
    if (dist < 0 || dist > 3 || dtype < 0 || dtype > 3) return -1;
    fpenv_guard env = fpenv_enter();
    for (uint64_t j = 0; j < n; ++j) {
        uint64_t g = offset + j;
        uint32_t w[4];
        if (dist == KBO_DIST_STUDENT_T3) {
            /* one whole block per element */
            kbo_stream_block(seed, stream_id, sub, g, w);
            float v = fmaf(kbo_student_t3(w), p1, p0);
            if (dtype == KBO_F32) ((float*)dst)[j] = v;
            else if (dtype == KBO_F16) ((uint16_t*)dst)[j] = kbo_f32_to_f16(v);
            else ((uint16_t*)dst)[j] = kbo_f32_to_bf16(v);
            continue;
        }
        kbo_stream_block(seed, stream_id, sub, g >> 2, w);
        unsigned word = (unsigned)(g & 3u);
        if (dist == KBO_DIST_U32) {
            ((uint32_t*)dst)[j] = w[word];
            continue;
        }
        float v;
        if (dist == KBO_DIST_UNIFORM) {
            v = kbo_uniform(w[word], p0, p1);
        } else {
            unsigned pair = word >> 1;
            float z = kbo_normal01(w[2 * pair], w[2 * pair + 1], (int)(word & 1u));
            v = fmaf(z, p1, p0);
        }
        if (dtype == KBO_F32) ((float*)dst)[j] = v;
        else if (dtype == KBO_F16) ((uint16_t*)dst)[j] = kbo_f32_to_f16(v);
        else ((uint16_t*)dst)[j] = kbo_f32_to_bf16(v);
    }
    fpenv_leave(env);
    return 0;
}

/* ---------------------------------------------------------------------------
 * Screening: the numeric half of the policy-gated correctness check.
 * ------------------------------------------------------------------------- */
static void neumaier_add(double* sum, double* comp, double x) {
    double t = *sum + x;
    if (isinf(t)) { /* an infinite term (an overflowed difference): the sum is +inf */
        *sum = t;
        return;
    }
    if (fabs(*sum) >= fabs(x)) *comp += (*sum - t) + x;
    else *comp += (x - t) + *sum;
    *sum = t;
}

void kbo_partial_init(kbo_partial* p) {
    memset(p, 0, sizeof *p);
}

/* Storage bits and exact binary32 value of element i. */
static void load_elem(int dtype, const void* base, uint64_t i, uint32_t* bits, float* val) {
    if (dtype == KBO_F32) {
        uint32_t u = ((const uint32_t*)base)[i];
        *bits = u;
        *val = bits_f32(u);
    } else {
        uint16_t h = ((const uint16_t*)base)[i];
        *bits = h;
        *val = dtype == KBO_F16 ? kbo_f16_to_f32(h) : kbo_bf16_to_f32(h);
    }
}

int kbo_match(float c, float r, float atol, float rtol, uint32_t flags) {
    float d = fabsf(c - r);
    /* the tolerance: a binary32 product, then a binary32 sum (no fused
     * multiply-add); a non-finite reference admits only c == r */
    float tol = isfinite(r) ? atol + rtol * fabsf(r) : -1.0f;
    if (c == r) return 1; /* IEEE equality: +0 == -0, equal infinities */
    if (d <= tol) return 1;
    if ((flags & KBO_EQUAL_NAN) && isnan(c) && isnan(r)) return 1;
    return 0;
}

int kbo_screen_range(int dtype, const void* ref, const void* cand, uint64_t lo, uint64_t hi,
                     float atol, float rtol, uint32_t flags, kbo_partial* p) {
    if (dtype != KBO_F32 && dtype != KBO_F16 && dtype != KBO_BF16) return -1;
    fpenv_guard env = fpenv_enter();
    for (uint64_t i = lo; i < hi; ++i) {
        uint32_t cb, rb;
        float c, r;
        load_elem(dtype, cand, i, &cb, &c);
        load_elem(dtype, ref, i, &rb, &r);
        p->numel++;
        /* 1. bitwise identity on raw storage */
        p->bitdiff |= cb ^ rb;
        /* 2. non-finite values of the candidate */
        if (isnan(c)) p->nan_count++;
        else if (c == INFINITY) p->pos_inf_count++;
        else if (c == -INFINITY) p->neg_inf_count++;
        /* 3. match under |c - r| <= atol + rtol*|r| */
        if (!kbo_match(c, r, atol, rtol, flags)) p->mismatches++;
        /* 4. maxima; comparisons with NaN are false, so NaN never enters */
        float d = fabsf(c - r);
        if (d > p->max_abs_err) p->max_abs_err = d;
        float q = d / fabsf(r); /* x/0 = +inf, 0/0 and inf/inf = NaN (skipped) */
        if (q > p->max_rel_err) p->max_rel_err = q;
        /* 5. squared-error sums; each term is exact in binary64 */
        if (isfinite(c) && isfinite(r)) neumaier_add(&p->sum_sq_diff, &p->sum_sq_diff_comp,
                                                     (double)d * (double)d);
        if (isfinite(r)) neumaier_add(&p->sum_sq_ref, &p->sum_sq_ref_comp,
                                      (double)r * (double)r);
    }
    fpenv_leave(env);
    return 0;
}

void kbo_merge(kbo_partial* into, const kbo_partial* from) {
    into->numel += from->numel;
    into->mismatches += from->mismatches;
    into->nan_count += from->nan_count;
    into->pos_inf_count += from->pos_inf_count;
    into->neg_inf_count += from->neg_inf_count;
    neumaier_add(&into->sum_sq_diff, &into->sum_sq_diff_comp, from->sum_sq_diff);
    into->sum_sq_diff_comp += from->sum_sq_diff_comp;
    neumaier_add(&into->sum_sq_ref, &into->sum_sq_ref_comp, from->sum_sq_ref);
    into->sum_sq_ref_comp += from->sum_sq_ref_comp;
    if (from->max_abs_err > into->max_abs_err) into->max_abs_err = from->max_abs_err;
    if (from->max_rel_err > into->max_rel_err) into->max_rel_err = from->max_rel_err;
    into->bitdiff |= from->bitdiff;
}

void kbo_finalize(const kbo_partial* p, kbo_stats* out) {
    double ssd = isinf(p->sum_sq_diff) ? p->sum_sq_diff : p->sum_sq_diff + p->sum_sq_diff_comp;
    double ssr = isinf(p->sum_sq_ref) ? p->sum_sq_ref : p->sum_sq_ref + p->sum_sq_ref_comp;
    out->numel = p->numel;
    out->mismatches = p->mismatches;
    out->nan_count = p->nan_count;
    out->pos_inf_count = p->pos_inf_count;
    out->neg_inf_count = p->neg_inf_count;
    out->sum_sq_diff = ssd;
    out->sum_sq_ref = ssr;
    /* relative L2 error sqrt(sum d^2 / sum r^2); 0/0 -> 0, x/0 -> +inf */
    out->rel_l2 = ssr > 0.0 ? sqrt(ssd / ssr) : (ssd == 0.0 ? 0.0 : INFINITY);
    out->max_abs_err = p->max_abs_err;
    out->max_rel_err = p->max_rel_err;
    out->bitwise_equal = p->bitdiff == 0;
    out->passed = p->mismatches == 0;
}

int kbo_screen(int dtype, const void* ref, const void* cand, uint64_t n, float atol, float rtol,
               uint32_t flags, kbo_stats* out) {
    kbo_partial p;
    kbo_partial_init(&p);
    int rc = kbo_screen_range(dtype, ref, cand, 0, n, atol, rtol, flags, &p);
    if (rc) return rc;
    kbo_finalize(&p, out);
    return 0;
}

int kbo_locate(int dtype, const void* ref, const void* cand, uint64_t n, float atol, float rtol,
               uint32_t flags, float max_abs, float max_rel, kbo_locate_t* out) {
    if (dtype != KBO_F32 && dtype != KBO_F16 && dtype != KBO_BF16) return -1;
    fpenv_guard env = fpenv_enter();
    out->first_mismatch = out->max_abs_index = out->max_rel_index = -1;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t cb, rb;
        float c, r;
        load_elem(dtype, cand, i, &cb, &c);
        load_elem(dtype, ref, i, &rb, &r);
        float d = fabsf(c - r);
        float q = d / fabsf(r);
        if (out->first_mismatch < 0 && !kbo_match(c, r, atol, rtol, flags))
            out->first_mismatch = (int64_t)i;
        if (out->max_abs_index < 0 && max_abs > 0.0f && d == max_abs) out->max_abs_index = (int64_t)i;
        if (out->max_rel_index < 0 && max_rel > 0.0f && q == max_rel) out->max_rel_index = (int64_t)i;
    }
    fpenv_leave(env);
    return 0;
}

/* ---------------------------------------------------------------------------
 * Bulk forms (loops over the single-element definitions above).
 * ------------------------------------------------------------------------- */
void kbo_f32_to_f16_n(const float* in, uint16_t* out, uint64_t n) {
    fpenv_guard env = fpenv_enter();
    for (uint64_t i = 0; i < n; ++i) out[i] = kbo_f32_to_f16(in[i]);
    fpenv_leave(env);
}

void kbo_f32_to_bf16_n(const float* in, uint16_t* out, uint64_t n) {
    for (uint64_t i = 0; i < n; ++i) out[i] = kbo_f32_to_bf16(in[i]);
}

void kbo_f16_to_f32_n(const uint16_t* in, float* out, uint64_t n) {
    fpenv_guard env = fpenv_enter();
    for (uint64_t i = 0; i < n; ++i) out[i] = kbo_f16_to_f32(in[i]);
    fpenv_leave(env);
}

void kbo_bf16_to_f32_n(const uint16_t* in, float* out, uint64_t n) {
    for (uint64_t i = 0; i < n; ++i) out[i] = kbo_bf16_to_f32(in[i]);
}

void kbo_uniform_n(const uint32_t* x, float a, float b, float* out, uint64_t n) {
    fpenv_guard env = fpenv_enter();
    for (uint64_t i = 0; i < n; ++i) out[i] = kbo_uniform(x[i], a, b);
    fpenv_leave(env);
}

void kbo_match16_n(int dtype, const uint16_t* c, const uint16_t* r, float atol, float rtol,
                   uint32_t flags, uint8_t* out, uint64_t n) {
    fpenv_guard env = fpenv_enter();
    for (uint64_t i = 0; i < n; ++i) {
        float cv = dtype == KBO_F16 ? kbo_f16_to_f32(c[i]) : kbo_bf16_to_f32(c[i]);
        float rv = dtype == KBO_F16 ? kbo_f16_to_f32(r[i]) : kbo_bf16_to_f32(r[i]);
        out[i] = (uint8_t)kbo_match(cv, rv, atol, rtol, flags);
    }
    fpenv_leave(env);
}
