/*
 * kbo.h -- plain CPU oracle for the candidate-screening path.
 *
 * TEST INFRASTRUCTURE ONLY.  The test suite, the package smoke check and the
 * benchmark's CPU-baseline leg are the only callers.  The HIP library never
 * includes, links or calls anything declared here, and this file includes
 * nothing from the HIP library: the two sides are written independently and
 * compared.
 *
 * What the oracle computes (paper: "KernelBrain", Section 3):
 *   - the correctness indicator K(p) of Section 3.1 for one output tensor,
 *     i.e. the numeric check of the Verifier in Section 3.4 ("Evaluation
 *     Plane"), evaluated element by element against a reference output under
 *     |c - r| <= atol + rtol*|r|, with the per-candidate statistics listed on
 *     kbo_partial below;
 *   - the seeded inputs such tests run on: a Philox4x32-10 counter-based
 *     stream (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as
 *     1, 2, 3", SC'11) mapped to uniform and normal floats;
 *   - the rung benchmarker's statistics over timing samples (kbo_rung.c):
 *     mean, quantiles and tail ratios per shape, speedups, and the runtime
 *     score of Eq. 2.
 *
 * Enumerations use the same numeric codes as the library's C interface so
 * that a test can pass one code to both sides; that interface is the only
 * thing the two sides have in common.
 */
#ifndef KBO_H
#define KBO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { KBO_F32 = 0, KBO_F16 = 1, KBO_BF16 = 2, KBO_U32 = 3 };
enum { KBO_DIST_U32 = 0, KBO_DIST_UNIFORM = 1, KBO_DIST_NORMAL = 2, KBO_DIST_STUDENT_T3 = 3 };
enum { KBO_EQUAL_NAN = 1u };

/* Philox4x32-10 block function (SC'11, Section 4 "Philox"): ten rounds of
 * two 32x32->64 multiplies and xors, key bumped by the Weyl constants between
 * rounds.  in = counter (x0..x3), key = (k0, k1). */
void kbo_philox4x32_10(const uint32_t in[4], const uint32_t key[2], uint32_t out[4]);

/* Block b of stream (stream_id, sub) under seed: key = (lo32(seed),
 * hi32(seed)), counter = (lo32(b), hi32(b), sub, stream_id). */
void kbo_stream_block(uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t b,
                      uint32_t out[4]);

/* u = (x >> 8) * 2^-24, exact, in [0, 1). */
float kbo_u01(uint32_t x);
/* U(a, b) value: fmaf(u, fl32(b - a), a), one rounding. */
float kbo_uniform(uint32_t x, float a, float b);
/* Box-Muller on one word pair in binary64: u1 = (xa + 1) 2^-32, u2 = xb 2^-32,
 * rho = sqrt(-2 ln u1), theta = 2 pi u2 (2 pi rounded to binary64); the
 * cosine and sine branches rho cos(theta), rho sin(theta), unrounded. */
void kbo_box_muller64(uint32_t xa, uint32_t xb, double* zc, double* zs);
/* Standard normal from one word pair by the Box-Muller transform, in
 * binary64 then rounded once to binary32.  odd = 0 takes the cosine branch,
 * odd = 1 the sine branch. */
float kbo_normal01(uint32_t xa, uint32_t xb, int odd);

/* IEEE 754 conversions, round to nearest even. */
uint16_t kbo_f32_to_f16(float f);
uint16_t kbo_f32_to_bf16(float f);
float kbo_f16_to_f32(uint16_t h);
float kbo_bf16_to_f32(uint16_t h);

/* Fill dst[0..n) with elements offset..offset+n-1 of the stream.
 * dist U32 needs dtype U32; UNIFORM takes [p0, p1); NORMAL takes mean p0,
 * standard deviation p1; STUDENT_T3 takes location p0 and scale p1, element g
 * being kbo_student_t3 of block g.  16-bit dtypes round the binary32 value
 * to nearest even.  Returns 0, or -1 for an invalid (dtype, dist) pair. */
int kbo_gen(void* dst, int dtype, uint64_t n, int dist, float p0, float p1,
            uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset);

/* ---- derived inputs (kbo_derived.c) ---- */

/* Student-t with 3 degrees of freedom from one block's four words: the four
 * binary64 normals z0, z1 (Box-Muller on words 0, 1) and z2, z3 (words 2, 3),
 * t = z0 / sqrt(((z1^2 + z2^2) + z3^2) / 3) in binary64 (the ratio of a
 * normal to the root of an independent chi-square over its 3 degrees of
 * freedom), then rounded once to binary32. */
double kbo_student_t3_64(const uint32_t w[4]);
float kbo_student_t3(const uint32_t w[4]);

/* Softmax of one row of binary32 logits x[0..n), n >= 1, in binary64:
 * m = max x, e_j = exp(x_j - m), s = e_0 + e_1 + ... (left to right),
 * out_j = e_j / s rounded once to binary32. */
void kbo_softmax_row(const float* x, uint64_t n, float* out);
/* Rows row0 .. row0 + rows - 1 of a [*][cols] softmax tensor whose logits are
 * the NORMAL stream (mean 0, standard deviation sigma): logit (i, j) is
 * element i cols + j of kbo_gen(F32, NORMAL, 0, sigma).  dst holds
 * rows * cols binary32 values.  Returns 0, or -1 for cols = 0. */
int kbo_gen_softmax_rows(float* dst, uint64_t row0, uint64_t rows, uint64_t cols, float sigma,
                         uint64_t seed, uint32_t stream_id, uint32_t sub);

/* m distinct indices in [0, n), in draw order: draw j = 0, 1, 2, ... is
 * ((w1 << 32) | w0) mod n of block j of the stream; a draw equal to an
 * earlier accepted index is skipped.  Returns 0, or -1 unless 1 <= n and
 * m <= n. */
int kbo_gen_indices(uint64_t* out, uint32_t m, uint64_t n, uint64_t seed, uint32_t stream_id,
                    uint32_t sub);

/* Planted changes of a seeded candidate (dst[j] from src[j], element g =
 * offset + j; dst may be src).  x is src widened to binary32, and "narrow"
 * rounds a binary32 value to the dtype (nearest even), a NaN result becoming
 * the dtype's positive quiet NaN (f32 0x7FC00000, f16 0x7E00, bf16 0x7FC0).  u(g) is the uniform
 * [0, 1) value of word g mod 4 of block g / 4 (as kbo_gen UNIFORM with
 * [0, 1)), U(g) the one with [a, b), and N(g) the NORMAL element g with mean
 * 0 and standard deviation a; ops 6 and 7 use the four words w0..w3 of
 * block g and take only F32.
 *   1 ADD_UNIFORM         narrow(x + U(g))
 *   2 REL_UNIFORM         narrow(fmaf(x, U(g), x))
 *   3 ADD_NORMAL          narrow(x + N(g))
 *   4 SCALE_WHERE         u(g) < p ? narrow(x * a) : src
 *   5 FLIP_LSB_WHERE      u(g) < p ? storage bits ^ 1 : src
 *   6 SPECIALS            with v = u01(w0), the sign s = w1 >> 31 and the
 *                         mantissa (w2 & 0x7FFFFF) | 1: v < a: the subnormal
 *                         of that sign and mantissa; else v < b: zero of
 *                         sign s; else v < p: infinity of sign s; else src
 *                         (a <= b <= p are cumulative thresholds)
 *   7 ZERO_SUBNORMAL_REL  with v = u01(w0) and d = the [a, b) value of w1:
 *                         v < p: a zero changes sign, a subnormal becomes
 *                         the zero of its sign, a finite normal becomes
 *                         fmaf(x, d, x), an infinity or NaN is kept; else src
 * Returns 0, or -1 for an unknown op or an op/dtype pair not defined. */
enum {
    KBO_PERTURB_ADD_UNIFORM = 1,
    KBO_PERTURB_REL_UNIFORM = 2,
    KBO_PERTURB_ADD_NORMAL = 3,
    KBO_PERTURB_SCALE_WHERE = 4,
    KBO_PERTURB_FLIP_LSB_WHERE = 5,
    KBO_PERTURB_SPECIALS = 6,
    KBO_PERTURB_ZERO_SUBNORMAL_REL = 7
};
int kbo_perturb(void* dst, const void* src, int dtype, uint64_t n, int op, float a, float b, float p,
                uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset);

/* Set dst[idx[i]] for i < m (indices >= n are skipped): mode 1 the quiet
 * NaN of the dtype (f32 0x7FC00000, f16 0x7E00, bf16 0x7FC0); mode 2 the
 * infinity with the sign bit of ref[idx[i]].  Returns 0, or -1 for an
 * unknown mode or dtype. */
enum { KBO_SCATTER_NAN = 1, KBO_SCATTER_INF_SIGN_OF_REF = 2 };
int kbo_scatter(void* dst, const void* ref, int dtype, uint64_t n, const uint64_t* idx, uint32_t m,
                int mode);

/* Mergeable per-candidate screening state over a range of elements.  Sums are
 * Neumaier-compensated binary64 (value = sum + comp). */
typedef struct {
    uint64_t numel;
    uint64_t mismatches;
    uint64_t nan_count;
    uint64_t pos_inf_count;
    uint64_t neg_inf_count;
    double sum_sq_diff, sum_sq_diff_comp;
    double sum_sq_ref, sum_sq_ref_comp;
    float max_abs_err;
    float max_rel_err;
    uint32_t bitdiff;  /* OR over elements of (storage bits of c) ^ (storage bits of r) */
    uint32_t _pad;
} kbo_partial;

/* Final per-candidate statistics. */
typedef struct {
    uint64_t numel, mismatches, nan_count, pos_inf_count, neg_inf_count;
    double sum_sq_diff, sum_sq_ref, rel_l2;
    float max_abs_err, max_rel_err;
    int32_t bitwise_equal;
    int32_t passed;
} kbo_stats;

void kbo_partial_init(kbo_partial* p);
/* Accumulate elements [lo, hi) of (ref, cand) into p.  dtype F32, F16 or
 * BF16; both buffers hold raw storage of that dtype. */
int kbo_screen_range(int dtype, const void* ref, const void* cand, uint64_t lo, uint64_t hi,
                     float atol, float rtol, uint32_t flags, kbo_partial* p);
/* into <- into (+) from: counts add, maxima take the max, bit differences OR,
 * sums add. */
void kbo_merge(kbo_partial* into, const kbo_partial* from);
void kbo_finalize(const kbo_partial* p, kbo_stats* out);
/* Whole-tensor convenience: init, one range [0, n), finalize. */
int kbo_screen(int dtype, const void* ref, const void* cand, uint64_t n, float atol, float rtol,
               uint32_t flags, kbo_stats* out);

/* The single-element match predicate. */
int kbo_match(float c, float r, float atol, float rtol, uint32_t flags);

/* Positions in one candidate, for the diagnostics fed back about a failed
 * candidate: the smallest element index i
 *   first_mismatch: with kbo_match(c_i, r_i) false;
 *   max_abs_index:  with |fl(c_i - r_i)| == max_abs (only if max_abs > 0);
 *   max_rel_index:  with fl(|fl(c_i - r_i)| / |r_i|) == max_rel (only if
 *                   max_rel > 0);
 * each -1 when no element qualifies.  max_abs and max_rel are the
 * candidate's maxima (kbo_stats). */
typedef struct {
    int64_t first_mismatch, max_abs_index, max_rel_index;
} kbo_locate_t;
int kbo_locate(int dtype, const void* ref, const void* cand, uint64_t n, float atol, float rtol,
               uint32_t flags, float max_abs, float max_rel, kbo_locate_t* out);

/* Elementwise bulk forms of the maps above, for exhaustive sweeps. */
void kbo_f32_to_f16_n(const float* in, uint16_t* out, uint64_t n);
void kbo_f32_to_bf16_n(const float* in, uint16_t* out, uint64_t n);
void kbo_f16_to_f32_n(const uint16_t* in, float* out, uint64_t n);
void kbo_bf16_to_f32_n(const uint16_t* in, float* out, uint64_t n);
void kbo_uniform_n(const uint32_t* x, float a, float b, float* out, uint64_t n);
/* out[i] = match(widen(c[i]), widen(r[i])) for 16-bit storage c, r. */
void kbo_match16_n(int dtype, const uint16_t* c, const uint16_t* r, float atol, float rtol,
                   uint32_t flags, uint8_t* out, uint64_t n);

/* ---- rung benchmarker statistics (kbo_rung.c) ---- */

/* One (candidate, shape) row of timing samples (us). */
typedef struct {
    double mean, p50, p90, p95, p99;
    double tail90, tail95, tail99; /* p90/p50, p95/p50, p99/p50 */
    double speedup;                /* baseline row mean / this row mean */
    int32_t n, valid;
} kbo_row_t;

/* One candidate at one rung. */
typedef struct {
    double latency, score, speedup;
    int32_t valid, _pad;
} kbo_score_t;

/* The p-quantile of x[0..n) sorted ascending, n >= 1 (linear interpolation
 * at position (n - 1) p). */
double kbo_quantile_sorted(const double* x, int n, double p);
/* Statistics of one row (speedup left NaN). */
void kbo_row_stats(const double* t, int n, kbo_row_t* out);
/* 1e6 / max(1, latency) + alpha rung + beta budget. */
double kbo_rung_score_of(double latency, int rung, double budget, double alpha, double beta);
/* Every row of samples[n_cands][n_shapes][n_iter] and every candidate's
 * score; base = the baseline candidate's index, or -1 for none (speedups
 * NaN).  Returns 0, or -1 on bad sizes. */
int kbo_rung_stats(const double* samples, int n_cands, int n_shapes, int n_iter, int base,
                   int rung, double budget, double alpha, double beta, kbo_row_t* rows,
                   kbo_score_t* scores);

/* Promotion decision over n candidates' scores (valid[i] = 0 for invalid
 * candidates, whose score is -inf): rank[i] = position of candidate i (0 =
 * best), order[r] = candidate at position r, promoted[i] = 1 for the first
 * ceil(n_eligible num / den) valid non-baseline candidates in rank order and
 * for a valid baseline.  base = -1 for none.  Returns 0, or -1 on bad
 * arguments (0 <= num <= den, den >= 1). */
int kbo_rung_promote(const double* score, const int32_t* valid, int n, int base, int num, int den,
                     int32_t* rank, int32_t* order, int32_t* promoted);

/* Table A.1's columns from per-rung counts: fail_pct[r] = 100 failed[r] /
 * entering[r], promo_pct[r] = 100 promoted[r] / original. */
int kbo_rung_survival(const int32_t* entering, const int32_t* failed, const int32_t* promoted,
                      int n_rungs, int original, double* fail_pct, double* promo_pct);

#ifdef __cplusplus
}
#endif
#endif /* KBO_H */
