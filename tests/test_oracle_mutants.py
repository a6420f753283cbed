"""The oracle's pins catch plausible mistakes in the oracle.

Each case plants one mistake (a dropped term, a wrong comparison, a wrong
operand, sign, index or constant) in a copy of the oracle's C source,
builds that copy, and runs the pins that cover the function it touches in a
child process pointed at the copy (KBO_LIB).  At least one pin must fail.
Only pins take part, never the stored golden records (which the oracle
itself wrote).  The planted mistakes live here, in the test, on the CPU;
the oracle's own sources are never modified."""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from oracle import build as oracle_build  # noqa: E402

SCREEN = ["tests/test_oracle_screen.py"]
PHILOX = ["tests/test_oracle_philox.py"]
# (the two exhaustive narrowing tests take a minute; the sampled one stands in for them)
MAPS = ["tests/test_oracle_maps.py", "-k", "not f32_to_f16_all_inputs and not f32_to_bf16_all_inputs"]
RUNG = ["tests/test_oracle_rung.py"]
LOCATE = ["tests/test_oracle_locate.py"]
DERIVED = ["tests/test_oracle_derived.py"]

# (name, source file, text, replacement, pins)
MUTANTS = [
    ("le_becomes_lt", "kbo.c", "if (d <= tol) return 1;", "if (d < tol) return 1;", SCREEN),
    ("tolerance_fused", "kbo.c", "float tol = isfinite(r) ? atol + rtol * fabsf(r) : -1.0f;",
     "float tol = isfinite(r) ? fmaf(rtol, fabsf(r), atol) : -1.0f;", SCREEN),
    ("tolerance_scaled_by_candidate", "kbo.c", "float tol = isfinite(r) ? atol + rtol * fabsf(r) : -1.0f;",
     "float tol = isfinite(r) ? atol + rtol * fabsf(c) : -1.0f;", SCREEN),
    ("equality_clause_dropped", "kbo.c", "if (c == r) return 1; /*", "if (0) return 1; /*", SCREEN),
    ("equal_nan_ignored", "kbo.c", "if ((flags & KBO_EQUAL_NAN) && isnan(c) && isnan(r)) return 1;",
     "if (0) return 1;", SCREEN),
    ("rel_error_over_candidate", "kbo.c", "float q = d / fabsf(r); /* x/0", "float q = d / fabsf(c); /* x/0",
     SCREEN),
    ("ref_squares_include_infinities", "kbo.c", "if (isfinite(r)) neumaier_add(&p->sum_sq_ref",
     "if (!isnan(r)) neumaier_add(&p->sum_sq_ref", SCREEN),
    ("diff_squares_include_infinities", "kbo.c",
     "if (isfinite(c) && isfinite(r)) neumaier_add(&p->sum_sq_diff",
     "if (!isnan(d)) neumaier_add(&p->sum_sq_diff", SCREEN),
    ("bitwise_on_values", "kbo.c", "p->bitdiff |= cb ^ rb;", "p->bitdiff |= (uint32_t)(c != r);", SCREEN),
    ("negative_inf_counted_as_positive", "kbo.c", "else if (c == -INFINITY) p->neg_inf_count++;",
     "else if (c == -INFINITY) p->pos_inf_count++;", SCREEN),
    ("rel_l2_without_sqrt", "kbo.c", "out->rel_l2 = ssr > 0.0 ? sqrt(ssd / ssr)",
     "out->rel_l2 = ssr > 0.0 ? (ssd / ssr)", SCREEN),
    ("philox_multiplier", "kbo.c", "#define PHILOX_M0 0xD2511F53u", "#define PHILOX_M0 0xD2511F55u", PHILOX),
    ("philox_words_crossed", "kbo.c", "uint32_t y0 = hi1 ^ x1 ^ k0;", "uint32_t y0 = hi0 ^ x1 ^ k0;", PHILOX),
    ("philox_key_schedule", "kbo.c", "k1 += PHILOX_W1;", "k1 += PHILOX_W0;", PHILOX),
    ("stream_counter_words_swapped", "kbo.c",
     "uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), sub, stream_id};",
     "uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), stream_id, sub};", PHILOX),
    ("uniform_wrong_bits", "kbo.c", "return (float)(x >> 8) * 0x1p-24f;", "return (float)(x >> 9) * 0x1p-23f;",
     MAPS),
    ("normal_sin_cos_swapped", "kbo.c", "*zc = rho * cos(theta);\n    *zs = rho * sin(theta);",
     "*zc = rho * sin(theta);\n    *zs = rho * cos(theta);", MAPS),
    ("normal_u1_without_offset", "kbo.c", "double u1 = ((double)xa + 1.0) * 0x1p-32;",
     "double u1 = ((double)xa + 0.5) * 0x1p-32;", MAPS),
    ("quantile_position", "kbo_rung.c", "const double h = (double)(n - 1) * p;",
     "const double h = (double)n * p;", RUNG),
    ("speedup_inverted", "kbo_rung.c", "r->speedup = r->valid ? b / r->mean : NAN;",
     "r->speedup = r->valid ? r->mean / b : NAN;", RUNG),
    ("score_alpha_beta_swapped", "kbo_rung.c", "return lead + (alpha * (double)rung + beta * budget);",
     "return lead + (beta * (double)rung + alpha * budget);", RUNG),
    ("score_latency_floor_dropped", "kbo_rung.c", "const double lead = 1e6 / (latency > 1.0 ? latency : 1.0);",
     "const double lead = 1e6 / latency;", RUNG),
    ("score_rung_term_dropped", "kbo_rung.c", "return lead + (alpha * (double)rung + beta * budget);",
     "return lead + (beta * budget);", RUNG),
    ("locate_first_mismatch_last", "kbo.c",
     "if (out->first_mismatch < 0 && !kbo_match(c, r, atol, rtol, flags))",
     "if (!kbo_match(c, r, atol, rtol, flags))", LOCATE),
    ("locate_max_abs_last", "kbo.c", "if (out->max_abs_index < 0 && max_abs > 0.0f && d == max_abs)",
     "if (max_abs > 0.0f && d == max_abs)", LOCATE),
    ("locate_max_rel_of_candidate", "kbo.c", "float q = d / fabsf(r);\n        if (out->first_mismatch",
     "float q = d / fabsf(c);\n        if (out->first_mismatch", LOCATE),
    # the promotion decision and the survival table
    ("promote_ties_to_higher_index", "kbo_rung.c", "return key[j] > key[i] || (key[j] == key[i] && j < i);",
     "return key[j] > key[i] || (key[j] == key[i] && j > i);", RUNG),
    ("promote_keep_rounded_down", "kbo_rung.c", "((long long)n_eligible * num + den - 1) / den",
     "((long long)n_eligible * num) / den", RUNG),
    ("promote_invalid_baseline", "kbo_rung.c", "p = valid[i] != 0;", "p = 1;", RUNG),
    ("promote_baseline_counted_eligible", "kbo_rung.c", "n_eligible += valid[i] && i != base;",
     "n_eligible += valid[i];", RUNG),
    ("promote_invalid_ranked_by_score", "kbo_rung.c",
     "key[i] = valid[i] && !isnan(score[i]) ? score[i] : -INFINITY;",
     "key[i] = !isnan(score[i]) ? score[i] : -INFINITY;", RUNG),
    ("survival_fail_over_original", "kbo_rung.c",
     "100.0 * (double)failed[r] / (double)entering[r]", "100.0 * (double)failed[r] / (double)original", RUNG),
    # binary32 -> binary16 / bfloat16 rounding and back
    ("rounding_ties_away", "kbo.c", "if (rem > half || (rem == half && (q & 1))) q++;",
     "if (rem >= half) q++;", MAPS),
    ("f16_overflow_saturates", "kbo.c", "mag = enc >= 0x7c00u ? 0x7c00u : (uint32_t)enc;",
     "mag = enc >= 0x7c00u ? 0x7bffu : (uint32_t)enc;", MAPS),
    ("f16_subnormal_scale", "kbo.c", "q = shift_rne(m, -e - 1);", "q = shift_rne(m, -e);", MAPS),
    ("bf16_nan_truncated", "kbo.c", "if (mag > 0x7f800000u) return (uint16_t)(sign | 0x7fc0u);",
     "if (mag > 0x7f800000u) return (uint16_t)(sign | (mag >> 16));", MAPS),
    ("f16_widen_subnormal_scale", "kbo.c", "ldexpf((float)man, -24)", "ldexpf((float)man, -25)", MAPS),
    # derived inputs: Student-t, softmax rows, index draws, planted changes
    ("t3_numerator_from_sine", "kbo_derived.c", "return z0 / sqrt(chi2 / 3.0);",
     "return z1 / sqrt(chi2 / 3.0);", DERIVED),
    ("t3_two_degrees_of_freedom", "kbo_derived.c", "double chi2 = (z1 * z1 + z2 * z2) + z3 * z3;",
     "double chi2 = (z1 * z1 + z2 * z2);", DERIVED),
    ("t3_not_divided_by_3", "kbo_derived.c", "return z0 / sqrt(chi2 / 3.0);", "return z0 / sqrt(chi2);",
     DERIVED),
    ("t3_numerator_in_chi_square", "kbo_derived.c", "double chi2 = (z1 * z1 + z2 * z2) + z3 * z3;",
     "double chi2 = (z0 * z0 + z2 * z2) + z3 * z3;", DERIVED),
    ("softmax_max_not_taken", "kbo_derived.c", "if (x[j] > m) m = x[j];", "if (0) m = x[j];", DERIVED),
    ("softmax_sum_in_binary32", "kbo_derived.c", "double s = 0.0;", "float s = 0.0f;", DERIVED),
    ("softmax_row_offset_dropped", "kbo_derived.c", "(row0 + i) * cols);", "i * cols);", DERIVED),
    ("indices_words_swapped", "kbo_derived.c", "(((uint64_t)w[1] << 32) | w[0])",
     "(((uint64_t)w[0] << 32) | w[1])", DERIVED),
    ("indices_repeats_kept", "kbo_derived.c", "if (!seen) out[have++] = x;", "out[have++] = x;", DERIVED),
    ("indices_block_shifted", "kbo_derived.c", "kbo_stream_block(seed, stream_id, sub, j, w);",
     "kbo_stream_block(seed, stream_id, sub, j + 1, w);", DERIVED),
    ("perturb_word_of_local_index", "kbo_derived.c", "const uint32_t word = w[g & 3u];",
     "const uint32_t word = w[j & 3u];", DERIVED),
    ("perturb_rel_not_fused", "kbo_derived.c", "store(dtype, dst, j, fmaf(x, kbo_uniform(word, a, b), x));",
     "store(dtype, dst, j, x * kbo_uniform(word, a, b) + x);", DERIVED),
    ("perturb_mask_inverted", "kbo_derived.c", "if (kbo_u01(word) < p) store(dtype, dst, j, x * a);",
     "if (kbo_u01(word) >= p) store(dtype, dst, j, x * a);", DERIVED),
    ("specials_sign_from_word0", "kbo_derived.c", "const uint32_t sign = w[1] & 0x80000000u;",
     "const uint32_t sign = w[0] & 0x80000000u;", DERIVED),
    ("specials_thresholds_not_cumulative", "kbo_derived.c", "else if (v < b) out = sign;",
     "else if (v < b - a) out = sign;", DERIVED),
    ("specials_mantissa_may_be_even", "kbo_derived.c", "(w[2] & 0x7FFFFFu) | 1u;", "(w[2] & 0x7FFFFFu);",
     DERIVED),
    ("flush_keeps_subnormal", "kbo_derived.c", "else if (mag < 0x00800000u) out = bits & 0x80000000u;",
     "else if (mag < 0x00800000u) out = bits;", DERIVED),
    ("relative_change_from_word0", "kbo_derived.c", "fmaf(x, kbo_uniform(w[1], a, b), x)",
     "fmaf(x, kbo_uniform(w[0], a, b), x)", DERIVED),
    ("scatter_infinity_unsigned", "kbo_derived.c", "(sign | 0x7F800000u)", "0x7F800000u", DERIVED),
    ("created_nan_not_canonical", "kbo_derived.c", "    if (isnan(v)) {\n        if (dtype == KBO_F32)",
     "    if (0) {\n        if (dtype == KBO_F32)", DERIVED),
]


def _run_mutant(tmp, name, src, text, repl, pins):
    """Build the oracle with one planted mistake and run the pins against
    it: (pytest's exit code, the tail of its output)."""
    os.makedirs(tmp, exist_ok=True)
    odir = os.path.join(ROOT, "oracle")
    for f in os.listdir(odir):
        if f.endswith((".c", ".h")):
            shutil.copy(os.path.join(odir, f), os.path.join(tmp, f))
    path = os.path.join(tmp, src)
    with open(path) as f:
        code = f.read()
    if code.count(text) != 1:
        return -1, "mutation site of %s not found exactly once" % name
    with open(path, "w") as f:
        f.write(code.replace(text, repl))
    lib = os.path.join(tmp, "libkbo_mutant.so")
    sources = [os.path.join(tmp, os.path.basename(s)) for s in oracle_build.SOURCES]
    subprocess.run(["gcc", *oracle_build.CFLAGS, *sources, "-o", lib, "-lm"], check=True,
                   capture_output=True, text=True)
    env = dict(os.environ, KBO_LIB=lib)
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                          *pins], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return res.returncode, res.stdout[-2000:]


@pytest.fixture(scope="module")
def mutant_results(tmp_path_factory):
    """Every mutant, built and run against its pins, a few at a time."""
    base = str(tmp_path_factory.mktemp("mutants"))
    with ThreadPoolExecutor(max_workers=max(1, min(6, (os.cpu_count() or 2) - 1))) as ex:
        futs = {m[0]: ex.submit(_run_mutant, os.path.join(base, m[0]), *m) for m in MUTANTS}
        return {k: f.result() for k, f in futs.items()}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
@pytest.mark.parametrize("name", [m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(mutant_results, name):
    rc, out = mutant_results[name]
    # pytest exits with 1 when a test failed (2: interrupted or not collected)
    assert rc == 1, "mutant %s: pins exited with %d (1 = a pin failed):\n%s" % (name, rc, out)
