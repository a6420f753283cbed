/* The whole screening path from plain C on the GPU, with no Python and no
 * torch: device buffers from hipMalloc, a seeded N(0,1) reference from
 * kb_gen_inputs, three candidates made from it with exact expectations (a
 * copy; a copy with one element moved by half its tolerance; a copy with one
 * element moved far out of tolerance), kb_screen, kb_screen_stats, and
 * kb_screen_locate.  Prints one line per check; returns nonzero on failure.
 * Every buffer is sized for the n elements the calls are given. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "kb.h"

static int fails = 0;

static void check(int ok, const char* what) {
    printf("%s %s\n", ok ? "ok  " : "FAIL", what);
    fflush(stdout);
    if (!ok) fails++;
}

#define HIP_OK(x)                                                     \
    do {                                                              \
        hipError_t e_ = (x);                                          \
        if (e_ != hipSuccess) {                                       \
            printf("FAIL %s: %s\n", #x, hipGetErrorString(e_));       \
            return 1;                                                 \
        }                                                             \
    } while (0)

static kb_tensor vec(const void* data, int64_t n) {
    kb_tensor t;
    memset(&t, 0, sizeof t);
    t.data = data;
    t.dtype = KB_F32;
    t.ndim = 1;
    t.shape[0] = n;
    t.strides[0] = 1;
    return t;
}

int main(void) {
    const uint64_t n = (1u << 20) + 77;  /* several chunks and a ragged tail */
    const uint64_t q = 123457, p = n - 5;  /* the two moved elements */
    const float atol = 1e-5f, rtol = 1e-5f;
    float *ref = NULL, *cand[3] = {NULL, NULL, NULL};
    HIP_OK(hipMalloc((void**)&ref, n * sizeof(float)));
    for (int k = 0; k < 3; ++k) HIP_OK(hipMalloc((void**)&cand[k], n * sizeof(float)));
    check(kb_gen_inputs(ref, KB_F32, n, KB_DIST_NORMAL, 0.0f, 1.0f, 0, 0, 0, 0, NULL) == KB_OK,
          "kb_gen_inputs: N(0,1), seed 0");
    for (int k = 0; k < 3; ++k) HIP_OK(hipMemcpy(cand[k], ref, n * sizeof(float), hipMemcpyDeviceToDevice));
    float rq, rp;
    HIP_OK(hipMemcpy(&rq, ref + q, sizeof(float), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(&rp, ref + p, sizeof(float), hipMemcpyDeviceToHost));
    const float inside = rq + 0.5f * (atol + rtol * fabsf(rq));
    const float outside = rp + 1.0f;
    HIP_OK(hipMemcpy(cand[1] + q, &inside, sizeof(float), hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(cand[2] + p, &outside, sizeof(float), hipMemcpyHostToDevice));

    const kb_tensor r = vec(ref, (int64_t)n);
    const kb_tensor c[3] = {vec(cand[0], (int64_t)n), vec(cand[1], (int64_t)n), vec(cand[2], (int64_t)n)};
    const size_t ws_bytes = kb_screen_workspace_bytes(3, n, KB_F32);
    check(ws_bytes > 0, "kb_screen_workspace_bytes");
    void* ws = NULL;
    kb_stats* d_stats = NULL;
    kb_locate* d_loc = NULL;
    HIP_OK(hipMalloc(&ws, ws_bytes));
    HIP_OK(hipMalloc((void**)&d_stats, 3 * sizeof(kb_stats)));
    HIP_OK(hipMalloc((void**)&d_loc, 3 * sizeof(kb_locate)));
    check(kb_screen_workspace_init(ws, ws_bytes, NULL) == KB_OK, "kb_screen_workspace_init");
    check(kb_screen(&r, c, 3, atol, rtol, 0, ws, ws_bytes, d_stats, NULL) == KB_OK, "kb_screen");
    kb_stats h[3];
    kb_summary s;
    int32_t passed[3];
    check(kb_screen_stats(d_stats, 3, h, &s, passed, NULL) == KB_OK, "kb_screen_stats");
    check(passed[0] == 1 && passed[1] == 1 && passed[2] == 0, "verdicts: pass, pass, fail");
    check(s.n_passed == 2 && s.n_failed == 1 && s.first_failed == 2, "summary");
    check(h[0].bitwise_equal == 1 && h[0].mismatches == 0 && h[0].max_abs_err == 0.0f, "the copy is identical");
    check(h[1].bitwise_equal == 0 && h[1].mismatches == 0 && h[1].max_abs_err == fabsf(inside - rq),
          "one element inside its tolerance");
    check(h[2].mismatches == 1 && h[2].max_abs_err == fabsf(outside - rp) && h[2].numel == n,
          "one element outside: one mismatch, its difference the max");
    check(kb_screen_locate(&r, c, 3, atol, rtol, 0, d_stats, d_loc, NULL) == KB_OK, "kb_screen_locate");
    kb_locate loc[3];
    HIP_OK(hipMemcpy(loc, d_loc, sizeof loc, hipMemcpyDeviceToHost));
    check(loc[0].first_mismatch == -1 && loc[0].max_abs_index == -1, "no positions in the copy");
    check(loc[1].first_mismatch == -1 && loc[1].max_abs_index == (int64_t)q, "max abs at the moved element");
    check(loc[2].first_mismatch == (int64_t)p && loc[2].max_abs_index == (int64_t)p, "first mismatch at it");
    check(kb_screen(&r, c, 3, atol, rtol, 0, ws, 1, d_stats, NULL) == KB_ERR_WORKSPACE,
          "a short workspace is KB_ERR_WORKSPACE");
    hipFree(d_loc);
    hipFree(d_stats);
    hipFree(ws);
    for (int k = 0; k < 3; ++k) hipFree(cand[k]);
    hipFree(ref);
    printf("%s\n", fails ? "FAILED" : "PASSED");
    return fails != 0;
}
