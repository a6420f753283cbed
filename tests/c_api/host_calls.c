/* A plain C11 client of the library's interface: it includes the header,
 * links libkb.so, and makes the calls that need no GPU -- the policy gate,
 * the verdict of host records, the rung survival table, the workspace size,
 * an argument error and its text, and the version.  Prints one line per
 * check and returns nonzero on the first failure. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "kb.h"

static int fails = 0;

static void check(int ok, const char* what) {
    printf("%s %s\n", ok ? "ok  " : "FAIL", what);
    if (!ok) fails++;
}

static kb_tensor tensor(const void* data, int dtype, int64_t rows, int64_t cols) {
    kb_tensor t;
    memset(&t, 0, sizeof t);
    t.data = data;
    t.dtype = dtype;
    t.ndim = 2;
    t.shape[0] = rows;
    t.shape[1] = cols;
    t.strides[0] = cols;
    t.strides[1] = 1;
    return t;
}

int main(void) {
    static float r[12], c[12];
    kb_tensor ref = tensor(r, KB_F32, 3, 4);
    kb_tensor cands[5];
    cands[0] = tensor(c, KB_F32, 3, 4);
    cands[1] = tensor(NULL, KB_F32, 3, 4);
    cands[2] = tensor(c, KB_F16, 3, 4);
    cands[3] = tensor(c, KB_F32, 4, 3);
    cands[4] = tensor(c, KB_F32, 3, 4);
    cands[4].strides[0] = 1;
    cands[4].strides[1] = 3;
    int32_t status[5];
    check(kb_policy_check(&ref, cands, 5, status) == KB_OK, "kb_policy_check returns KB_OK");
    check(status[0] == KB_STATUS_OK && status[1] == KB_REJECT_NULL && status[2] == KB_REJECT_DTYPE &&
              status[3] == KB_REJECT_SHAPE && status[4] == KB_REJECT_LAYOUT,
          "gate statuses: ok, null, dtype, shape, layout");

    kb_stats recs[3];
    memset(recs, 0, sizeof recs);
    recs[0].numel = 12;
    recs[1].numel = 12;
    recs[1].mismatches = 2;
    recs[2].status = KB_REJECT_SHAPE;
    kb_summary s;
    int32_t passed[3];
    check(kb_summarize(recs, 3, &s, passed) == KB_OK, "kb_summarize returns KB_OK");
    check(s.n_candidates == 3 && s.n_passed == 1 && s.n_failed == 1 && s.n_rejected == 1 &&
              s.first_passed == 0 && s.first_failed == 1,
          "summary counts");
    check(passed[0] == 1 && passed[1] == 0 && passed[2] == 0, "per-candidate verdicts");

    const int32_t entering[2] = {10, 4}, failed[2] = {2, 1}, promoted[2] = {4, 1};
    double fail_pct[2], promo_pct[2];
    check(kb_rung_survival(entering, failed, promoted, 2, 10, fail_pct, promo_pct) == KB_OK,
          "kb_rung_survival returns KB_OK");
    check(fabs(fail_pct[0] - 20.0) < 1e-12 && fabs(fail_pct[1] - 25.0) < 1e-12, "Fail% per rung");

    check(kb_screen_workspace_bytes(4, 1u << 20, KB_F32) > 0, "kb_screen_workspace_bytes is positive");
    check(kb_screen_workspace_bytes(4, 1u << 20, 99) == 0, "kb_screen_workspace_bytes is 0 for a bad dtype");

    check(kb_policy_check(NULL, cands, 5, status) == KB_ERR_INVALID_ARG, "a null reference is KB_ERR_INVALID_ARG");
    const char* e = kb_last_error();
    check(e != NULL && strlen(e) > 0, "kb_last_error describes it");
    check(kb_version() > 0, "kb_version");
    printf("%s\n", fails ? "FAILED" : "PASSED");
    return fails != 0;
}
