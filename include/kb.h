/*
 * kb.h -- C interface of the MI355X candidate-screening library (libkb.so).
 *
 * The library is the data-parallel hot path of the low-cost screening stage of
 * a budget-aware, multi-fidelity kernel search ("KernelBrain", Section 3).
 * There, every candidate first passes a policy check V(p) -- its output must
 * satisfy the shape and dtype constraints of the reference (Section 3.2,
 * "Policy check") -- and the Verifier then checks its output against the
 * reference output (Section 3.4, "Evaluation Plane"); the result is the
 * correctness indicator K(p) of the problem formulation (Section 3.1), and
 * Algorithm 1 discards a candidate that fails either gate before any
 * benchmarking budget is spent.  Section 3.3 (Observation 2) relies on such
 * wrong outputs being rejected in milliseconds.  This library does that check
 * for K candidate outputs at once, in one coalesced pass over HBM, on the
 * seeded inputs it can also generate.
 *
 * Three subsystems:
 *   kb_gen_inputs   seeded inputs: a Philox4x32-10 counter-based stream
 *                   (Salmon et al., SC'11) mapped to u32, uniform, normal or
 *                   Student-t values (fp32, fp16, bf16), and the derived
 *                   inputs of the screening workloads (kb_gen_softmax_rows,
 *                   kb_gen_indices, kb_gen_perturb, kb_gen_scatter);
 *   kb_screen       policy gate + one pass over the reference and the K
 *                   candidates computing, per candidate, the mismatch count
 *                   under |c - r| <= atol + rtol*|r|, max abs and max rel
 *                   error, NaN / +Inf / -Inf counts, a bitwise-identity flag
 *                   and the relative L2 error (kb_screen_ex: also the
 *                   positions of the first mismatch and of the maxima);
 *   kb_screen_stats reads the per-candidate records back and gives the
 *                   pass/fail verdict of each candidate.
 * Around them: the separate position pass (kb_screen_locate), multi-output
 * candidates (kb_screen_multi), the rung benchmarker's statistics and
 * promotion decision (kb_rung_stats, kb_rung_promote, kb_rung_survival), and
 * kb_screen_noalloc for callers that cannot allocate.
 *
 * Conventions
 *   - Every function is extern "C" and returns an int status: KB_OK (0) or a
 *     negative KB_ERR_* code.  On error nothing is launched and
 *     kb_last_error() describes the problem.  No C++ exception crosses the
 *     interface.
 *   - Pointers marked "device" are HIP device memory on the current device;
 *     "host" pointers are ordinary host memory.  The caller owns every
 *     buffer and keeps it alive until the stream reaches the call.
 *   - kb_gen_inputs and kb_screen are asynchronous and stream-ordered on the
 *     given hipStream_t (NULL = the default stream).  kb_screen_stats
 *     synchronizes that stream.
 *   - The library allocates no device memory and keeps no mutable state
 *     beyond the calling thread's error text and a per-process cache of
 *     kernel occupancy queries (and, for kb_screen_noalloc, the address of
 *     its fixed device scratch on each device).  A call with more than
 *     KB_INLINE_CANDS candidates is given a launch-table buffer of the
 *     caller's pinned host memory (kb_screen_ex, kb_screen_multi).
 *   - Device buffers must be 16-byte aligned (hipMalloc and torch
 *     allocations are); element counts may be anything, including 0.
 *   - A "data pointer" of a tensor points at element 0; strides are in
 *     elements.
 */
#ifndef KB_H
#define KB_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KB_MAX_DIMS 8

/* Element types.  KB_U32 exists for the generator's raw word stream only. */
typedef enum kb_dtype { KB_F32 = 0, KB_F16 = 1, KB_BF16 = 2, KB_U32 = 3 } kb_dtype;

/* Generator distributions. */
typedef enum kb_dist {
    KB_DIST_U32 = 0,
    KB_DIST_UNIFORM = 1,
    KB_DIST_NORMAL = 2,
    KB_DIST_STUDENT_T3 = 3
} kb_dist;

/* Call-level status codes (function return values). */
enum {
    KB_OK = 0,
    KB_ERR_INVALID_ARG = -1, /* null pointer, bad count, bad tolerance, bad flags */
    KB_ERR_DTYPE = -2,       /* unknown dtype, or a dtype the call does not take */
    KB_ERR_WORKSPACE = -3,   /* workspace missing or smaller than required */
    KB_ERR_ALIGNMENT = -4,   /* a device pointer is not 16-byte aligned */
    KB_ERR_HIP = -5          /* a HIP runtime call failed (text in kb_last_error) */
};

/* Per-candidate policy status (kb_stats.status); a candidate that fails the
 * gate is not read and is reported with zero statistics and passed = 0. */
enum {
    KB_STATUS_OK = 0,
    KB_REJECT_NULL = 1,   /* candidate data pointer is NULL (and it is not empty) */
    KB_REJECT_DTYPE = 2,  /* dtype differs from the reference */
    KB_REJECT_SHAPE = 3,  /* ndim or a dimension differs from the reference */
    KB_REJECT_LAYOUT = 4  /* not dense row-major (strides of a contiguous tensor) */
};

/* kb_screen flags. */
enum {
    KB_EQUAL_NAN = 1u << 0, /* a NaN candidate element matches a NaN reference element */
    KB_FAIL_FAST = 1u << 1  /* stop reading a candidate once a mismatch is seen (kb_screen) */
};

/* A tensor view.  data: device pointer to element 0 (may be NULL for a
 * candidate, which the policy gate then rejects).  dtype: a kb_dtype.
 * shape[0..ndim) and strides[0..ndim) in elements; ndim in [0, KB_MAX_DIMS]
 * (ndim = 0 is a scalar with one element). */
typedef struct kb_tensor {
    const void* data;
    int32_t dtype;
    int32_t ndim;
    int64_t shape[KB_MAX_DIMS];
    int64_t strides[KB_MAX_DIMS];
} kb_tensor;

/* Per-candidate screening record, 80 bytes, written to device memory by
 * kb_screen (kb_summarize and kb_screen_stats give each record's pass/fail
 * verdict K(p)).  For a candidate that passed the policy gate:
 *   numel          elements compared (= reference numel);
 *   mismatches     elements with NOT match, where match means c == r
 *                  (IEEE equality: +0 == -0, equal infinities), or
 *                  |c - r| <= atol + rtol*|r| with a finite r, or -- with
 *                  KB_EQUAL_NAN -- c and r both NaN.  c and r are the exact
 *                  binary32 widenings of the stored values; c - r, rtol*|r|
 *                  and the sum are each rounded to binary32 (no fused
 *                  multiply-add);
 *   nan_count, pos_inf_count, neg_inf_count   non-finite candidate elements;
 *   sum_sq_diff    sum of (c - r)^2 over elements where c and r are finite,
 *                  each term the binary64 square of the binary32 difference;
 *   sum_sq_ref     sum of r^2 over elements where r is finite (the same for
 *                  every candidate);
 *   rel_l2         sqrt(sum_sq_diff / sum_sq_ref); 0 if both are 0, +inf if
 *                  only sum_sq_ref is 0;
 *   max_abs_err    max over elements of |c - r| (binary32), NaN ignored,
 *                  0 if none;
 *   max_rel_err    max over elements of |c - r| / |r| (binary32 division),
 *                  NaN quotients (0/0, inf/inf) ignored, 0 if none;
 *   bitwise_equal  1 iff every stored element is bit-identical;
 *   status         KB_STATUS_OK (KB_ERR_WORKSPACE, every other field zero,
 *                  when the call found its workspace not clean).
 * Counts, flags and maxima are exact; the two sums are binary64 sums in a
 * fixed order (deterministic from call to call, within 1e-6 relative of the
 * exact sums).  A rejected candidate has status = KB_REJECT_* and every
 * other field zero.
 *
 * With KB_FAIL_FAST a candidate that has a mismatch may be stopped early:
 * its record then describes only the elements that were compared, numel
 * being their count (<= the reference numel) and every other field the
 * definition above restricted to them (sum_sq_ref included); mismatches is
 * still >= 1, so the verdict is the same.  Which elements were compared
 * depends on timing.  A candidate without mismatch is always read in full:
 * its counts, flags and maxima equal those written without the flag, and its
 * two sums (and rel_l2) agree with them within 1e-6 relative -- the same
 * definition, summed over another split of the work, so not always the same
 * bits. */
typedef struct kb_stats {
    uint64_t numel;
    uint64_t mismatches;
    uint64_t nan_count;
    uint64_t pos_inf_count;
    uint64_t neg_inf_count;
    double sum_sq_diff;
    double sum_sq_ref;
    double rel_l2;
    float max_abs_err;
    float max_rel_err;
    int32_t bitwise_equal;
    int32_t status;
} kb_stats;

/* Verdict summary over the candidates of one call. */
typedef struct kb_summary {
    int32_t n_candidates;
    int32_t n_passed;     /* status OK and mismatches == 0: K(p) = 1 */
    int32_t n_rejected;   /* failed the policy gate */
    int32_t n_failed;     /* passed the gate, mismatches > 0 */
    int32_t first_passed; /* lowest index that passed, -1 if none */
    int32_t first_failed; /* lowest index rejected or failed, -1 if none */
} kb_summary;

/* Positions in one candidate (kb_screen_locate, or kb_screen_ex with
 * opts.d_loc): element indices in the flattened tensor, -1 where no element
 * qualifies.
 *   first_mismatch  smallest i that does not match;
 *   max_abs_index   smallest i with |fl(c_i - r_i)| == max_abs_err
 *                   (-1 when max_abs_err is 0);
 *   max_rel_index   smallest i with fl(|fl(c_i - r_i)| / |r_i|) == max_rel_err
 *                   (-1 when max_rel_err is 0);
 *   reserved        -1. */
typedef struct kb_locate {
    int64_t first_mismatch;
    int64_t max_abs_index;
    int64_t max_rel_index;
    int64_t reserved;
} kb_locate;

/* Launch configuration of a kb_screen call (reported, for measurement). */
typedef struct kb_launch {
    int32_t group_size;       /* candidates per work-group (KG) */
    int32_t n_groups;         /* candidate groups */
    int32_t blocks_per_group; /* work-groups per candidate group */
    int32_t threads;          /* threads per work-group */
    int64_t grid;             /* total work-groups */
} kb_launch;

/* ------------------------------------------------------------------ gate -- */

/* Policy gate V(p) of Section 3.2 restricted to what an output tensor shows:
 * for each candidate, status[k] = KB_STATUS_OK, or the first failing check in
 * the order NULL, DTYPE, SHAPE, LAYOUT.  Host only; launches nothing.
 *   ref, cands: host arrays of descriptors (cands has n_cands entries);
 *   status: host array of n_cands int32.
 * Errors: KB_ERR_INVALID_ARG (null arrays, n_cands < 0, ref ndim out of
 * range, ref data NULL with numel > 0), KB_ERR_DTYPE (reference dtype not
 * F32/F16/BF16). */
int kb_policy_check(const kb_tensor* ref, const kb_tensor* cands, int n_cands,
                    int32_t* status);

/* ---------------------------------------------------------------- screen -- */

/* Bytes of device workspace kb_screen needs for n_cands candidates of numel
 * elements of dtype (0 on invalid arguments).  A pure function of its
 * arguments (no device query). */
size_t kb_screen_workspace_bytes(int n_cands, uint64_t numel, int dtype);

/* Bytes of device workspace a kb_screen_ex call with positions (opts->d_loc)
 * needs: kb_screen_workspace_bytes plus the per-work-group position partials
 * (0 on invalid arguments).  Such a workspace serves calls with and without
 * positions for the same sizes. */
size_t kb_screen_positions_workspace_bytes(int n_cands, uint64_t numel, int dtype);

/* Zero-fill a workspace (a fill kernel, stream-ordered; no memset node, so
 * it may be captured in a graph).  A workspace must be zero-filled this way
 * (or otherwise) once after it is allocated, and again before it is used for
 * a call with other (n_cands, numel, dtype) or after anything else wrote to
 * it.  kb_screen keeps cross-work-group counters in it and leaves them zero
 * when the call completes, so consecutive calls with the same sizes need
 * nothing.  A call that finds a counter that did not begin at zero (the
 * contract broken, or a call cut short) does not trust it: the records of
 * the affected candidates get status KB_ERR_WORKSPACE, and kb_screen_stats,
 * kb_summarize and kb_summarize_multi then return KB_ERR_WORKSPACE, so a
 * dirty workspace gives an error, never wrong records (up to a 2^-32 chance
 * per counter that a leftover value passes the check).
 *   workspace: device, 16-byte aligned; workspace_bytes: multiple of 16.
 * Errors: KB_ERR_WORKSPACE, KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_screen_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The launch kb_screen would use for these sizes (KB_ERR_* on bad args). */
int kb_screen_launch(int n_cands, uint64_t numel, int dtype, kb_launch* out);

/* Screen n_cands candidate outputs against one reference output (Section 3.1
 * correctness indicator, Section 3.4 Verifier), stream-ordered on `stream`.
 *   ref          host descriptor of the reference; device data, contiguous,
 *                dtype F32, F16 or BF16;
 *   cands        host array of n_cands descriptors (n_cands >= 1); each is
 *                gated by kb_policy_check and, if accepted, read once;
 *   atol, rtol   finite, >= 0 (binary32);
 *   flags        0 or a combination of KB_EQUAL_NAN and KB_FAIL_FAST.
 *                KB_FAIL_FAST is the early-reject mode of the screening
 *                step (Section 3.3, Observation 2: a candidate with wrong
 *                output is to be turned away in milliseconds): every wave polls a per-candidate "failed"
 *                word in the workspace with each chunk it reads, a wave
 *                that finds a mismatch sets it, and a candidate known to
 *                have failed is no longer read (see kb_stats for what its
 *                record then holds); work-groups whose candidates have all
 *                failed stop reading the reference too;
 *   workspace    device scratch of workspace_bytes >=
 *                kb_screen_workspace_bytes(n_cands, numel, dtype),
 *                zero-filled as kb_screen_workspace_init describes; one
 *                workspace must not be used by two calls that can run
 *                concurrently;
 *   d_stats      n_cands kb_stats written by the kernel: device memory, or
 *                pinned host memory mapped for the device (hipHostMalloc),
 *                which lets a pipelined caller read the records without a
 *                copy once the stream has passed the call.
 * Candidate k's record goes to d_stats[k].  At most KB_INLINE_CANDS
 * candidates: the launch table travels in the kernel arguments; more need
 * kb_screen_ex with a host table.  Returns KB_OK once the work is enqueued.
 * Errors (nothing launched): KB_ERR_INVALID_ARG, KB_ERR_DTYPE,
 * KB_ERR_WORKSPACE (workspace too small, or more than KB_INLINE_CANDS
 * candidates), KB_ERR_ALIGNMENT (reference, accepted candidate, workspace or
 * d_stats not 16-byte aligned), KB_ERR_HIP. */
int kb_screen(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol,
              float rtol, uint32_t flags, void* workspace, size_t workspace_bytes,
              kb_stats* d_stats, hipStream_t stream);

/* Candidates whose launch table (16 bytes per candidate) travels in the
 * kernel arguments. */
#define KB_INLINE_CANDS 128

/* Options of kb_screen_ex (all-zero = none). */
typedef struct kb_screen_opts {
    /* Launch table of a call with more than KB_INLINE_CANDS candidates:
     * pinned host memory (hipHostMalloc, or a pinned torch tensor) owned by
     * the caller, 16-byte aligned, of host_table_bytes >=
     * kb_screen_host_table_bytes(n_cands).  The library writes the table
     * there during the call and the kernels read it from there, so the caller
     * leaves it untouched until the stream has passed the call (reusing it
     * earlier, e.g. for the next call, races).  Ignored for smaller calls. */
    void* host_table;
    size_t host_table_bytes;
    /* NULL, or n_cands kb_locate (device memory or mapped pinned host
     * memory, 16-byte aligned): the positions that kb_screen_locate would
     * find, found in the same pass over HBM as the records (the element-level
     * detail of a failed candidate's feedback, Section 3.4).  Not with
     * KB_FAIL_FAST.  Every position is the smallest qualifying element index,
     * so the result does not depend on the launch. */
    kb_locate* d_loc;
} kb_screen_opts;

/* Bytes of pinned host memory kb_screen_ex needs for n_cands candidates:
 * 0 for n_cands <= KB_INLINE_CANDS (and for n_cands < 1). */
size_t kb_screen_host_table_bytes(int n_cands);

/* kb_screen with options (opts may be NULL: then exactly kb_screen).
 * Errors as for kb_screen; KB_ERR_WORKSPACE also when a host table is needed
 * and missing or short, or when d_loc is given and the workspace is smaller
 * than kb_screen_positions_workspace_bytes; KB_ERR_ALIGNMENT when the host
 * table or d_loc is misaligned; KB_ERR_INVALID_ARG for d_loc with
 * KB_FAIL_FAST. */
int kb_screen_ex(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol,
                 float rtol, uint32_t flags, void* workspace, size_t workspace_bytes,
                 kb_stats* d_stats, const kb_screen_opts* opts, hipStream_t stream);

/* Bytes of the fixed device scratch of kb_screen_noalloc (enough for any call
 * with at most KB_INLINE_CANDS candidates). */
#define KB_NOALLOC_SCRATCH_BYTES (16u << 20)

/* kb_screen for callers that cannot allocate device memory -- code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  The
 * same screen and records as kb_screen (the same kernels and launch), with
 * the workspace replaced by a fixed scratch array in the library: this call
 * allocates nothing (no hipMalloc, no hipFree, no allocating library routine)
 * and needs no workspace argument.
 *   ref, cands, n_cands, atol, rtol, flags, d_stats, stream   as for kb_screen;
 *   n_cands <= KB_INLINE_CANDS, and the call's workspace size
 *   (kb_screen_workspace_bytes) at most KB_NOALLOC_SCRATCH_BYTES, which holds
 *   for every such call.
 * Scratch: KB_NOALLOC_SCRATCH_BYTES of device memory per device, held from
 * the first call on that device until the process ends; its address is
 * looked up on that first call (with the device current).  Every call on a
 * device shares that device's scratch and leaves its contents there; each
 * call first zero-fills the part that must begin at zero (one small fill
 * kernel on `stream`).  So two calls that can overlap on one device -- on
 * two streams, or from two threads -- race and give wrong records; calls on
 * different devices do not interfere.
 * Errors (nothing launched): as for kb_screen, KB_ERR_INVALID_ARG for more
 * than KB_INLINE_CANDS candidates or a device index beyond 63, KB_ERR_WORKSPACE
 * when the call would need more scratch, KB_ERR_HIP. */
int kb_screen_noalloc(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol,
                      float rtol, uint32_t flags, kb_stats* d_stats, hipStream_t stream);

/* The verdict of each of n_cands records already in host memory (host only):
 * candidate k passes -- K(p) = 1 for its output -- iff status is
 * KB_STATUS_OK and mismatches is 0 (Section 3.1's correctness indicator;
 * Algorithm 1 rejects a candidate that fails the policy check or the
 * Verifier's test).  passed: optional host array of n_cands flags (1 =
 * passed); summary: optional counts.  Errors: KB_ERR_INVALID_ARG,
 * KB_ERR_WORKSPACE (a record has that status: see kb_screen_workspace_init). */
int kb_summarize(const kb_stats* h_stats, int n_cands, kb_summary* summary, int32_t* passed);

/* Copy n_cands records from device d_stats to host h_stats (may be NULL),
 * synchronize `stream`, and give the verdicts of kb_summarize in *summary
 * and passed[] (each may be NULL).  This is the readback and verdict step of
 * Algorithm 1's reject-on-failure gates.  Errors: KB_ERR_INVALID_ARG,
 * KB_ERR_HIP, KB_ERR_WORKSPACE (the call that wrote the records found its
 * workspace not clean; see kb_screen_workspace_init). */
int kb_screen_stats(const kb_stats* d_stats, int n_cands, kb_stats* h_stats,
                    kb_summary* summary, int32_t* passed, hipStream_t stream);

/* Positions of the first mismatch and of the maxima of each candidate: the
 * element-level detail that the feedback about a failed candidate carries
 * (Section 3.4: the check's log is passed on to the next generation step).
 * A second, optional pass over the same buffers, stream-ordered after the
 * kb_screen call whose records it uses.
 *   ref, cands, n_cands, atol, rtol, flags   as given to kb_screen;
 *   stats    the n_cands records kb_screen wrote for them (device memory or
 *            mapped pinned host memory; read by the kernel);
 *   d_loc    n_cands kb_locate written by the kernels (device memory or
 *            mapped pinned host memory), 16-byte aligned.
 * KB_FAIL_FAST in flags is accepted and has no effect here; where a record
 * was written under it for a stopped candidate, the max indices refer to the
 * maxima that record holds.
 * Rejected candidates get -1 everywhere.  A wave stops scanning for a
 * position once it has found one (later elements have larger indices), so a
 * candidate with an early mismatch costs little.  No workspace is needed.
 * Errors (nothing launched): KB_ERR_INVALID_ARG, KB_ERR_DTYPE,
 * KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_screen_locate(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol,
                     float rtol, uint32_t flags, const kb_stats* stats, kb_locate* d_loc,
                     hipStream_t stream);

/* ---------------------------------------------------------- multi-output -- */

/* Most outputs per candidate kb_screen_multi takes. */
#define KB_MAX_OUTPUTS 64

/* Bytes of device workspace kb_screen_multi needs (0 on invalid arguments):
 * the sum, over outputs, of kb_screen_workspace_bytes for that output's
 * reference, each rounded up to 256.  Zero-filled as for kb_screen. */
size_t kb_screen_multi_workspace_bytes(const kb_tensor* refs, int n_outputs, int n_cands);

/* Bytes of pinned host table kb_screen_multi needs: n_outputs times
 * kb_screen_host_table_bytes(n_cands) (each output has its own table). */
size_t kb_screen_multi_host_table_bytes(int n_outputs, int n_cands);

/* Screen candidates whose output is a tuple of n_outputs tensors against a
 * tuple of references (a kernel returning several tensors: the
 * correctness indicator K(p) of Section 3.1 then needs all of them, and the
 * policy check of Section 3.2 covers each output's shape and dtype).
 *   refs        host array of n_outputs reference descriptors (as for
 *               kb_screen; outputs may differ in dtype and shape);
 *   cands       host array [n_cands][n_outputs] of descriptors, candidate-
 *               major;
 *   atol, rtol  host arrays of n_outputs tolerances;
 *   flags       as for kb_screen, applied to every output;
 *   d_stats     n_outputs * n_cands records, output-major: output o of
 *               candidate k at d_stats[o * n_cands + k];
 *   opts        as for kb_screen_ex (may be NULL; d_loc must be NULL); a host
 *               table must hold kb_screen_multi_host_table_bytes(n_outputs,
 *               n_cands).
 * One gate over all outputs: candidate k is accepted only if every output
 * passes kb_policy_check against its reference; otherwise no output of it
 * is read and every one of its records has status = the first failing check
 * of the first failing output (in output order).  Accepted candidates get
 * the kb_screen record of each output.  The outputs are screened one after
 * another on `stream`.  Errors (nothing launched) as for kb_screen. */
int kb_screen_multi(const kb_tensor* refs, int n_outputs, const kb_tensor* cands, int n_cands,
                    const float* atol, const float* rtol, uint32_t flags, void* workspace,
                    size_t workspace_bytes, kb_stats* d_stats, const kb_screen_opts* opts,
                    hipStream_t stream);

/* Verdict over multi-output records in host memory (output-major, as
 * kb_screen_multi writes them): a candidate passes iff every output has
 * status OK and no mismatch; it counts as rejected if any output was
 * rejected, else as failed.  passed: optional host array of n_cands flags. */
int kb_summarize_multi(const kb_stats* h_stats, int n_outputs, int n_cands, kb_summary* summary,
                       int32_t* passed);

/* ------------------------------------------------------------------ rung -- */

/* Longest row of timing samples kb_rung_stats takes. */
#define KB_RUNG_MAX_ITER 4096

/* Statistics of one (candidate, shape) row of timing samples, 80 bytes.
 *   mean_us          (t_1 + ... + t_n) / n, the sum left to right in binary64
 *                    (Appendix A.5: the mean time per shape);
 *   pXX_us           the XX-th percentile: linear interpolation between the
 *                    order statistics around position h = (n - 1) XX/100,
 *                    counted from 0: x[k] + (h - k)(x[k+1] - x[k]),
 *                    k = floor(h), each operation rounded once;
 *   pXX_over_p50     the tail ratios of Table A.3;
 *   speedup_vs_base  the baseline's mean for the same shape / mean_us
 *                    (Appendix A.5), NaN without a baseline;
 *   n_samples        n;
 *   valid            1 iff every sample is finite and > 0 (else every
 *                    double field is NaN). */
typedef struct kb_sample_stats {
    double mean_us;
    double p50_us, p90_us, p95_us, p99_us;
    double p90_over_p50, p95_over_p50, p99_over_p50;
    double speedup_vs_base;
    int32_t n_samples;
    int32_t valid;
} kb_sample_stats;

/* One candidate at one rung, 32 bytes.
 *   latency_us       the mean over the rung's shapes of the row means, left
 *                    to right (Eq. 1's expectation over shapes, the shapes
 *                    weighted equally);
 *   score            S = 1e6 / max(1, latency_us) + (alpha rung + beta budget)
 *                    (Eq. 2 with gamma(r) = alpha r + beta b_r, Section 3.1:
 *                    the rung term summed first, then added); -inf for an
 *                    invalid candidate;
 *   speedup_vs_base  the baseline's latency / latency_us;
 *   valid            1 iff all the candidate's rows are valid. */
typedef struct kb_rung_score {
    double latency_us;
    double score;
    double speedup_vs_base;
    int32_t valid;
    int32_t reserved;
} kb_rung_score;

/* The rung benchmarker's statistics (Sections 3.1-3.2, Appendices A.2 and
 * A.5), stream-ordered on `stream`:
 *   samples   device, [n_cands][n_shapes][n_iter] timing samples in us
 *             (binary64, 8-byte aligned), one row per (candidate, shape);
 *   n_iter    timed iterations per row, 1..KB_RUNG_MAX_ITER;
 *   base      the baseline candidate's index, or -1 for none;
 *   rung      r >= 0; budget: b_r (finite, >= 0; the caller's unit, e.g. the
 *             rung's repeat count); alpha, beta: finite (the paper uses 0.02
 *             and 0.01);
 *   rows      device, n_cands * n_shapes kb_sample_stats (8-byte aligned);
 *   scores    device, n_cands kb_rung_score (8-byte aligned).
 * Every field is the definition's value to the last bit.  No workspace.
 * Errors (nothing launched): KB_ERR_INVALID_ARG, KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_rung_stats(const double* samples, int n_cands, int n_shapes, int n_iter, int base, int rung,
                  double budget, double alpha, double beta, kb_sample_stats* rows,
                  kb_rung_score* scores, hipStream_t stream);

/* The promotion decision D of Section 3.4 (Algorithm 1's promote-or-prune
 * step) over one rung's candidates, stream-ordered on `stream`:
 *   scores    device, n_cands kb_rung_score (as kb_rung_stats writes them);
 *             the ranking key is `score` for a valid candidate and -inf for
 *             an invalid one or a NaN score;
 *   base      the baseline's index, or -1 for none;
 *   frac_num / frac_den   the promoted fraction, 0 <= num <= den, den >= 1;
 *   rank      device, n_cands int32: candidate i's position, 0 = best;
 *             higher keys first, equal keys by the lower index (the
 *             deterministic tie-break);
 *   order     device, n_cands int32: the candidate at each position;
 *   promoted  device, n_cands int32: 1 for the first
 *             ceil(n_eligible frac_num / frac_den) valid non-baseline
 *             candidates in rank order (n_eligible = their count, computed
 *             in integers) and for a valid baseline, which is always
 *             carried to the next rung (Fig. 4 shows the baseline promoted
 *             beside the top candidates at every rung); 0 for the pruned.
 * All arrays 4-byte aligned (scores 8).  n_cands <= KB_PROMOTE_MAX.
 * Errors (nothing launched): KB_ERR_INVALID_ARG, KB_ERR_ALIGNMENT, KB_ERR_HIP. */
#define KB_PROMOTE_MAX 65536
int kb_rung_promote(const kb_rung_score* scores, int n_cands, int base, int frac_num, int frac_den,
                    int32_t* rank, int32_t* order, int32_t* promoted, hipStream_t stream);

/* Per-rung survival, the columns of Table A.1 (host only, no device work):
 *   fail_pct[r]  = 100 failed[r] / entering[r] (0 when nothing entered);
 *   promo_pct[r] = 100 promoted[r] / original (the initial pool, baseline
 *                  included).
 * Errors: KB_ERR_INVALID_ARG (null arrays, n_rungs < 1, original < 1, a
 * negative count, failed > entering). */
int kb_rung_survival(const int32_t* entering, const int32_t* failed, const int32_t* promoted,
                     int n_rungs, int original, double* fail_pct, double* promo_pct);

/* ------------------------------------------------------------- generator -- */

/* Fill device dst[0..n) with elements offset .. offset+n-1 of the seeded
 * stream (seed, stream_id, sub):
 *   Philox4x32-10 block b has key (lo32(seed), hi32(seed)) and counter
 *   (lo32(b), hi32(b), sub, stream_id); element g is word g mod 4 of block
 *   g / 4.  So any element can be regenerated on its own (random access), and
 *   disjoint (stream_id, sub) pairs give independent streams.
 *   KB_DIST_U32      dtype KB_U32: the word itself;
 *   KB_DIST_UNIFORM  u = (x >> 8) * 2^-24 in [0, 1), value fmaf(u, p1 - p0, p0)
 *                    with p1 - p0 rounded to binary32 (a value in [p0, p1]);
 *   KB_DIST_NORMAL   Box-Muller on the word pair of g's half-block (words 0,1
 *                    or 2,3): u1 = (x_a + 1) 2^-32, u2 = x_b 2^-32,
 *                    z = sqrt(-2 ln u1) * (cos or sin)(2 pi u2) in binary64
 *                    (cosine for even g, sine for odd g), rounded to
 *                    binary32; value fmaf(z, p1, p0) (mean p0, std dev p1);
 *   KB_DIST_STUDENT_T3  Student's t with 3 degrees of freedom from all four
 *                    words of block g (not g / 4): the binary64 normals z0,
 *                    z1 of words 0, 1 and z2, z3 of words 2, 3 (as above,
 *                    unrounded), t = z0 / sqrt(((z1^2 + z2^2) + z3^2) / 3) in
 *                    binary64, rounded to binary32; value fmaf(t, p1, p0).
 *                    A heavy-tailed output (its fourth moment is infinite).
 *   F16 / BF16 dtypes round the binary32 value to nearest even.
 * dst: device, 16-byte aligned.  Errors: KB_ERR_INVALID_ARG (null dst with
 * n > 0, non-finite p0/p1), KB_ERR_DTYPE (U32 with a float distribution or
 * the reverse), KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_gen_inputs(void* dst, int dtype, uint64_t n, int dist, float p0, float p1,
                  uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset,
                  hipStream_t stream);

/* ------------------------------------------------- derived seeded inputs --
 * The synthetic outputs a screen is measured on, built from the same stream:
 * a reference and candidates with planted differences (the Verifier checks
 * a candidate's output against the reference's on seeded inputs, Sections
 * 3.1 and 3.4).  All stream-ordered on `stream`, device buffers 16-byte
 * aligned, nothing launched on error. */

/* Rows of softmax probabilities: dst is a [rows][cols] binary32 tensor (dtype
 * KB_F32 only); its logits are the NORMAL stream with mean 0 and standard
 * deviation sigma (logit (i, j) is element i cols + j of kb_gen_inputs(F32,
 * NORMAL, 0, sigma)), and each row is, in binary64, m = max x,
 * p_j = exp(x_j - m) / sum_k exp(x_k - m), rounded once to binary32.  The
 * binary64 row sum is a fixed tree (the same bits on every call; within
 * rounding of a left-to-right sum).  Every p_j > 0 unless it underflows.
 * Errors: KB_ERR_INVALID_ARG (cols = 0 with rows > 0, null dst, sigma not
 * finite), KB_ERR_DTYPE, KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_gen_softmax_rows(void* dst, int dtype, uint64_t rows, uint64_t cols, float sigma,
                        uint64_t seed, uint32_t stream_id, uint32_t sub, hipStream_t stream);

/* Most indices kb_gen_indices draws. */
#define KB_MAX_INDICES 4096

/* m distinct element indices in [0, n), in draw order, to device dst[0..m)
 * (uint64): draw j = 0, 1, 2, ... is ((w1 << 32) | w0) mod n of block j of
 * the stream (seed, stream_id, sub); a draw equal to an earlier one is
 * skipped.  Requires 1 <= m <= KB_MAX_INDICES and 2 m <= n (each draw is then
 * new with probability at least 1/2; a draw count cap of 2^20, never reached
 * in practice, bounds the kernel, and entries it did not fill would be
 * UINT64_MAX).  Errors: KB_ERR_INVALID_ARG, KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_gen_indices(uint64_t* dst, uint32_t m, uint64_t n, uint64_t seed, uint32_t stream_id,
                   uint32_t sub, hipStream_t stream);

/* Planted changes (kb_gen_perturb ops).  x is src[j] widened to binary32 and
 * "narrow" rounds a binary32 value to the dtype (nearest even); a NaN result
 * is stored as the dtype's positive quiet NaN (0x7FC00000, 0x7E00, 0x7FC0),
 * whatever NaN the arithmetic produced.  For element g = offset + j: u(g) is
 * kb_gen_inputs(UNIFORM, 0, 1) element g, U(g) the UNIFORM [a, b) element g,
 * N(g) the NORMAL element g with mean 0 and standard deviation a; ops 6 and 7
 * take the four words w0..w3 of block g and the dtype KB_F32 only, and
 * u01(w) = (w >> 8) 2^-24. */
enum {
    KB_PERTURB_ADD_UNIFORM = 1,      /* narrow(x + U(g)) */
    KB_PERTURB_REL_UNIFORM = 2,      /* narrow(fmaf(x, U(g), x)): relative noise, one rounding */
    KB_PERTURB_ADD_NORMAL = 3,       /* narrow(x + N(g)) */
    KB_PERTURB_SCALE_WHERE = 4,      /* u(g) < p ? narrow(x * a) : src[j] */
    KB_PERTURB_FLIP_LSB_WHERE = 5,   /* u(g) < p ? storage bits ^ 1 : src[j] */
    KB_PERTURB_SPECIALS = 6,         /* v = u01(w0), sign = top bit of w1: v < a: the subnormal
                                        with mantissa (w2 & 0x7FFFFF) | 1; else v < b: zero; else
                                        v < p: infinity; else src[j] (a <= b <= p cumulative) */
    KB_PERTURB_ZERO_SUBNORMAL_REL = 7 /* v = u01(w0), d = the [a, b) value of w1: v < p: a zero
                                         flips its sign, a subnormal becomes the zero of its sign,
                                         a finite normal x becomes fmaf(x, d, x), an infinity or
                                         NaN stays; else src[j] */
};

/* dst[j] = op(src[j]) for j < n (dst may equal src; dtype F32, F16 or BF16).
 * Errors: KB_ERR_INVALID_ARG (unknown op, a, b or p not finite, null
 * pointers with n > 0, offset + n overflowing), KB_ERR_DTYPE (ops 6-7 on a
 * 16-bit dtype), KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_gen_perturb(void* dst, const void* src, int dtype, uint64_t n, int op, float a, float b,
                   float p, uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset,
                   hipStream_t stream);

/* Scatter modes. */
enum {
    KB_SCATTER_NAN = 1,             /* the dtype's quiet NaN: 0x7FC00000, 0x7E00 (f16), 0x7FC0 (bf16) */
    KB_SCATTER_INF_SIGN_OF_REF = 2  /* the infinity with the sign bit of ref[idx] */
};

/* For i < m: dst[idx[i]] = the mode's value (an index >= n is skipped).
 * dst, ref: device tensors of n elements of dtype; idx: device uint64[m].
 * Errors: KB_ERR_INVALID_ARG, KB_ERR_DTYPE, KB_ERR_ALIGNMENT, KB_ERR_HIP. */
int kb_gen_scatter(void* dst, const void* ref, int dtype, uint64_t n, const uint64_t* idx, uint32_t m,
                   int mode, hipStream_t stream);

/* ----------------------------------------------------------------- misc -- */

/* Text of the last error on the calling thread (empty if none); valid until
 * the next kb_* call on this thread. */
const char* kb_last_error(void);

/* Interface version: major * 10000 + minor * 100 + patch. */
int kb_version(void);

#ifdef __cplusplus
}
#endif
#endif /* KB_H */
