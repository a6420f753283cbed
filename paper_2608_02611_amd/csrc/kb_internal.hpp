// kb_internal.hpp -- declarations shared by the library's translation units
// (host side): kernel launchers and the screening launch plan.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/kb.h"

namespace kb {

// One entry of the launch table.  The table holds the accepted candidates
// in call order, then the rejected candidates: one entry per candidate.  (The
// last candidate group is padded inside the kernel with the reference, which
// it compares but writes no record for.)
struct CandEntry {
    const void* data;  // device pointer (NULL for rejected entries)
    int32_t index;     // position in the caller's candidate array, -1 for padding
    int32_t status;    // KB_STATUS_OK or KB_REJECT_*
};

// Per-(work-group, candidate) partial statistics, kept as arrays of fields so
// that the finishing work-group reads them coalesced.
enum PartField : int {
    PF_MISM = 0,
    PF_NAN,
    PF_PINF,
    PF_NINF,
    PF_MAXABS,
    PF_MAXREL,
    PF_BITDIFF,
    PF_COUNT
};
// Fail-fast launches keep one more plane: elements compared.
constexpr int PF_NREAD = PF_COUNT;
constexpr int kPartPlanes = PF_COUNT + 1;

// Work split and workspace layout of one kb_screen call.
struct ScreenPlan {
    int dtype;
    int n_cands;          // all candidates
    int n_acc;            // candidates that passed the policy gate
    int kg;               // candidates per candidate group (kernel template)
    int n_groups;         // ceil(n_acc / kg)
    int blocks_per_group; // stripes: a multiple of 8 (XCD count)
    int threads;
    uint64_t numel;
    uint64_t n_vec;       // full 16-byte vectors per tensor
    int n_super;          // ceil(blocks_per_group / 16): first-level combine groups
    int ff_round;         // fail-fast launch: candidate groups per round
    int wide;             // launch the 5-waves-per-SIMD build (use_wide_kernel)
    // workspace byte offsets; core_total ends what every call uses, total
    // adds the position-search partials (calls with positions only)
    size_t off_tickets1, off_tickets2, off_ff_flags, off_table, off_part_u32, off_part_ssd,
        off_part_ssr, off_part_ssrc, off_part2, off_part2_ssr, core_total, off_part_idx, off_part2_idx, total;
};

// Position-search partials: per (work-group, candidate), the smallest
// mismatching element index, and the smallest element index at which the
// max abs error and the max rel error are reached (all ones: none).
enum IdxField : int { IX_FIRST_MISMATCH = 0, IX_MAX_ABS, IX_MAX_REL, IX_COUNT };
struct Part2Idx {
    uint64_t ix[IX_COUNT];
};

// Second-level partial of one candidate: the combine of up to 16 work-groups.
struct Part2 {
    uint64_t mism, nan, pinf, ninf;
    uint32_t maxabs, maxrel, bitdiff, pad;
    double ssd;
    uint64_t nread;  // fail-fast only: elements compared
    double ssr;      // fail-fast only: the candidate's own sum of r^2
};

// Launch geometry and workspace layout.  The layout depends only on
// (n_cands, numel, dtype); resident_blocks (work-groups of the chosen kernel
// that fit on the device at once, 0 if unknown) sizes the launch, and
// serial_groups selects the fail-fast geometry (the groups one after
// another, each over the whole device).
bool make_plan(int n_cands, int n_acc, uint64_t numel, int dtype, int resident_blocks,
               bool serial_groups, ScreenPlan* plan);

// Candidates per group the plan picks for n_cands candidates.
int plan_group_size(int n_cands, int dtype);

// Whether a plain launch takes the screening kernel built for 5 waves per
// SIMD (fp32, 4 candidates per group, at least 2^22 elements).  fp32 at 4
// candidates needs 99 VGPRs, which allocate as 104: 4 waves per SIMD.  Built
// for 5 it fits 96 with a 16-byte spill.  Measured: 12% faster on 2^30 fp32
// elements per tensor; 5% slower on 2^18 elements (1024 candidates), whose
// 2048 work-groups make two whole rounds at 4 per CU but not at 5.
constexpr uint64_t kWideMinNumel = 1ull << 22;
inline bool use_wide_kernel(int dtype, int kg, bool fail_fast, uint64_t numel, bool loc = false) {
    return dtype == KB_F32 && kg == 4 && !fail_fast && !loc && numel >= kWideMinNumel;
}

// Work-groups of the screening kernel for (dtype, kg, fail-fast, wide,
// positions) resident per CU (occupancy query, cached), or 0 on failure.
int screen_blocks_per_cu(int dtype, int kg, bool fail_fast, bool wide = false, bool loc = false);

// Candidate groups per round of a fail-fast launch (see make_plan).
constexpr int kFailFastRound = 2;

// Launch tables of up to this many candidates travel in the kernel
// arguments; larger ones are read from the caller's pinned host memory.
constexpr int kInlineCands = 128;

struct InlineTable {
    CandEntry e[kInlineCands];
};

// Device-side parameters of the screening kernel.
struct ScreenParams {
    const void* ref;
    const CandEntry* table;
    uint64_t numel;
    uint64_t n_vec;
    float atol;
    float rtol;
    uint32_t flags;
    int n_acc;
    int n_cands;
    int n_table;         // table entries: the accepted, then the rejected candidates
    int rej_start;       // first rejected entry (n_acc)
    int table_inline;    // 1: the table is the kernel argument, 0: p.table (host memory)
    int n_groups;
    int blocks_per_group;
    int n_super;
    int ff_round;        // fail-fast: candidate groups per round of the grid
    uint32_t tag;        // this call's tag (nonzero): marks its tickets and fail-fast words
    uint64_t* tickets1;  // [n_groups][n_super] tagged tickets: (tag << 32) | arrivals
    uint64_t* tickets2;  // [n_groups]
    uint32_t* ff_flags;  // fail-fast words: [n_groups * KG][1 + n_super] lines of 32 words
    uint32_t* part_u32;  // [kPartPlanes][n_acc][blocks_per_group]
    double* part_ssd;    // [n_acc][blocks_per_group]
    double* part_ssr;    // [n_groups][blocks_per_group]
    double* part_ssrc;   // fail-fast: [n_acc][blocks_per_group] per-candidate sums of r^2
    Part2* part2;        // [n_acc][n_super]
    double* part2_ssr;   // [n_groups][n_super]
    uint64_t* part_idx;  // positions: [IX_COUNT][n_acc][blocks_per_group]
    Part2Idx* part2_idx; // positions: [n_acc][n_super]
    kb_stats* stats;     // caller's records, indexed by CandEntry::index
    kb_locate* loc;      // positions launch: the caller's positions, indexed like stats
};

// tab: the launch table when it is inline (n_cands <= kInlineCands), else
// ignored (p.table points at the caller's copy).  fail_fast selects the
// early-reject variant of the kernel, loc the variant that also finds the
// positions (p.loc); never both.
hipError_t launch_screen(const ScreenPlan& plan, const ScreenParams& p, const InlineTable& tab,
                         bool fail_fast, bool loc, hipStream_t stream);
// Zero-fill n bytes of device memory (workspace initialisation).
hipError_t launch_zero_fill(void* dst, size_t n, hipStream_t stream);
// Records for calls with no element to read (numel == 0 or no accepted
// candidate): every record written from the table alone (and, with loc,
// every position -1).
hipError_t launch_records_only(const CandEntry* table, const InlineTable& tab, int table_inline,
                               int n_table, uint64_t numel, kb_stats* stats, kb_locate* loc,
                               hipStream_t stream);

// Position search (kb_screen_locate): up to kLocateBatch candidates per
// launch, their table in the kernel arguments.
constexpr int kLocateBatch = 128;
struct LocEntry {
    const void* data;
    int32_t index;  // position in the caller's candidate array
    int32_t pad;
};
struct LocTable {
    LocEntry e[kLocateBatch];
};
struct LocateParams {
    const void* ref;
    uint64_t numel;
    float atol;
    float rtol;
    uint32_t flags;
    int n;        // candidates in this launch
    int stripes;  // work-groups per candidate
    const kb_stats* stats;
    kb_locate* out;
};
hipError_t launch_locate(int dtype, const LocateParams& p, const LocTable& tab, hipStream_t stream);
// Work-groups of the position-search kernel for dtype resident per CU
// (occupancy query, cached), or 0 on failure.
int locate_blocks_per_cu(int dtype);
// Fill n_words 32-bit words with value.
hipError_t launch_fill_u32(void* dst, uint64_t n_words, uint32_t value, hipStream_t stream);

hipError_t launch_gen(void* dst, int dtype, uint64_t n, int dist, float p0, float p1,
                      uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset,
                      hipStream_t stream);
// Derived seeded inputs (kb_gen.hip); arguments validated by the caller.
hipError_t launch_gen_t3(void* dst, int dtype, uint64_t n, float p0, float p1, uint64_t seed,
                         uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream);
hipError_t launch_softmax_rows(float* dst, uint64_t rows, uint64_t cols, float sigma, uint64_t seed,
                               uint32_t stream_id, uint32_t sub, hipStream_t stream);
hipError_t launch_indices(uint64_t* dst, uint32_t m, uint64_t n, uint64_t seed, uint32_t stream_id,
                          uint32_t sub, hipStream_t stream);
hipError_t launch_perturb(void* dst, const void* src, int dtype, uint64_t n, int op, float a, float b,
                          float p, uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset,
                          hipStream_t stream);
hipError_t launch_scatter(void* dst, const void* ref, int dtype, uint64_t n, const uint64_t* idx,
                          uint32_t m, int mode, hipStream_t stream);

}  // namespace kb
