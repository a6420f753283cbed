// kb_internal.hpp -- declarations shared by the library's translation units
// (host side): kernel launchers and the screening launch plan.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/kb.h"

namespace kb {

// One entry of the candidate table uploaded to the workspace: accepted
// candidates first (in call order), then rejected ones.
struct CandEntry {
    const void* data;  // device pointer (NULL for rejected entries)
    int32_t index;     // position in the caller's candidate array
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

// Work split and workspace layout of one kb_screen call.
struct ScreenPlan {
    int dtype;
    int n_cands;          // all candidates
    int n_acc;            // candidates that passed the policy gate
    int kg;               // candidates per candidate group (kernel template)
    int n_groups;         // ceil(n_acc / kg)
    int blocks_per_group; // multiple of 8 (XCD count)
    int threads;
    uint64_t numel;
    uint64_t n_vec;       // full 16-byte vectors per tensor
    // workspace byte offsets
    size_t off_tickets, off_table, off_part_u32, off_part_ssd, off_part_ssr, total;
};

// Launch geometry and workspace layout for (n_cands candidates, all accepted).
bool make_plan(int n_cands, int n_acc, uint64_t numel, int dtype, ScreenPlan* plan);

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
    int n_groups;
    int blocks_per_group;
    uint32_t* tickets;
    uint32_t* part_u32;  // [PF_COUNT][n_acc][blocks_per_group]
    double* part_ssd;    // [n_acc][blocks_per_group]
    double* part_ssr;    // [n_groups][blocks_per_group]
    kb_stats* stats;     // caller's records, indexed by CandEntry::index
};

hipError_t launch_screen(const ScreenPlan& plan, const ScreenParams& p, hipStream_t stream);
// Records for calls with no element to read (numel == 0 or no accepted
// candidate): every record written from the table alone.
hipError_t launch_records_only(const CandEntry* table, int n_cands, uint64_t numel,
                               kb_stats* stats, hipStream_t stream);

hipError_t launch_gen(void* dst, int dtype, uint64_t n, int dist, float p0, float p1,
                      uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset,
                      hipStream_t stream);

}  // namespace kb
