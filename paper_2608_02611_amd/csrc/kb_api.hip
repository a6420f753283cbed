// kb_api.hip -- host side of the C interface (include/kb.h): argument
// validation, the policy gate, launch planning and the statistics readback.
#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdlib>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <vector>

#include "kb_device.hpp"
#include "kb_internal.hpp"
#include "kb_rung.hpp"

// Fixed device scratch of kb_screen_noalloc: a workspace for callers that
// cannot allocate.  Each device that runs the library holds its own copy
// until the process ends.  Host code never uses this name as an address:
// kb::noalloc_scratch() asks the runtime for the copy on the current device.
static __device__ __align__(256) unsigned char scratch[KB_NOALLOC_SCRATCH_BYTES];

namespace kb {
namespace {

// The last error of the calling thread, a fixed buffer (setting it allocates
// nothing).
thread_local char g_error[512];

void clear_error() { g_error[0] = '\0'; }

int fail(int code, const char* fmt, ...) {
    char buf[sizeof g_error];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    std::memcpy(g_error, buf, sizeof g_error);
    return code;
}

int fail_hip(hipError_t e, const char* what) {
    return fail(KB_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool is_float_dtype(int dt) { return dt == DT_F32 || dt == DT_F16 || dt == DT_BF16; }
size_t elem_size(int dt) { return dt == DT_F32 || dt == DT_U32 ? 4 : 2; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

uint64_t tensor_numel(const kb_tensor& t) {
    uint64_t n = 1;
    for (int i = 0; i < t.ndim; ++i) n *= (uint64_t)t.shape[i];
    return n;
}

bool shape_valid(const kb_tensor& t) {
    if (t.ndim < 0 || t.ndim > KB_MAX_DIMS) return false;
    for (int i = 0; i < t.ndim; ++i)
        if (t.shape[i] < 0) return false;
    return true;
}

// Dense row-major: the stride of every dimension of size > 1 is the product
// of the sizes after it.
bool is_contiguous(const kb_tensor& t) {
    if (tensor_numel(t) == 0) return true;
    int64_t expect = 1;
    for (int i = t.ndim - 1; i >= 0; --i) {
        if (t.shape[i] != 1 && t.strides[i] != expect) return false;
        expect *= t.shape[i];
    }
    return true;
}

int32_t gate_one(const kb_tensor& ref, const kb_tensor& c) {
    // NULL data is a missing output, unless the candidate is a valid empty tensor
    if (c.data == nullptr && !(shape_valid(c) && tensor_numel(c) == 0)) return KB_REJECT_NULL;
    if (c.dtype != ref.dtype) return KB_REJECT_DTYPE;
    if (!shape_valid(c) || c.ndim != ref.ndim) return KB_REJECT_SHAPE;
    for (int i = 0; i < ref.ndim; ++i)
        if (c.shape[i] != ref.shape[i]) return KB_REJECT_SHAPE;
    if (!is_contiguous(c)) return KB_REJECT_LAYOUT;
    return KB_STATUS_OK;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Launch tuning override for measurement sweeps: KB_SCREEN_TUNE="kg=16,blocks=1024"
// caps the candidates per group (1, 2, 4, 8 or 16) and sets the target total
// number of work-groups; "ffround=N" sets the fail-fast groups per round.
// Read once per process; unset (the normal case), the built-in choice
// applies.
struct Tuning {
    int kg_cap = 0, blocks_total = 0, ff_round = 0;  // 0 = not overridden
};

const Tuning& tuning() {
    static const Tuning t = [] {
        Tuning r;
        const char* s = std::getenv("KB_SCREEN_TUNE");
        if (s == nullptr) return r;
        int v;
        const char* k = std::strstr(s, "kg=");
        if (k && std::sscanf(k + 3, "%d", &v) == 1 && (v == 1 || v == 2 || v == 4 || v == 8 || v == 16))
            r.kg_cap = v;
        const char* b = std::strstr(s, "blocks=");
        if (b && std::sscanf(b + 7, "%d", &v) == 1 && v >= 8 && v <= (1 << 20)) r.blocks_total = v;
        const char* f = std::strstr(s, "ffround=");
        if (f && std::sscanf(f + 8, "%d", &v) == 1 && v >= 1) r.ff_round = v;
        return r;
    }();
    return t;
}

// A tag for one screening call: odd (the self-checking tickets need it), and
// in practice different from any value a workspace word holds unless this
// call wrote it (the kernel marks its tickets and fail-fast words with it; see
// the kernel).  Derived from the monotonic clock, so the library keeps no
// state for it.
uint32_t call_tag() {
    uint64_t x = (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
    // MurmurHash3's 64-bit finalizer: every input bit reaches every output bit
    x ^= x >> 33;
    x *= 0xFF51AFD7ED558CCDull;
    x ^= x >> 33;
    x *= 0xC4CEB9FE1A85EC53ull;
    x ^= x >> 33;
    return ((uint32_t)x ^ (uint32_t)(x >> 32)) | 1u;
}

// Address of `scratch` on each device, looked up once per device (with that
// device current) and kept for the process.
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];

// The scratch's address on device `dev` (the current device), in *out;
// KB_OK or an error code.
int noalloc_scratch(int dev, void** out) {
    if (dev < 0 || dev >= kMaxDevices)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_noalloc: device %d beyond the %d the library tracks",
                    dev, kMaxDevices);
    void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return fail(KB_ERR_HIP, "kb_screen_noalloc: hipGetSymbolAddress(scratch): %s",
                        hipGetErrorString(e));
        g_scratch_addr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return KB_OK;
}

// A record that a kernel wrote with status KB_ERR_WORKSPACE: the call found
// a ticket word of its workspace that did not begin at zero.
int dirty_workspace_error(const kb_stats* st, int n) {
    for (int k = 0; k < n; ++k)
        if (st[k].status == KB_ERR_WORKSPACE)
            return fail(KB_ERR_WORKSPACE,
                        "candidate %d: the screening call found its workspace not clean (zero-fill it "
                        "with kb_screen_workspace_init after allocating it and before using it for other "
                        "sizes); the records of that call are not valid", k);
    return KB_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// Launch plan.
// ---------------------------------------------------------------------------

// Work-groups of the screening kernel for (dtype, kg) resident on the
// current device at once; 0 if the device cannot be queried (then the plan
// falls back to a fixed total).
int resident_blocks(int dtype, int kg, bool fail_fast = false, bool wide = false, bool loc = false) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    return cus * screen_blocks_per_cu(dtype, kg, fail_fast, wide, loc);
}
int plan_group_size(int n_cands, int dtype) {
    // Measured on the five screening workloads: groups of 4 for fp32 and
    // for short candidate lists, 8 for long lists of 16-bit tensors (the
    // reference is then re-read by fewer groups).
    int kg_cap = (dtype != DT_F32 && n_cands >= 32) ? 8 : 4;
    if (tuning().kg_cap > 0) kg_cap = tuning().kg_cap;
    int kg = 1;
    while (kg < n_cands && kg < kg_cap) kg *= 2;
    return kg;
}

bool make_plan(int n_cands, int n_acc, uint64_t numel, int dtype, int resident_blocks,
               bool serial_groups, ScreenPlan* plan) {
    if (n_cands < 1 || n_acc < 0 || n_acc > n_cands || !is_float_dtype(dtype)) return false;
    ScreenPlan P{};
    P.dtype = dtype;
    P.n_cands = n_cands;
    P.n_acc = n_acc;
    P.threads = 256;
    P.numel = numel;
    const uint64_t vec = 16 / elem_size(dtype);
    P.n_vec = numel / vec;
    // Candidates per group: all of them when few, else 8 (chosen from n_cands
    // so that the workspace sized for n_cands always suffices).
    P.kg = plan_group_size(n_cands, dtype);
    const int groups_max = (n_cands + P.kg - 1) / P.kg;
    P.n_groups = n_acc > 0 ? (n_acc + P.kg - 1) / P.kg : 0;
    // Work-groups per candidate group (stripes; a multiple of 8, the XCD count):
    //  - at least enough that one work-group sees fewer than 2^31 elements
    //    (32-bit partial counts), at most one per 8 chunks of 512 elements
    //    (so small tensors get at most 16 stripes and a one-level finish);
    //  - plain launch: one round of the work-groups that are resident on the
    //    device at once (occupancy of the chosen kernel x CUs), spread over
    //    the candidate groups -- the grid is persistent, each wave strides
    //    over the chunks -- unless a tuning override sets the total; at most
    //    about 4096 work-groups in all;
    //  - fail-fast launch (serial_groups): the groups are screened in rounds
    //    of ff_round groups, one round after another, and a round is one
    //    set of resident work-groups (stripes = resident / ff_round, at most
    //    2048).  Measured on the 16- and 64-candidate workloads, rounds of 2
    //    groups balance best: with 1 the reference is re-read once per group,
    //    with all groups in one round the work-groups of failed groups idle;
    //  - the workspace is laid out for the bound C_ws, independent of the
    //    device, and the launch never exceeds it.
    const uint64_t n_chunks = numel / 512;
    const uint64_t c_work = align_up((n_chunks + 7) / 8, 8);
    const uint64_t min_c = align_up(numel / (1ull << 31) + 1, 8);
    auto clamp_c = [&](uint64_t c) {
        if (c > c_work) c = c_work;
        if (c < min_c) c = min_c;
        if (c < 8) c = 8;
        return c;
    };
    const uint64_t c_plain = clamp_c(align_up((4096 + groups_max - 1) / groups_max, 8));
    const uint64_t c_ws = clamp_c(c_plain > 2048 ? c_plain : 2048);
    if (c_ws > (1u << 20)) return false;
    int blocks_total = tuning().blocks_total;
    const int ff_round = tuning().ff_round > 0 ? tuning().ff_round : kFailFastRound;
    if (blocks_total <= 0) blocks_total = resident_blocks > 0 ? resident_blocks : 2048;
    const int groups = P.n_groups > 0 ? P.n_groups : 1;
    P.ff_round = ff_round < groups ? ff_round : groups;
    uint64_t C;
    if (serial_groups) {
        C = align_up(((uint64_t)blocks_total + P.ff_round - 1) / P.ff_round, 8);
        if (C > c_ws) C = c_ws;
    } else {
        C = align_up(((uint64_t)blocks_total + groups - 1) / groups, 8);
        if (C > c_plain) C = c_plain;
    }
    if (C < min_c) C = min_c;
    if (C < 8) C = 8;
    P.blocks_per_group = (int)C;
    const uint64_t Cw = c_ws;  // layout stride bound
    // Workspace layout, sized for the group count of n_cands.  The tagged
    // tickets (8 bytes each) come first, then the fail-fast words (one
    // 128-byte line each).
    P.n_super = (int)((C + 15) / 16);
    const int super_ws = (int)((Cw + 15) / 16);
    size_t off = 0;
    P.off_tickets2 = off;
    off += (size_t)groups_max * 8;
    P.off_tickets1 = off;
    off += (size_t)groups_max * super_ws * 8;
    off = align_up(off, 256);
    P.off_ff_flags = off;
    off = align_up(off + (size_t)groups_max * P.kg * (size_t)(1 + super_ws) * 128, 256);
    P.off_part_u32 = off;
    off = align_up(off + (size_t)kPartPlanes * n_cands * Cw * 4, 256);
    P.off_part_ssd = off;
    off = align_up(off + (size_t)n_cands * Cw * 8, 256);
    P.off_part_ssr = off;
    off = align_up(off + (size_t)groups_max * Cw * 8, 256);
    P.off_part_ssrc = off;
    off = align_up(off + (size_t)n_cands * Cw * 8, 256);
    P.off_part2 = off;
    off = align_up(off + (size_t)n_cands * super_ws * sizeof(Part2), 256);
    P.off_part2_ssr = off;
    off = align_up(off + (size_t)groups_max * super_ws * 8, 256);
    P.core_total = off;
    P.off_part_idx = off;
    off = align_up(off + (size_t)IX_COUNT * n_cands * Cw * 8, 256);
    P.off_part2_idx = off;
    off = align_up(off + (size_t)n_cands * super_ws * sizeof(Part2Idx), 256);
    P.total = off;
    *plan = P;
    return true;
}

}  // namespace kb

namespace kb {

// Host memory a call must be given for its launch table: none when the table
// (one entry per candidate) travels in the kernel arguments.
size_t host_table_bytes(int n_cands) {
    return n_cands <= kInlineCands ? 0 : align_up((size_t)n_cands * sizeof(CandEntry), 256);
}

// The screen of n_cands candidates whose gate statuses are already known
// (status[k] == KB_STATUS_OK: read and compared; otherwise a record of
// that status, not read).  Shared by kb_screen, kb_screen_ex, kb_screen_multi
// and kb_screen_noalloc; `who` names the caller in error messages.  The
// caller has validated ref, cands, n_cands, atol, rtol and flags.
// host_table: caller-owned pinned host memory of at least
// host_table_bytes(n_cands) bytes when the table does not fit the kernel
// arguments (the kernels then read it there), else ignored.  d_loc: NULL, or
// the candidates' positions, found in the same pass.
int screen_with_status(const char* who, const kb_tensor* ref, const kb_tensor* cands, int n_cands,
                       const int32_t* status, float atol, float rtol, uint32_t flags, void* workspace,
                       size_t workspace_bytes, void* host_table, size_t host_table_size,
                       kb_stats* d_stats, kb_locate* d_loc, hipStream_t stream) {
    const bool fail_fast = (flags & KB_FAIL_FAST) != 0;
    const bool loc = d_loc != nullptr;
    if (fail_fast && loc)
        return fail(KB_ERR_INVALID_ARG, "%s: positions are not found under KB_FAIL_FAST", who);
    if (!is_contiguous(*ref)) return fail(KB_ERR_INVALID_ARG, "%s: reference is not contiguous", who);
    const uint64_t numel = tensor_numel(*ref);
    const int dtype = ref->dtype;
    // the positions variant keeps 512-element chunk numbers (and two tail
    // codes after them) in 32 bits
    if (loc && numel / 512 + 2 > 0xFFFFFFFFull)
        return fail(KB_ERR_INVALID_ARG, "%s: positions need fewer than 2^41 elements", who);
    int n_acc = 0;
    for (int k = 0; k < n_cands; ++k) n_acc += status[k] == KB_STATUS_OK;

    ScreenPlan P;
    const int kg = plan_group_size(n_cands, dtype);
    const bool wide = use_wide_kernel(dtype, kg, fail_fast, numel, loc);
    if (!make_plan(n_cands, n_acc, numel, dtype, resident_blocks(dtype, kg, fail_fast, wide, loc), fail_fast, &P))
        return fail(KB_ERR_INVALID_ARG, "%s: no launch plan (numel=%llu)", who,
                    (unsigned long long)numel);
    const size_t need = loc ? P.total : P.core_total;
    if (workspace == nullptr || workspace_bytes < need)
        return fail(KB_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", who, workspace_bytes, need);
    if (!aligned16(ref->data) || !aligned16(workspace) || !aligned16(d_stats) || !aligned16(d_loc))
        return fail(KB_ERR_ALIGNMENT, "%s: reference, workspace, d_stats or d_loc not 16-byte aligned", who);
    for (int k = 0; k < n_cands; ++k)
        if (status[k] == KB_STATUS_OK && !aligned16(cands[k].data))
            return fail(KB_ERR_ALIGNMENT, "%s: candidate %d data not 16-byte aligned", who, k);

    // Launch table: the accepted candidates in call order, then the rejected
    // ones (one entry per candidate).  Up to kInlineCands entries travel in
    // the kernel arguments; a longer table is written to the caller's pinned
    // host memory, which the kernels read directly.
    const int n_table = n_cands;
    const bool table_inline = n_table <= kInlineCands;
    const size_t need_table = host_table_bytes(n_cands);
    if (!table_inline && (host_table == nullptr || host_table_size < need_table))
        return fail(KB_ERR_WORKSPACE,
                    "%s: %d candidates need a pinned host table of %zu bytes (kb_screen_ex), %zu given",
                    who, n_cands, need_table, host_table == nullptr ? (size_t)0 : host_table_size);
    if (!table_inline && !aligned16(host_table))
        return fail(KB_ERR_ALIGNMENT, "%s: host table not 16-byte aligned", who);
    InlineTable tab;
    CandEntry* t = table_inline ? tab.e : (CandEntry*)host_table;
    {
        int w = 0;
        for (int k = 0; k < n_cands; ++k)
            if (status[k] == KB_STATUS_OK) t[w++] = CandEntry{cands[k].data, k, KB_STATUS_OK};
        for (int k = 0; k < n_cands; ++k)
            if (status[k] != KB_STATUS_OK) t[w++] = CandEntry{nullptr, k, status[k]};
    }
    const CandEntry* d_table = table_inline ? nullptr : (const CandEntry*)host_table;
    char* ws = (char*)workspace;
    P.wide = wide ? 1 : 0;
    hipError_t e;
    if (n_acc == 0 || numel == 0) {
        e = launch_records_only(d_table, tab, table_inline ? 1 : 0, n_table, numel, d_stats, d_loc, stream);
        if (e != hipSuccess) return fail(KB_ERR_HIP, "%s: records launch: %s", who, hipGetErrorString(e));
        return KB_OK;
    }
    ScreenParams p{};
    p.ref = ref->data;
    p.table = d_table;
    p.numel = numel;
    p.n_vec = P.n_vec;
    p.atol = atol;
    p.rtol = rtol;
    p.flags = flags;
    p.n_acc = n_acc;
    p.n_cands = n_cands;
    p.n_table = n_table;
    p.rej_start = n_acc;
    p.table_inline = table_inline ? 1 : 0;
    p.n_groups = P.n_groups;
    p.blocks_per_group = P.blocks_per_group;
    p.n_super = P.n_super;
    p.ff_round = P.ff_round;
    p.tag = call_tag();
    p.tickets1 = (uint64_t*)(ws + P.off_tickets1);
    p.tickets2 = (uint64_t*)(ws + P.off_tickets2);
    p.ff_flags = (uint32_t*)(ws + P.off_ff_flags);
    p.part_u32 = (uint32_t*)(ws + P.off_part_u32);
    p.part_ssd = (double*)(ws + P.off_part_ssd);
    p.part_ssr = (double*)(ws + P.off_part_ssr);
    p.part_ssrc = (double*)(ws + P.off_part_ssrc);
    p.part2 = (Part2*)(ws + P.off_part2);
    p.part2_ssr = (double*)(ws + P.off_part2_ssr);
    p.part_idx = loc ? (uint64_t*)(ws + P.off_part_idx) : nullptr;
    p.part2_idx = loc ? (Part2Idx*)(ws + P.off_part2_idx) : nullptr;
    p.stats = d_stats;
    p.loc = d_loc;
    e = launch_screen(P, p, tab, fail_fast, loc, stream);
    if (e != hipSuccess) return fail(KB_ERR_HIP, "%s: kernel launch: %s", who, hipGetErrorString(e));
    return KB_OK;
}

}  // namespace kb

using namespace kb;

extern "C" {

const char* kb_last_error(void) { return g_error; }

int kb_version(void) { return 20000; }

int kb_policy_check(const kb_tensor* ref, const kb_tensor* cands, int n_cands, int32_t* status) {
    clear_error();
    if (ref == nullptr || status == nullptr || n_cands < 0 || (n_cands > 0 && cands == nullptr))
        return fail(KB_ERR_INVALID_ARG, "kb_policy_check: null argument or negative count");
    if (!shape_valid(*ref)) return fail(KB_ERR_INVALID_ARG, "reference shape invalid");
    if (ref->data == nullptr && tensor_numel(*ref) != 0)
        return fail(KB_ERR_INVALID_ARG, "reference data is NULL");
    if (!is_float_dtype(ref->dtype))
        return fail(KB_ERR_DTYPE, "reference dtype %d is not F32, F16 or BF16", ref->dtype);
    for (int k = 0; k < n_cands; ++k) status[k] = gate_one(*ref, cands[k]);
    return KB_OK;
}

size_t kb_screen_workspace_bytes(int n_cands, uint64_t numel, int dtype) {
    ScreenPlan P;
    if (!make_plan(n_cands, n_cands, numel, dtype, 0, false, &P)) return 0;
    return P.core_total;
}

size_t kb_screen_positions_workspace_bytes(int n_cands, uint64_t numel, int dtype) {
    ScreenPlan P;
    if (!make_plan(n_cands, n_cands, numel, dtype, 0, false, &P)) return 0;
    return P.total;
}

int kb_screen_launch(int n_cands, uint64_t numel, int dtype, kb_launch* out) {
    clear_error();
    if (out == nullptr) return fail(KB_ERR_INVALID_ARG, "kb_screen_launch: out is NULL");
    if (!is_float_dtype(dtype)) return fail(KB_ERR_DTYPE, "dtype %d not screenable", dtype);
    ScreenPlan P;
    const int kg = plan_group_size(n_cands, dtype);
    if (!make_plan(n_cands, n_cands, numel, dtype,
                   resident_blocks(dtype, kg, false, use_wide_kernel(dtype, kg, false, numel)), false, &P))
        return fail(KB_ERR_INVALID_ARG, "no launch plan for n_cands=%d numel=%llu", n_cands,
                    (unsigned long long)numel);
    out->group_size = P.kg;
    out->n_groups = P.n_groups;
    out->blocks_per_group = P.blocks_per_group;
    out->threads = P.threads;
    out->grid = (int64_t)P.n_groups * P.blocks_per_group;
    return KB_OK;
}

// Checks shared by the screening entry points (no device work).
static int check_screen_args(const char* who, const kb_tensor* ref, const kb_tensor* cands, int n_cands,
                             float atol, float rtol, uint32_t flags, const kb_stats* d_stats) {
    if (ref == nullptr || cands == nullptr || d_stats == nullptr)
        return fail(KB_ERR_INVALID_ARG, "%s: null ref, cands or d_stats", who);
    if (n_cands < 1) return fail(KB_ERR_INVALID_ARG, "%s: n_cands = %d < 1", who, n_cands);
    if (!std::isfinite(atol) || !std::isfinite(rtol) || atol < 0.f || rtol < 0.f)
        return fail(KB_ERR_INVALID_ARG, "%s: atol and rtol must be finite and >= 0", who);
    if (flags & ~(uint32_t)(KB_EQUAL_NAN | KB_FAIL_FAST))
        return fail(KB_ERR_INVALID_ARG, "%s: unknown flags 0x%x", who, flags);
    return KB_OK;
}

size_t kb_screen_host_table_bytes(int n_cands) { return n_cands < 1 ? 0 : host_table_bytes(n_cands); }

int kb_screen_noalloc(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol,
                      float rtol, uint32_t flags, kb_stats* d_stats, hipStream_t stream) {
    clear_error();
    int rc = check_screen_args("kb_screen_noalloc", ref, cands, n_cands, atol, rtol, flags, d_stats);
    if (rc != KB_OK) return rc;
    if (n_cands > KB_INLINE_CANDS)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_noalloc: %d candidates, at most %d", n_cands,
                    KB_INLINE_CANDS);
    int32_t status[KB_INLINE_CANDS];  // on the stack: nothing is allocated
    rc = kb_policy_check(ref, cands, n_cands, status);
    if (rc != KB_OK) return rc;
    ScreenPlan P;
    const uint64_t numel = tensor_numel(*ref);
    if (!make_plan(n_cands, n_cands, numel, ref->dtype, 0, false, &P))
        return fail(KB_ERR_INVALID_ARG, "kb_screen_noalloc: no launch plan (numel=%llu)",
                    (unsigned long long)numel);
    if (P.core_total > (size_t)KB_NOALLOC_SCRATCH_BYTES)
        return fail(KB_ERR_WORKSPACE, "kb_screen_noalloc: the call needs %zu bytes of scratch, the fixed "
                    "scratch holds %zu", P.core_total, (size_t)KB_NOALLOC_SCRATCH_BYTES);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail_hip(e, "kb_screen_noalloc: hipGetDevice");
    void* ws = nullptr;
    rc = noalloc_scratch(dev, &ws);
    if (rc != KB_OK) return rc;
    // The scratch holds what the last call on this device left, laid out for
    // that call's sizes: zero this call's counters and fail-fast words (the
    // words that must begin at zero) with the fill kernel, stream-ordered.
    e = launch_zero_fill(ws, P.off_part_u32, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_screen_noalloc: fill launch");
    return screen_with_status("kb_screen_noalloc", ref, cands, n_cands, status, atol, rtol, flags, ws,
                              (size_t)KB_NOALLOC_SCRATCH_BYTES, nullptr, 0, d_stats, nullptr, stream);
}

int kb_screen_ex(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol, float rtol,
                 uint32_t flags, void* workspace, size_t workspace_bytes, kb_stats* d_stats,
                 const kb_screen_opts* opts, hipStream_t stream) {
    clear_error();
    int rc = check_screen_args("kb_screen", ref, cands, n_cands, atol, rtol, flags, d_stats);
    if (rc != KB_OK) return rc;
    std::vector<int32_t> status((size_t)n_cands);
    rc = kb_policy_check(ref, cands, n_cands, status.data());
    if (rc != KB_OK) return rc;
    return screen_with_status("kb_screen", ref, cands, n_cands, status.data(), atol, rtol, flags,
                              workspace, workspace_bytes, opts ? opts->host_table : nullptr,
                              opts ? opts->host_table_bytes : 0, d_stats, opts ? opts->d_loc : nullptr, stream);
}

int kb_screen(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol, float rtol,
              uint32_t flags, void* workspace, size_t workspace_bytes, kb_stats* d_stats,
              hipStream_t stream) {
    return kb_screen_ex(ref, cands, n_cands, atol, rtol, flags, workspace, workspace_bytes, d_stats,
                        nullptr, stream);
}

// Multi-output candidates: the workspace of output o starts at the sum of
// the 256-byte-aligned single-output sizes of outputs 0..o-1.
static bool multi_layout(const kb_tensor* refs, int n_outputs, int n_cands, size_t* offsets,
                         size_t* total) {
    size_t off = 0;
    for (int o = 0; o < n_outputs; ++o) {
        if (!shape_valid(refs[o]) || !is_float_dtype(refs[o].dtype)) return false;
        const size_t b = kb_screen_workspace_bytes(n_cands, tensor_numel(refs[o]), refs[o].dtype);
        if (b == 0) return false;
        if (offsets) offsets[o] = off;
        off += align_up(b, 256);
    }
    *total = off;
    return true;
}

size_t kb_screen_multi_workspace_bytes(const kb_tensor* refs, int n_outputs, int n_cands) {
    if (refs == nullptr || n_outputs < 1 || n_outputs > KB_MAX_OUTPUTS || n_cands < 1) return 0;
    size_t total = 0;
    return multi_layout(refs, n_outputs, n_cands, nullptr, &total) ? total : 0;
}

size_t kb_screen_multi_host_table_bytes(int n_outputs, int n_cands) {
    if (n_outputs < 1 || n_outputs > KB_MAX_OUTPUTS || n_cands < 1) return 0;
    return (size_t)n_outputs * host_table_bytes(n_cands);
}

int kb_screen_multi(const kb_tensor* refs, int n_outputs, const kb_tensor* cands, int n_cands,
                    const float* atol, const float* rtol, uint32_t flags, void* workspace,
                    size_t workspace_bytes, kb_stats* d_stats, const kb_screen_opts* opts,
                    hipStream_t stream) {
    clear_error();
    if (refs == nullptr || cands == nullptr || atol == nullptr || rtol == nullptr || d_stats == nullptr)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_multi: null refs, cands, atol, rtol or d_stats");
    if (n_outputs < 1 || n_outputs > KB_MAX_OUTPUTS || n_cands < 1)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_multi: n_outputs = %d or n_cands = %d out of range",
                    n_outputs, n_cands);
    for (int o = 0; o < n_outputs; ++o)
        if (!std::isfinite(atol[o]) || !std::isfinite(rtol[o]) || atol[o] < 0.f || rtol[o] < 0.f)
            return fail(KB_ERR_INVALID_ARG, "kb_screen_multi: atol/rtol of output %d not finite and >= 0",
                        o);
    if (flags & ~(uint32_t)(KB_EQUAL_NAN | KB_FAIL_FAST))
        return fail(KB_ERR_INVALID_ARG, "kb_screen_multi: unknown flags 0x%x", flags);
    if (opts != nullptr && opts->d_loc != nullptr)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_multi: positions (d_loc) are not found for multi-output screens");
    // One gate over all outputs: a candidate is accepted only if every output
    // passes; otherwise every output's record carries the first failing
    // check, in output order.
    std::vector<int32_t> combined((size_t)n_cands, KB_STATUS_OK), st((size_t)n_cands);
    std::vector<kb_tensor> col((size_t)n_cands);
    for (int o = 0; o < n_outputs; ++o) {
        for (int k = 0; k < n_cands; ++k) col[k] = cands[(size_t)k * n_outputs + o];
        const int rc = kb_policy_check(&refs[o], col.data(), n_cands, st.data());
        if (rc != KB_OK) {
            char why[sizeof g_error];
            std::memcpy(why, g_error, sizeof why);
            return fail(rc, "kb_screen_multi: reference %d: %s", o, why);
        }
        if (!is_contiguous(refs[o]))
            return fail(KB_ERR_INVALID_ARG, "kb_screen_multi: reference %d is not contiguous", o);
        for (int k = 0; k < n_cands; ++k)
            if (combined[k] == KB_STATUS_OK) combined[k] = st[k];
    }
    std::vector<size_t> offs((size_t)n_outputs);
    size_t total = 0;
    if (!multi_layout(refs, n_outputs, n_cands, offs.data(), &total))
        return fail(KB_ERR_INVALID_ARG, "kb_screen_multi: no workspace layout");
    if (workspace == nullptr || workspace_bytes < total)
        return fail(KB_ERR_WORKSPACE, "kb_screen_multi: workspace of %zu bytes, %zu needed",
                    workspace_bytes, total);
    // Validate every output before launching anything.
    if (!aligned16(workspace) || !aligned16(d_stats))
        return fail(KB_ERR_ALIGNMENT, "kb_screen_multi: workspace or d_stats not 16-byte aligned");
    for (int o = 0; o < n_outputs; ++o) {
        if (!aligned16(refs[o].data))
            return fail(KB_ERR_ALIGNMENT, "kb_screen_multi: reference %d not 16-byte aligned", o);
        for (int k = 0; k < n_cands; ++k)
            if (combined[k] == KB_STATUS_OK && !aligned16(cands[(size_t)k * n_outputs + o].data))
                return fail(KB_ERR_ALIGNMENT, "kb_screen_multi: candidate %d output %d not 16-byte aligned",
                            k, o);
    }
    // Each output's launch table gets its own region of the host table (the
    // outputs' kernels are in flight together).
    const size_t tab_bytes = host_table_bytes(n_cands);
    char* htab = opts ? (char*)opts->host_table : nullptr;
    if (tab_bytes > 0 && (htab == nullptr || opts->host_table_bytes < (size_t)n_outputs * tab_bytes))
        return fail(KB_ERR_WORKSPACE, "kb_screen_multi: %d candidates need a pinned host table of %zu bytes",
                    n_cands, (size_t)n_outputs * tab_bytes);
    char* ws = (char*)workspace;
    for (int o = 0; o < n_outputs; ++o) {
        for (int k = 0; k < n_cands; ++k) col[k] = cands[(size_t)k * n_outputs + o];
        const size_t bytes = (o + 1 < n_outputs ? offs[o + 1] : total) - offs[o];
        const int rc = screen_with_status("kb_screen_multi", &refs[o], col.data(), n_cands, combined.data(),
                                          atol[o], rtol[o], flags, ws + offs[o], bytes,
                                          htab ? htab + (size_t)o * tab_bytes : nullptr, tab_bytes,
                                          d_stats + (size_t)o * n_cands, nullptr, stream);
        if (rc != KB_OK) return rc;
    }
    return KB_OK;
}

int kb_summarize_multi(const kb_stats* h_stats, int n_outputs, int n_cands, kb_summary* summary,
                       int32_t* passed) {
    clear_error();
    if (h_stats == nullptr || summary == nullptr || n_outputs < 1 || n_cands < 0)
        return fail(KB_ERR_INVALID_ARG, "kb_summarize_multi: null argument or bad count");
    const int dirty = dirty_workspace_error(h_stats, n_outputs * n_cands);
    if (dirty != KB_OK) return dirty;
    kb_summary s{n_cands, 0, 0, 0, -1, -1};
    for (int k = 0; k < n_cands; ++k) {
        bool rejected = false, failed = false;
        for (int o = 0; o < n_outputs; ++o) {
            const kb_stats& st = h_stats[(size_t)o * n_cands + k];
            if (st.status != KB_STATUS_OK) rejected = true;
            else if (st.mismatches != 0) failed = true;
        }
        const bool ok = !rejected && !failed;
        if (passed) passed[k] = ok ? 1 : 0;
        if (ok) {
            s.n_passed++;
            if (s.first_passed < 0) s.first_passed = k;
            continue;
        }
        if (rejected) s.n_rejected++;
        else s.n_failed++;
        if (s.first_failed < 0) s.first_failed = k;
    }
    *summary = s;
    return KB_OK;
}

int kb_rung_stats(const double* samples, int n_cands, int n_shapes, int n_iter, int base, int rung,
                  double budget, double alpha, double beta, kb_sample_stats* rows,
                  kb_rung_score* scores, hipStream_t stream) {
    clear_error();
    if (samples == nullptr || rows == nullptr || scores == nullptr)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_stats: null samples, rows or scores");
    if (n_cands < 1 || n_shapes < 1 || n_iter < 1 || n_iter > KB_RUNG_MAX_ITER)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_stats: n_cands=%d n_shapes=%d n_iter=%d out of range",
                    n_cands, n_shapes, n_iter);
    if ((int64_t)n_cands * n_shapes > (1 << 30))
        return fail(KB_ERR_INVALID_ARG, "kb_rung_stats: too many rows");
    if (base < -1 || base >= n_cands)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_stats: base %d not in [-1, %d)", base, n_cands);
    if (rung < 0 || !std::isfinite(budget) || budget < 0.0 || !std::isfinite(alpha) ||
        !std::isfinite(beta))
        return fail(KB_ERR_INVALID_ARG, "kb_rung_stats: bad rung, budget, alpha or beta");
    if (((uintptr_t)samples & 7u) || ((uintptr_t)rows & 7u) || ((uintptr_t)scores & 7u))
        return fail(KB_ERR_ALIGNMENT, "kb_rung_stats: samples, rows or scores not 8-byte aligned");
    RungParams p{n_cands, n_shapes, n_iter, base, rung, budget, alpha, beta};
    hipError_t e = launch_rung_stats(p, samples, rows, scores, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_rung_stats: launch");
    return KB_OK;
}

int kb_rung_promote(const kb_rung_score* scores, int n_cands, int base, int frac_num, int frac_den,
                    int32_t* rank, int32_t* order, int32_t* promoted, hipStream_t stream) {
    clear_error();
    if (scores == nullptr || rank == nullptr || order == nullptr || promoted == nullptr)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_promote: null scores, rank, order or promoted");
    if (n_cands < 1 || n_cands > KB_PROMOTE_MAX)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_promote: n_cands = %d not in [1, %d]", n_cands,
                    KB_PROMOTE_MAX);
    if (base < -1 || base >= n_cands)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_promote: base %d not in [-1, %d)", base, n_cands);
    if (frac_den < 1 || frac_num < 0 || frac_num > frac_den)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_promote: fraction %d/%d not in [0, 1]", frac_num,
                    frac_den);
    if (((uintptr_t)scores & 7u) || ((uintptr_t)rank & 3u) || ((uintptr_t)order & 3u) ||
        ((uintptr_t)promoted & 3u))
        return fail(KB_ERR_ALIGNMENT, "kb_rung_promote: misaligned array");
    hipError_t e = launch_rung_promote(scores, n_cands, base, frac_num, frac_den, rank, order,
                                       promoted, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_rung_promote: launch");
    return KB_OK;
}

int kb_rung_survival(const int32_t* entering, const int32_t* failed, const int32_t* promoted,
                     int n_rungs, int original, double* fail_pct, double* promo_pct) {
    clear_error();
    if (entering == nullptr || failed == nullptr || promoted == nullptr || fail_pct == nullptr ||
        promo_pct == nullptr || n_rungs < 1 || original < 1)
        return fail(KB_ERR_INVALID_ARG, "kb_rung_survival: null array or bad count");
    for (int r = 0; r < n_rungs; ++r)
        if (entering[r] < 0 || failed[r] < 0 || promoted[r] < 0 || failed[r] > entering[r])
            return fail(KB_ERR_INVALID_ARG, "kb_rung_survival: inconsistent counts at rung %d", r);
    for (int r = 0; r < n_rungs; ++r) {
        fail_pct[r] = entering[r] > 0 ? 100.0 * (double)failed[r] / (double)entering[r] : 0.0;
        promo_pct[r] = 100.0 * (double)promoted[r] / (double)original;
    }
    return KB_OK;
}

int kb_screen_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream) {
    clear_error();
    if (workspace == nullptr || workspace_bytes == 0)
        return fail(KB_ERR_WORKSPACE, "kb_screen_workspace_init: no workspace");
    if (!aligned16(workspace) || (workspace_bytes & 15u))
        return fail(KB_ERR_ALIGNMENT, "kb_screen_workspace_init: workspace not 16-byte aligned/sized");
    hipError_t e = launch_zero_fill(workspace, workspace_bytes, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_screen_workspace_init: fill launch");
    return KB_OK;
}

int kb_summarize(const kb_stats* h_stats, int n_cands, kb_summary* summary, int32_t* passed) {
    clear_error();
    if (h_stats == nullptr || n_cands < 0)
        return fail(KB_ERR_INVALID_ARG, "kb_summarize: null records or negative count");
    const int dirty = dirty_workspace_error(h_stats, n_cands);
    if (dirty != KB_OK) return dirty;
    kb_summary s{n_cands, 0, 0, 0, -1, -1};
    for (int k = 0; k < n_cands; ++k) {
        const kb_stats& st = h_stats[k];
        // K(p) for one output: accepted by the gate and no mismatching element
        const bool ok = st.status == KB_STATUS_OK && st.mismatches == 0;
        if (passed) passed[k] = ok ? 1 : 0;
        if (ok) {
            s.n_passed++;
            if (s.first_passed < 0) s.first_passed = k;
            continue;
        }
        if (st.status != KB_STATUS_OK) s.n_rejected++;
        else s.n_failed++;
        if (s.first_failed < 0) s.first_failed = k;
    }
    if (summary) *summary = s;
    return KB_OK;
}

int kb_screen_stats(const kb_stats* d_stats, int n_cands, kb_stats* h_stats, kb_summary* summary,
                    int32_t* passed, hipStream_t stream) {
    clear_error();
    if (d_stats == nullptr || n_cands < 0)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_stats: null d_stats or negative count");
    std::vector<kb_stats> tmp;
    kb_stats* dst = h_stats;
    if (dst == nullptr && (summary != nullptr || passed != nullptr)) {
        tmp.resize((size_t)n_cands);
        dst = tmp.data();
    }
    if (n_cands > 0 && dst != nullptr) {
        hipError_t e = hipMemcpyAsync(dst, d_stats, (size_t)n_cands * sizeof(kb_stats),
                                      hipMemcpyDeviceToHost, stream);
        if (e != hipSuccess) return fail_hip(e, "kb_screen_stats: hipMemcpyAsync");
    }
    hipError_t e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail_hip(e, "kb_screen_stats: hipStreamSynchronize");
    if (dst != nullptr) return kb_summarize(dst, n_cands, summary, passed);
    return KB_OK;  // (without a host copy there is nothing to check)
}

int kb_screen_locate(const kb_tensor* ref, const kb_tensor* cands, int n_cands, float atol,
                     float rtol, uint32_t flags, const kb_stats* stats, kb_locate* d_loc,
                     hipStream_t stream) {
    clear_error();
    if (ref == nullptr || cands == nullptr || stats == nullptr || d_loc == nullptr)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_locate: null ref, cands, stats or d_loc");
    if (n_cands < 1) return fail(KB_ERR_INVALID_ARG, "kb_screen_locate: n_cands = %d < 1", n_cands);
    if (!std::isfinite(atol) || !std::isfinite(rtol) || atol < 0.f || rtol < 0.f)
        return fail(KB_ERR_INVALID_ARG, "kb_screen_locate: atol and rtol must be finite and >= 0");
    if (flags & ~(uint32_t)(KB_EQUAL_NAN | KB_FAIL_FAST))
        return fail(KB_ERR_INVALID_ARG, "kb_screen_locate: unknown flags 0x%x", flags);
    std::vector<int32_t> status((size_t)n_cands);
    int rc = kb_policy_check(ref, cands, n_cands, status.data());
    if (rc != KB_OK) return rc;
    if (!is_contiguous(*ref)) return fail(KB_ERR_INVALID_ARG, "reference is not contiguous");
    if (!aligned16(ref->data) || !aligned16(d_loc))
        return fail(KB_ERR_ALIGNMENT, "kb_screen_locate: reference or d_loc not 16-byte aligned");
    for (int k = 0; k < n_cands; ++k)
        if (status[k] == KB_STATUS_OK && !aligned16(cands[k].data))
            return fail(KB_ERR_ALIGNMENT, "kb_screen_locate: candidate %d not 16-byte aligned", k);
    const uint64_t numel = tensor_numel(*ref);
    // every position starts as "none" (all ones, -1 as int64)
    hipError_t e = launch_fill_u32(d_loc, (uint64_t)n_cands * sizeof(kb_locate) / 4, 0xFFFFFFFFu, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_screen_locate: fill");
    if (numel == 0) return KB_OK;
    LocateParams p{};
    p.ref = ref->data;
    p.numel = numel;
    p.atol = atol;
    p.rtol = rtol;
    p.flags = flags;
    p.stats = stats;
    p.out = d_loc;
    // Work-groups per candidate: the launch is one round of the work-groups
    // resident on the device at once (occupancy x CUs; a launch of more
    // makes a second, mostly idle round), spread over the launch's
    // candidates, a multiple of 8 (the XCD count), at least 8 and at most
    // one per 8 chunks.
    const uint64_t n_chunks = numel / 512;
    int resident = 0;
    {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
            resident = cus * locate_blocks_per_cu(ref->dtype);
    }
    if (resident <= 0) resident = 2048;
    LocTable tab;
    int k = 0;
    while (k < n_cands) {
        int n = 0;
        for (; k < n_cands && n < kLocateBatch; ++k)
            if (status[k] == KB_STATUS_OK) tab.e[n++] = LocEntry{cands[k].data, k, 0};
        if (n == 0) break;
        uint64_t stripes = (uint64_t)resident / n / 8 * 8;
        if (stripes < 8) stripes = 8;
        const uint64_t cap = n_chunks / 8 > 8 ? n_chunks / 8 / 8 * 8 : 8;
        if (stripes > cap) stripes = cap;
        p.n = n;
        p.stripes = (int)stripes;
        e = launch_locate(ref->dtype, p, tab, stream);
        if (e != hipSuccess) return fail_hip(e, "kb_screen_locate: kernel launch");
    }
    return KB_OK;
}

int kb_gen_inputs(void* dst, int dtype, uint64_t n, int dist, float p0, float p1, uint64_t seed,
                  uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream) {
    clear_error();
    if (dtype < DT_F32 || dtype > DT_U32) return fail(KB_ERR_DTYPE, "unknown dtype %d", dtype);
    if (dist < KB_DIST_U32 || dist > KB_DIST_STUDENT_T3)
        return fail(KB_ERR_INVALID_ARG, "unknown distribution %d", dist);
    if ((dist == KB_DIST_U32) != (dtype == DT_U32))
        return fail(KB_ERR_DTYPE, "distribution %d does not produce dtype %d", dist, dtype);
    if (!std::isfinite(p0) || !std::isfinite(p1))
        return fail(KB_ERR_INVALID_ARG, "p0 and p1 must be finite");
    if (n == 0) return KB_OK;
    if (dst == nullptr) return fail(KB_ERR_INVALID_ARG, "dst is NULL");
    if (!aligned16(dst)) return fail(KB_ERR_ALIGNMENT, "dst not 16-byte aligned");
    if (offset + n < offset) return fail(KB_ERR_INVALID_ARG, "offset + n overflows");
    hipError_t e = dist == KB_DIST_STUDENT_T3
                       ? launch_gen_t3(dst, dtype, n, p0, p1, seed, stream_id, sub, offset, stream)
                       : launch_gen(dst, dtype, n, dist, p0, p1, seed, stream_id, sub, offset, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_gen_inputs: kernel launch");
    return KB_OK;
}

int kb_gen_softmax_rows(void* dst, int dtype, uint64_t rows, uint64_t cols, float sigma, uint64_t seed,
                        uint32_t stream_id, uint32_t sub, hipStream_t stream) {
    clear_error();
    if (dtype != DT_F32) return fail(KB_ERR_DTYPE, "kb_gen_softmax_rows: dtype %d is not F32", dtype);
    if (!std::isfinite(sigma)) return fail(KB_ERR_INVALID_ARG, "kb_gen_softmax_rows: sigma not finite");
    if (rows == 0) return KB_OK;
    if (cols == 0) return fail(KB_ERR_INVALID_ARG, "kb_gen_softmax_rows: cols = 0");
    if (cols > ~0ull / rows) return fail(KB_ERR_INVALID_ARG, "kb_gen_softmax_rows: rows * cols overflows");
    if (dst == nullptr) return fail(KB_ERR_INVALID_ARG, "kb_gen_softmax_rows: dst is NULL");
    if (!aligned16(dst)) return fail(KB_ERR_ALIGNMENT, "kb_gen_softmax_rows: dst not 16-byte aligned");
    hipError_t e = launch_softmax_rows((float*)dst, rows, cols, sigma, seed, stream_id, sub, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_gen_softmax_rows: kernel launch");
    return KB_OK;
}

int kb_gen_indices(uint64_t* dst, uint32_t m, uint64_t n, uint64_t seed, uint32_t stream_id, uint32_t sub,
                   hipStream_t stream) {
    clear_error();
    if (m < 1 || m > KB_MAX_INDICES)
        return fail(KB_ERR_INVALID_ARG, "kb_gen_indices: m = %u not in [1, %d]", m, KB_MAX_INDICES);
    if (n < 2 * (uint64_t)m)
        return fail(KB_ERR_INVALID_ARG, "kb_gen_indices: n = %llu < 2 m", (unsigned long long)n);
    if (dst == nullptr) return fail(KB_ERR_INVALID_ARG, "kb_gen_indices: dst is NULL");
    if (!aligned16(dst)) return fail(KB_ERR_ALIGNMENT, "kb_gen_indices: dst not 16-byte aligned");
    hipError_t e = launch_indices(dst, m, n, seed, stream_id, sub, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_gen_indices: kernel launch");
    return KB_OK;
}

int kb_gen_perturb(void* dst, const void* src, int dtype, uint64_t n, int op, float a, float b, float p,
                   uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream) {
    clear_error();
    if (!is_float_dtype(dtype)) return fail(KB_ERR_DTYPE, "kb_gen_perturb: dtype %d not F32, F16 or BF16", dtype);
    if (op < KB_PERTURB_ADD_UNIFORM || op > KB_PERTURB_ZERO_SUBNORMAL_REL)
        return fail(KB_ERR_INVALID_ARG, "kb_gen_perturb: unknown op %d", op);
    if (op >= KB_PERTURB_SPECIALS && dtype != DT_F32)
        return fail(KB_ERR_DTYPE, "kb_gen_perturb: op %d takes F32 only", op);
    if (!std::isfinite(a) || !std::isfinite(b) || !std::isfinite(p))
        return fail(KB_ERR_INVALID_ARG, "kb_gen_perturb: a, b and p must be finite");
    if (n == 0) return KB_OK;
    if (dst == nullptr || src == nullptr) return fail(KB_ERR_INVALID_ARG, "kb_gen_perturb: dst or src is NULL");
    if (!aligned16(dst) || !aligned16(src))
        return fail(KB_ERR_ALIGNMENT, "kb_gen_perturb: dst or src not 16-byte aligned");
    if (offset + n < offset) return fail(KB_ERR_INVALID_ARG, "kb_gen_perturb: offset + n overflows");
    hipError_t e = launch_perturb(dst, src, dtype, n, op, a, b, p, seed, stream_id, sub, offset, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_gen_perturb: kernel launch");
    return KB_OK;
}

int kb_gen_scatter(void* dst, const void* ref, int dtype, uint64_t n, const uint64_t* idx, uint32_t m, int mode,
                   hipStream_t stream) {
    clear_error();
    if (!is_float_dtype(dtype)) return fail(KB_ERR_DTYPE, "kb_gen_scatter: dtype %d not F32, F16 or BF16", dtype);
    if (mode != KB_SCATTER_NAN && mode != KB_SCATTER_INF_SIGN_OF_REF)
        return fail(KB_ERR_INVALID_ARG, "kb_gen_scatter: unknown mode %d", mode);
    if (m == 0 || n == 0) return KB_OK;
    if (dst == nullptr || ref == nullptr || idx == nullptr)
        return fail(KB_ERR_INVALID_ARG, "kb_gen_scatter: dst, ref or idx is NULL");
    if (!aligned16(dst) || !aligned16(ref) || ((uintptr_t)idx & 7u))
        return fail(KB_ERR_ALIGNMENT, "kb_gen_scatter: dst or ref not 16-byte, or idx not 8-byte, aligned");
    hipError_t e = launch_scatter(dst, ref, dtype, n, idx, m, mode, stream);
    if (e != hipSuccess) return fail_hip(e, "kb_gen_scatter: kernel launch");
    return KB_OK;
}

}  // extern "C"
