// kb_screen.hip -- batched screening kernel for gfx950.
//
// One pass over the reference and K candidate outputs computing, per
// candidate, the statistics of the Verifier's output check (correctness
// indicator K(p), Sections 3.1 and 3.4): mismatches under
// |c - r| <= atol + rtol*|r|, NaN/+Inf/-Inf counts, bitwise identity, max
// abs error, max rel error and the two squared-error sums of the relative L2
// error.  The work is a streaming reduction bound by HBM bandwidth (no
// contraction, so no MFMA); the design goal is to spend fewer VALU
// instructions per (element, candidate) than HBM delivers elements.
//
// Work split.  Candidates that passed the policy gate are cut into groups of
// KG.  A work-group (4 waves) owns one candidate group and one stripe of the
// element range.  A wave handles 512-element chunks (8 elements per lane:
// one 16-byte load per tensor for 16-bit types, two for fp32), grid-striding
// over the group's waves so that consecutive waves read consecutive memory.
// Each reference chunk is loaded once and compared with the KG candidate
// chunks while it sits in registers.  Work-group ids are mapped so that the
// candidate groups of one stripe run on the same XCD (ids are dealt to the 8
// XCDs round robin), so a reference stripe fetched for one group is found in
// that XCD's L2 by the others.
//
// Two paths per (chunk, candidate), chosen per wave:
//   fast  -- all values finite and no extreme squared difference: per
//            element one subtract, one compare (match counts are popcounts of
//            wave ballots, kept in scalar registers), a max tree for the max
//            abs error, one multiply by a per-reference reciprocal for the
//            max-rel filter, and one fused multiply-add for the squared
//            difference (8 binary32 terms per lane, then one binary64 add);
//   exact -- the definition applied element by element (IEEE division,
//            binary64 squares, NaN/Inf classification), taken by a wave when
//            any lane sees a NaN, an infinity or a binary32 overflow of
//            (c - r)^2.
// Two narrower exact fix-ups run inside the fast path: binary64 squares for
// lanes whose differences are all below 2^-60 (where binary32 squares would
// underflow), and IEEE division for lanes whose filtered relative error may
// exceed the wave's exact running maximum.  Every count, flag and maximum is
// therefore exact; the sum of squares has relative error at most about
// 8 * 2^-24 (eight binary32 roundings per lane and chunk) before the binary64
// accumulation.
//
// Reduction.  Lane values -> 64-lane DPP reductions (wave-level counts are
// already scalar) -> LDS combine of the work-group's waves in wave order ->
// per-(work-group, candidate) partials in the workspace.  The last
// work-group of a candidate group to finish (atomic ticket after a release
// fence) combines its group's partials in a fixed order with 16 lanes per
// candidate and writes the kb_stats records, so the binary64 sums are the
// same bits on every call.
#include "kb_device.hpp"
#include "kb_internal.hpp"

namespace kb {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kE = 8;                 // elements per lane per chunk
constexpr int kChunk = 64 * kE;       // elements per wave per chunk
constexpr float kTiny = 0x1p-60f;     // below this binary32 squares may underflow

// Raw storage of one lane's 8 elements of a chunk.
template <int DT>
struct Raw {
    static constexpr int kWords = DT == DT_F32 ? 8 : 4;
    uint32_t w[kWords];
};

// Bytes of one tensor per 512-element chunk.
template <int DT>
constexpr uint64_t chunk_bytes() {
    return DT == DT_F32 ? 4 * kChunk : 2 * kChunk;
}

// Global (address space 1) pointers.  Tensor bases are wave-uniform and
// kept in scalar registers; a load adds the lane's 32-bit byte offset, so
// the address costs no vector instruction (global_load with a scalar base).
typedef const __attribute__((address_space(1))) char* gbytes;
typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) v4u32* gvec;

template <bool NT>
__device__ __forceinline__ v4u32 ld16(gvec p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}

// fp32: lane l holds elements 4l..4l+3 and 256+4l..256+4l+3 of the chunk
// (two fully coalesced 1 KB wave loads); 16-bit: elements 8l..8l+7.  NT
// marks the loads nontemporal: every candidate byte is used once, and
// streaming it past the caches leaves them to the reference, which the
// other candidate groups of the stripe re-read.  base is the chunk's first
// byte (wave-uniform), off = 16 * lane.
template <int DT, bool NT>
__device__ __forceinline__ Raw<DT> load_chunk(gbytes base, uint32_t off) {
    Raw<DT> x;
    const v4u32 a = ld16<NT>((gvec)(base + off));
    x.w[0] = a.x; x.w[1] = a.y; x.w[2] = a.z; x.w[3] = a.w;
    if constexpr (DT == DT_F32) {
        const v4u32 b = ld16<NT>((gvec)(base + off + 1024u));
        x.w[4] = b.x; x.w[5] = b.y; x.w[6] = b.z; x.w[7] = b.w;
    }
    return x;
}

// A pointer made explicitly wave-uniform (held in scalar registers).
__device__ __forceinline__ gbytes uniform_ptr(uint64_t v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (gbytes)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ gbytes uniform_ptr(const void* p) { return uniform_ptr((uint64_t)p); }
__device__ __forceinline__ gbytes uniform_ptr(gbytes p) { return uniform_ptr((uint64_t)p); }

template <int DT>
__device__ __forceinline__ float widen_bits(uint32_t bits) {
    if constexpr (DT == DT_F32) return __uint_as_float(bits);
    else if constexpr (DT == DT_F16) return f16_bits_to_f32(bits);
    else return bf16_bits_to_f32(bits);
}

// Element i (0..7) of a lane's chunk, widened exactly to binary32.
template <int DT>
__device__ __forceinline__ float elem(const Raw<DT>& x, int i) {
    if constexpr (DT == DT_F32) return __uint_as_float(x.w[i]);
    else if constexpr (DT == DT_F16) return f16_bits_to_f32((x.w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
    else return bf16_bits_to_f32(i & 1 ? (x.w[i >> 1] >> 16) : (x.w[i >> 1] & 0xFFFFu));
}

__device__ __forceinline__ uint32_t popc(uint64_t m) { return (uint32_t)__builtin_popcountll(m); }

// Number of lanes with |s| <= tol (a wave-uniform count).  The compare and
// the population count are one unit, so the 64-bit lane mask lives only in
// VCC: counting eight elements per candidate this way keeps no masks alive
// in scalar registers (which, with several candidates in flight, would
// spill to vector lanes and cost more than the compares themselves).  No
// wait states are needed between a VALU write of VCC and a SALU read.
__device__ __forceinline__ uint32_t count_within(float s, float tol) {
    uint32_t n;
    asm("v_cmp_le_f32_e64 vcc, |%1|, %2\n\ts_bcnt1_i32_b64 %0, vcc"
        : "=s"(n)
        : "v"(s), "v"(tol)
        : "vcc");
    return n;
}

// Cross-work-group hand-off without L2 maintenance.  Partials are written
// with agent-scope atomic stores (made coherent across XCDs by the store
// itself), the work-group waits for their completion, and only then takes a
// ticket with a relaxed agent-scope atomic.  The work-group that draws the
// last ticket reads the partials with agent-scope atomic loads, which return
// the coherent copy.  So no work-group writes back or invalidates its XCD's
// L2, which is what a device-scope fence costs here and which would also
// evict the lines other work-groups on the XCD are streaming.
__device__ __forceinline__ void complete_stores() { __builtin_amdgcn_s_waitcnt(0); }
template <class T>
__device__ __forceinline__ T ld_coherent(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Self-checking tickets.  Every arrival adds D = (tag << 32) | 1 to its
// 64-bit ticket word, the call's tag being odd.  A word that was zero when
// the call began (as every completed call leaves its words) holds j D after
// j arrivals, so its high half is always its low half times the tag (mod
// 2^32).  A word that began with anything else -- a value left by a call cut
// short, the partials of a call with other sizes laid out over it, or
// whatever the memory held -- fails that test: with the tag odd, an old
// value (h, l) passes only if h = l tag mod 2^32, which a nonzero leftover
// meets by chance with probability 2^-32.  So a leftover ticket cannot make
// a work-group that is not the last finish the group; a work-group that
// finds a failed test reports the workspace instead (the caller's readback
// then returns an error).  Arrivals stay single atomic adds, which the
// memory-side atomic unit serves back to back: claiming the word with a
// compare-exchange, per arrival or per work-group start, was measured to
// cost 7-15 us on the 16 x 4096^2 bf16 screen.  Returns the arrival number
// (1-based), or 0 when the word did not begin at zero.
__device__ __forceinline__ uint32_t ticket_arrive(uint64_t* t, uint32_t tag) {
    const uint64_t old =
        __hip_atomic_fetch_add(t, ((uint64_t)tag << 32) | 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t n = (uint32_t)old;
    return (uint32_t)(old >> 32) == n * tag ? n + 1u : 0u;
}

template <class T>
__device__ __forceinline__ void st_coherent(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent(double* p, double v) {
    st_coherent((uint64_t*)p, __builtin_bit_cast(uint64_t, v));
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
__device__ __forceinline__ float wave_max_f(float v) {
    return __uint_as_float(wave_max_u32(__float_as_uint(v)));
}

// Hides a value from the optimizer, so that work on it inside a rare branch
// is not hoisted into the common path (it would run for every chunk and
// keep registers live across the loop).
__device__ __forceinline__ void opaque(float& x) { asm volatile("" : "+v"(x)); }

// Max relative error.  The record holds max over elements of fl(d / |r|)
// (IEEE division, NaN quotients ignored); rounding is monotone, so this is
// also fl of the largest exact ratio.  A wave keeps O, the exact maximum of
// the quotients it has seen (wave-uniform, per candidate).  An element can
// raise it only if d / a > O, i.e. d - O a > 0, and fma(-O, a, d) has the
// sign of d - O a (one rounding; an exact zero stays zero), so
//   y = fma(-O, |r|, |c - r|) > 0
// is a filter that never misses (elements that tie O give y = 0 and are
// skipped).  A wave whose filter passes computes the IEEE quotients of the
// passing elements.  The one blind spot is underflow: y rounds to zero
// when 0 < d - O a < 2^-150, which can hide an exceeding element only if
// O a < 2^-125; lanes holding a nonzero |r| with O |r| < 2^-124 therefore
// take the exact test too -- unless O is an integer: then O a, like d, lies
// on the 2^-149 grid of binary32, so a nonzero d - O a is at least 2^-149
// and cannot underflow (the common case O = 1 of flushed subnormals).
//
// The waves of a work-group share what they learn: a wave that raises its
// O also raises the work-group's copy in LDS, which every wave reads with
// each chunk and takes into its own O.  A shared value is a quotient some
// wave of the work-group recorded, so the maximum over the waves is
// unchanged, and skipping elements with d / a <= O loses nothing; a stale
// value only filters less.  (Sharing across the grid through global atomics
// was measured to cost far more than it saves: every work-group contends
// for the same few words.)
//
// The largest quotient of one lane's elements that pass the filter (0 if
// none), and in `slot` the first slot that holds it (kE if none; a slot
// holding a quotient > O always passes, so this is the lane's first element
// of that quotient).  GUARD: the lane may be in the underflow case, so the
// sign of d - O a is taken in binary64 (the product of two binary32 values is
// exact there and one rounding keeps the sign); otherwise the binary32
// residual is exact.
template <bool GUARD>
__device__ __forceinline__ float rel_quotients(const float s[kE], const float r[kE], float O, uint32_t& slot) {
    float qm = 0.f;
    slot = kE;
#pragma unroll
    for (int i = 0; i < kE; ++i) {
        const float d = fabsf(s[i]);
        float a = fabsf(r[i]);
        // (opaque: the binary64 conversions stay in this rare path instead
        // of being hoisted into every chunk, where they would hold 16
        // registers across the candidate loop)
        if constexpr (GUARD) opaque(a);
        const bool pass = GUARD ? __builtin_fma(-(double)O, (double)a, (double)d) > 0.0
                                : fmaf(-O, a, d) > 0.f;
        if (pass) {
            const float q = d / a;
            if (q > qm) {
                qm = q;
                slot = i;
            }
        }
    }
    return qm;
}

// Non-finite counts (rare): per wave, per candidate, in LDS.
struct NonFinite {
    uint32_t nan, pinf, ninf;
};

// The definition, element by element, for a whole lane chunk of one
// candidate (every lane active).  Also the path for the ragged tail.
// Updates the wave's mismatch count, the lane's max abs error, the wave's
// max-rel O and non-finite counts, and adds the lane's binary64 squared
// differences to its LDS slot.  LOC: a rise of the lane's max abs error
// also records `code` (the chunk) in achunk.
// LOC also gives the lane's largest quotient in qm_out and its first slot in
// qslot (kE if no quotient is positive).
template <int DT, bool LOC>
__device__ __forceinline__ void exact_chunk(const Raw<DT>& cand, const float r_in[kE], float atol,
                                            float rtol, bool equal_nan, double* ssd_slot,
                                            uint32_t& mism, uint32_t& amax, uint32_t& achunk, uint32_t code,
                                            float& O, NonFinite& nf, float& qm_out, uint32_t& qslot) {
    float r[kE];
#pragma unroll
    for (int i = 0; i < kE; ++i) {
        r[i] = r_in[i];
        opaque(r[i]);
    }
    uint32_t nm = 0, nnan = 0, npinf = 0, nninf = 0;
    float ma = 0.f, qm = 0.f;
    double sd = 0.0;
    qslot = kE;
#pragma unroll
    for (int i = 0; i < kE; ++i) {
        const float c = elem<DT>(cand, i);
        const float ri = r[i];
        const bool cnan = __builtin_isnan(c);
        nnan += popc(ballot(cnan));
        npinf += popc(ballot(c == __builtin_inff()));
        nninf += popc(ballot(c == -__builtin_inff()));
        const float d = fabsf(c - ri);
        const float a = fabsf(ri);
        const bool rfin = __builtin_isfinite(ri);
        const float tol = rfin ? __fadd_rn(atol, __fmul_rn(rtol, a)) : -1.0f;
        const bool match = (c == ri) || (d <= tol) || (equal_nan && cnan && __builtin_isnan(ri));
        nm += popc(ballot(!match));
        ma = fmaxf(ma, d);       // NaN differences are ignored
        if constexpr (LOC) {
            const float q = d / a;
            if (q > qm) {        // NaN quotients (0/0, inf/inf) never are
                qm = q;
                qslot = i;
            }
        } else {
            qm = fmaxf(qm, d / a);   // so are 0/0 and inf/inf
        }
        if (rfin && __builtin_isfinite(c)) sd = __builtin_fma((double)d, (double)d, sd);
    }
    atomicAdd(ssd_slot, sd);
    mism += nm;
    if constexpr (LOC) {
        if (__float_as_uint(ma) > amax) {
            amax = __float_as_uint(ma);
            achunk = code;
        }
    } else {
        amax = max(amax, __float_as_uint(ma));
    }
    O = fmaxf(O, wave_max_f(qm));
    qm_out = qm;
    nf.nan += nnan;
    nf.pinf += npinf;
    nf.ninf += nninf;
}

// ----------------------------------------------------------- positions ---
// The position search inside the screening pass (LOC) keeps, per wave and
// candidate: the first chunk whose count shows a mismatch (a wave visits its
// chunks in increasing index order), searched for the element after the
// loop; the chunk in which each lane's running max abs error last rose
// (strictly, so its first occurrence), re-read after the loop; and the element
// of the wave's own max rel error, found when it rises.  In the common path
// only the max-abs chunk costs instructions (a compare and two selects in
// place of a max).
constexpr uint64_t kNone = ~0ull;

// Element offset within the chunk of slot i of `lane` (fp32: elements
// 4 lane .. 4 lane + 3 and 256 + 4 lane ..; 16-bit: 8 lane ..), increasing
// with i; kE (no slot) maps to all ones.
template <int DT>
__device__ __forceinline__ uint32_t slot_offset(int lane, uint32_t i) {
    if (i >= (uint32_t)kE) return 0xFFFFFFFFu;
    if constexpr (DT == DT_F32) return i < 4 ? 4u * lane + i : 256u + 4u * lane + (i - 4u);
    else return 8u * lane + i;
}

// The lane's first slot whose element does not match (the definition's
// predicate, special values included), kE if none.
template <int DT>
__device__ __forceinline__ uint32_t lane_first_mismatch(const Raw<DT>& cand, const float r[kE], float atol, float rtol,
                                                        bool equal_nan) {
    uint32_t slot = kE;
#pragma unroll
    for (int i = kE - 1; i >= 0; --i) {
        const float c = elem<DT>(cand, i);
        const float d = fabsf(c - r[i]);
        const float tol = __builtin_isfinite(r[i]) ? __fadd_rn(atol, __fmul_rn(rtol, fabsf(r[i]))) : -1.0f;
        const bool match = (c == r[i]) || (d <= tol) || (equal_nan && __builtin_isnan(c) && __builtin_isnan(r[i]));
        if (!match) slot = i;
    }
    return slot;
}

// The lane's first slot whose |c - r| has the bits m, kE if none.
template <int DT>
__device__ __forceinline__ uint32_t lane_abs_slot(const Raw<DT>& cand, const Raw<DT>& ref, uint32_t m) {
    uint32_t slot = kE;
#pragma unroll
    for (int i = kE - 1; i >= 0; --i)
        if (__float_as_uint(fabsf(elem<DT>(cand, i) - elem<DT>(ref, i))) == m) slot = i;
    return slot;
}

// A wave's position (wave-uniform v) into its LDS slot.
__device__ __forceinline__ void set_idx(uint64_t* slot, uint64_t v, int lane) {
    if (lane == 0) *slot = v;
}

// Raises the work-group's max-rel value of one candidate (rare; O >= 0, so
// the binary32 bits order like the values).
__device__ __forceinline__ void publish_rel(uint32_t* s_rel, float O, int lane) {
    if (lane == 0) atomicMax(s_rel, __float_as_uint(O));
}

// fp16 needs no guard at all: a nonzero binary32 difference of two fp16
// values is at least 2^-24 and |r| is below 2^16, so O > 0 means O >= 2^-40,
// and a nonzero |r| is at least 2^-24, so O |r| >= 2^-64 > 2^-124.
template <int DT>
constexpr bool kGuard = DT != DT_F16;

// 2|x| - 2 on the bits of x: zeros map to the top of the unsigned range, so
// an unsigned minimum over it picks the smallest nonzero magnitude.  (An
// opaque instruction, so the compiler keeps it on the widened bits.)
__device__ __forceinline__ uint32_t nz_key(float x) {
    uint32_t u;
    asm("v_lshl_add_u32 %0, %1, 1, -2" : "=v"(u) : "v"(__float_as_uint(x)));
    return u;
}

// The record of one accepted candidate from its combined statistics.
__device__ __forceinline__ void write_record(kb_stats* dst, uint64_t numel, uint64_t mi, uint64_t na,
                                             uint64_t pi, uint64_t ni, uint32_t ma, uint32_t mr,
                                             uint32_t bd, double sd, double sr) {
    kb_stats st;
    st.numel = numel;
    st.mismatches = mi;
    st.nan_count = na;
    st.pos_inf_count = pi;
    st.neg_inf_count = ni;
    st.sum_sq_diff = sd;
    st.sum_sq_ref = sr;
    st.rel_l2 = sr > 0.0 ? sqrt(sd / sr) : (sd == 0.0 ? 0.0 : __builtin_inf());
    st.max_abs_err = __uint_as_float(ma);
    st.max_rel_err = __uint_as_float(mr);
    st.bitwise_equal = bd == 0u ? 1 : 0;
    st.status = KB_STATUS_OK;
    *dst = st;
}

// Positions of one candidate (all ones: none -> -1).
__device__ __forceinline__ void write_loc(kb_locate* dst, uint64_t fm, uint64_t ai, uint64_t ri) {
    kb_locate l;
    l.first_mismatch = fm == kNone ? -1 : (int64_t)fm;
    l.max_abs_index = ai == kNone ? -1 : (int64_t)ai;
    l.max_rel_index = ri == kNone ? -1 : (int64_t)ri;
    l.reserved = -1;
    *dst = l;
}

// The launch table: the kernel argument, or the caller's pinned host copy.
__device__ __forceinline__ const CandEntry* table_of(const ScreenParams& p, const InlineTable& tab) {
    return p.table_inline ? tab.e : p.table;
}

// A work-group found a ticket word that did not begin at zero: the group
// cannot be finished reliably, so its candidates' records say so (status
// KB_ERR_WORKSPACE, every other field zero; the readback reports the error),
// and group 0 also writes the rejected candidates' records.  Every
// work-group of the group that finds it writes the same bytes.
__device__ __forceinline__ void report_dirty(const ScreenParams& p, const CandEntry* table, int g, int j0,
                                             int kg) {
    for (int j = threadIdx.x; j < kg; j += kThreads) {
        kb_stats st = {};
        st.status = KB_ERR_WORKSPACE;
        p.stats[table[j0 + j].index] = st;
        if (p.loc) write_loc(&p.loc[table[j0 + j].index], kNone, kNone, kNone);
    }
    if (g == 0) {
        for (int k = p.rej_start + (int)threadIdx.x; k < p.n_table; k += kThreads) {
            kb_stats st = {};
            st.status = table[k].status;
            p.stats[table[k].index] = st;
            if (p.loc) write_loc(&p.loc[table[k].index], kNone, kNone, kNone);
        }
    }
}

// Records (and, with positions, all -1 positions) of the rejected candidates
// (written by group 0's finisher).
__device__ __forceinline__ void write_rejected(const ScreenParams& p, const CandEntry* table) {
    for (int k = p.rej_start + (int)threadIdx.x; k < p.n_table; k += kThreads) {
        kb_stats st = {};
        st.status = table[k].status;
        p.stats[table[k].index] = st;
        if (p.loc) write_loc(&p.loc[table[k].index], kNone, kNone, kNone);
    }
}

// Per-wave results, combined across the work-group's waves in LDS.
struct WaveOut {
    uint32_t u[PF_COUNT];
    double ssd;
};

// Minimum waves per SIMD the register allocator must allow: 4 (at most 128
// VGPRs) where the kernel fits without spilling, else 2.
constexpr int min_waves(int dt, int kg) { return kg <= 4 || (kg == 8 && dt != DT_F32) ? 4 : 2; }

// Fail-fast words.  Per candidate slot of the launch table, a block of
// 1 + n_super lines of 128 bytes: line 0 holds the candidate's word (nonzero
// once it is known to have failed), line 1 + m that of super-group m (16
// consecutive stripes).  A work-group that finds a failure claims it in LDS
// (one claim per work-group), then exchanges its super-group's word, and
// only the first of the super-group sets the candidate's word; so each word
// sees at most 16 or n_super writers.  (Stores to one word from every
// work-group that fails at the same moment -- all of them, for a candidate
// that is wrong everywhere -- serialize at the memory and were measured to
// cost more than the whole pass.)  Every word lives on its own line.  A word
// means "failed" only when it holds this call's tag (p.tag), so a value left
// in the workspace by another call is never taken for a failure of this one.
__device__ __forceinline__ uint32_t* ff_word(const ScreenParams& p, int slot, int line) {
    return p.ff_flags + ((size_t)slot * (size_t)(1 + p.n_super) + (size_t)line) * 32u;
}

// Zero the fail-fast words of a candidate group (its finisher, once every
// work-group of the group is past its last poll).
__device__ __forceinline__ void clear_ff_words(const ScreenParams& p, int j0, int kgs) {
    const int lines = 1 + p.n_super;
    for (int i = threadIdx.x; i < kgs * lines; i += kThreads) st_coherent(ff_word(p, j0 + i / lines, i % lines), 0u);
}

// One work-group's part of the screen: candidate group g, element stripe
// `stripe`, then the finish of the group if this work-group is its last.
//
// FF: the fail-fast variant.  Every wave polls its group's candidate words
// with each chunk, and a wave that counts a mismatch publishes it (above).  A
// candidate that failed (here or elsewhere) is no longer loaded or compared
// by the wave, which then keeps, per candidate, the number of elements it
// compared and its sum of r^2 over them, so that the record of a stopped
// candidate describes exactly the elements compared.  The poll is issued
// with the chunk's loads and read at the end of the chunk, when those loads
// have been waited for anyway, so it adds no wait.  A candidate without
// mismatch is never stopped, and all its sums are formed in the same order
// as without FF (the same bits).
//
// LOC: the variant that also finds each candidate's positions (p.loc): the
// first mismatching element and the first elements at which the max abs and
// max rel errors are reached.  Per wave and candidate: the first mismatch is
// searched, after the loop, in the first chunk whose count showed one (the
// wave's chunks come in increasing index order, so later ones can only be
// larger); each lane keeps the chunk in which its max abs error last rose
// (strictly: the first chunk that holds its maximum), and after the loop the
// lanes holding the wave's maximum re-read that chunk for the element; the
// max-rel element is found in the chunk that raises the wave's own maximum.
// The max-rel filter still uses the work-group's shared value, lowered by
// one binary32 step so that elements tying it pass (see the fast path).  A
// wave's own maximum then skips values below the shared one, but every
// element that holds the final maximum passes the filter in its wave, and
// the first of them in the wave is recorded.  The positions are combined
// like the maxima (the smallest index among the parts that hold the
// maximum) in the same fixed orders, so they are the smallest qualifying
// indices whatever the launch.
template <int DT, int KG, bool FF, bool LOC>
__device__ __forceinline__ void screen_part(const ScreenParams& p, const InlineTable& tab, const int g,
                                            const int stripe) {
    static_assert(!(FF && LOC), "positions are not found under fail-fast");
    __shared__ double s_ssd[KG][kThreads];  // lane sums of squared differences
    __shared__ WaveOut s_out[kWaves][KG];
    __shared__ double s_ssr[kWaves];
    __shared__ NonFinite s_nf[kWaves][KG];
    __shared__ uint32_t s_rel[KG];  // work-group max-rel values (binary32 bits)
    __shared__ uint32_t s_arrival;  // this work-group's ticket (0: the workspace was not clean)
    __shared__ double s_sr1;        // single-level finish: the group's sum of r^2
    // fail-fast: per wave and candidate, elements compared and their sum of r^2
    __shared__ uint32_t s_nread[FF ? kWaves : 1][FF ? KG : 1];
    __shared__ double s_ssrc[FF ? kWaves : 1][FF ? KG : 1];
    __shared__ double s_sr1c[FF ? KG : 1];  // single-level finish, per candidate
    __shared__ uint32_t s_told[FF ? KG : 1];  // fail-fast: the work-group knows candidate j failed
    __shared__ uint64_t s_idx[LOC ? kWaves : 1][LOC ? KG : 1][IX_COUNT];  // positions per wave

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int j0 = g * KG;
    const int kg = min(KG, p.n_acc - j0);
    const bool equal_nan = (p.flags & KB_EQUAL_NAN) != 0;
    const float atol = p.atol, rtol = p.rtol;

    // Slots past the accepted candidates (the last group's padding) read the
    // reference, so all KG slots hold a readable tensor; they write no record.
    gbytes cand[KG];
#pragma unroll
    for (int j = 0; j < KG; ++j) {
        const int slot = j0 + j;
        cand[j] = uniform_ptr(slot < p.n_acc ? (p.table_inline ? tab.e[slot].data : p.table[slot].data) : p.ref);
    }
    const gbytes ref = uniform_ptr(p.ref);

    uint32_t mism[KG];  // wave-uniform mismatch counts
    uint32_t amax[KG];  // lane max abs error (binary32 bits, non-negative)
    uint32_t orel[KG];  // wave-uniform max rel error O (binary32 bits, non-negative)
    uint32_t bitdiff = 0u;  // bit j: candidate j differs somewhere in this wave's range
    // positions: bit j set once the wave's first mismatch of candidate j is
    // known (the index itself and that of O live in s_idx: they change
    // rarely, and registers are short)
    uint32_t fm_found = 0u;
    uint32_t achunk[KG];    // positions: the chunk of the lane's max abs error
#pragma unroll
    for (int j = 0; j < KG; ++j) {
        mism[j] = 0u;
        amax[j] = 0u;
        orel[j] = 0u;
        achunk[j] = 0u;
        s_ssd[j][threadIdx.x] = 0.0;
    }
    if (lane < KG) s_nf[wave][lane] = NonFinite{0u, 0u, 0u};
    if (LOC && lane < KG) {
#pragma unroll
        for (int x = 0; x < IX_COUNT; ++x) s_idx[wave][lane][x] = kNone;
    }
    if (threadIdx.x < KG) s_rel[threadIdx.x] = 0u;
    if (FF && threadIdx.x < KG) s_told[threadIdx.x] = 0u;
    double ssr = 0.0;
    // fail-fast state (wave-uniform): candidates still compared, chunks done
    uint32_t alive = (1u << kg) - 1u;
    uint32_t n_done = 0u;
    if constexpr (FF) {
        // candidates that failed before this work-group started are not read
        // at all (work-groups of a group whose candidates have all failed
        // then leave at once, freeing their CU for the others)
        const uint32_t early = (uint32_t)ballot(ld_coherent(ff_word(p, j0 + (lane & (KG - 1)), 0)) == p.tag) & alive;
        if (early != 0u && lane == 0) {
#pragma unroll
            for (int j = 0; j < KG; ++j) {
                if ((early >> j) & 1u) {
                    s_ssrc[wave][j] = 0.0;
                    s_nread[wave][j] = 0u;
                }
            }
        }
        // (kept explicitly wave-uniform: the per-candidate tests must stay
        // scalar branches, and the loads scalar-base loads)
        alive = __builtin_amdgcn_readfirstlane(alive & ~early);
    }
    __syncthreads();

    const uint32_t off = 16u * (uint32_t)lane;
    const uint64_t n_chunks = p.numel / kChunk;
    const uint64_t wstride = (uint64_t)p.blocks_per_group * kWaves;
    const uint64_t first = (uint64_t)stripe * kWaves + wave;
    // Wave priority in stages (plain launch).  Every wave has the same number
    // of chunks (within one), but the SIMD arbiter issues the oldest wave
    // first among waves of equal priority, so on a full device the oldest
    // work-groups of a CU ran ahead and the youngest ended their loops about
    // 40% later (measured per work-group with the real-time clock): the
    // device then spent the last fifth of the pass with ever fewer waves
    // reading.  A wave therefore starts at priority 3 and drops one level
    // after 1/2, 3/4 and 7/8 of its chunks.  A wave that runs ahead yields to
    // every wave not yet as far, the waves regroup at each step, and the
    // spread at the end is that of the last eighth only.  (Measured on the
    // 16 x 4096^2 bf16, 1024 x 256 x 1024 fp32, 64 x 8 x 2048 x 4096 fp16 and
    // 8 x 2^30 fp32 screens: 4.5%, 9%, 3.5% and 3.5% faster.)
    const uint64_t n_mine = first < n_chunks ? (n_chunks - first + wstride - 1) / wstride : 0;
    const uint64_t drop1 = n_mine / 2, drop2 = n_mine * 3 / 4, drop3 = n_mine * 7 / 8;
    uint64_t n_seen = 0;
    if constexpr (!FF) __builtin_amdgcn_s_setprio(3);
    for (uint64_t chunk = first; chunk < n_chunks && (!FF || alive != 0u); chunk += wstride) {
        if constexpr (!FF) {
            if (n_seen == drop1) __builtin_amdgcn_s_setprio(2);
            if (n_seen == drop2) __builtin_amdgcn_s_setprio(1);
            if (n_seen == drop3) __builtin_amdgcn_s_setprio(0);
            ++n_seen;
        }
        const uint64_t cb = chunk * chunk_bytes<DT>();
        // Re-materialise the lane offset inside the loop so that instruction
        // selection sees (scalar base + zero-extended 32-bit offset) and
        // emits scalar-base loads instead of 64-bit vector address adds.
        uint32_t o = off;
        asm volatile("" : "+v"(o));
        // the group's failed words (lane l polls candidate l mod KG)
        uint32_t polled = 0u;
        if constexpr (FF) polled = ld_coherent(ff_word(p, j0 + (lane & (KG - 1)), 0));
        const Raw<DT> rraw = load_chunk<DT, false>(uniform_ptr(ref + cb), o);
        Raw<DT> craw[KG];
#pragma unroll
        for (int j = 0; j < KG; ++j) {
            if constexpr (FF) {
                if (!((alive >> j) & 1u)) continue;
            }
            craw[j] = load_chunk<DT, true>(uniform_ptr(cand[j] + cb), o);
        }
        // the work-group's shared max-rel values
        if constexpr (!LOC) {
#pragma unroll
            for (int j = 0; j < KG; ++j)
                orel[j] = max(orel[j], (uint32_t)__builtin_amdgcn_readfirstlane(s_rel[j]));
        }
        const uint64_t ebase = chunk * kChunk;  // the chunk's first element

        // Reference side, once per element for all KG candidates.
        float r[kE], tol[kE];
        float rr = 0.f;
        uint32_t um = 0xFFFFFFFFu;  // smallest nonzero |r| (guard only)
#pragma unroll
        for (int i = 0; i < kE; ++i) {
            r[i] = elem<DT>(rraw, i);
            tol[i] = __fadd_rn(atol, __fmul_rn(rtol, fabsf(r[i])));
            rr = fmaf(r[i], r[i], rr);
            if constexpr (kGuard<DT>) um = min(um, nz_key(r[i]));
        }
        const float amin_nz = um >= 0xFFFFFFFEu ? __builtin_inff() : __uint_as_float((um + 2u) >> 1);
        // Reference squares: eight binary32 terms, exact in binary64 where
        // the binary32 sum could lose precision (tiny or non-finite).
        double rrd = (double)rr;
        // not in [2^-100, inf), NaN included, as one unsigned compare
        const bool rbad = __float_as_uint(rr) - 0x0D800000u >= 0x7F800000u - 0x0D800000u;
        if (ballot(rbad)) {
            if (rbad) {
                double t = 0.0;
#pragma unroll
                for (int i = 0; i < kE; ++i)
                    if (__builtin_isfinite(r[i])) t = __builtin_fma((double)r[i], (double)r[i], t);
                rrd = t;
            }
        }
        ssr += rrd;

#pragma unroll
        for (int j = 0; j < KG; ++j) {
            // Keep the scheduler from interleaving candidates: interleaving
            // multiplies the live registers, and all the chunk's loads were
            // issued above, so latency hiding is unaffected.
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (FF) {
                if (!((alive >> j) & 1u)) continue;
            }
            const Raw<DT>& cr = craw[j];
            // bitwise identity on raw storage, until a difference is known
            if (!((bitdiff >> j) & 1u)) {
                uint32_t x = 0;
#pragma unroll
                for (int w = 0; w < Raw<DT>::kWords; ++w) x |= cr.w[w] ^ rraw.w[w];
                if (ballot(x != 0u)) bitdiff |= 1u << j;
            }
            // fast path.  O: the max-rel filter's threshold.  Plain: the wave's
            // max, raised by the work-group's shared value.  Positions: the
            // larger of the wave's own max (Own) and the binary32 value just
            // below the shared value -- an element whose quotient ties the
            // shared value must still pass, as its index may be the smallest
            // (a quotient that rounds to t is above the value below t).
            uint32_t obits = orel[j];
            if constexpr (LOC) {
                const uint32_t t = __builtin_amdgcn_readfirstlane(s_rel[j]);
                obits = max(obits, t != 0u ? t - 1u : 0u);
            }
            const float O = __uint_as_float(obits);
            const float Own = __uint_as_float(orel[j]);
            float s[kE], y[kE];
            uint32_t nmatch = 0;
            float tmax = 0.f, acc = 0.f;
#pragma unroll
            for (int i = 0; i < kE; ++i) {
                s[i] = elem<DT>(cr, i) - r[i];
                nmatch += count_within(s[i], tol[i]);
                tmax = fmaxf(tmax, fabsf(s[i]));
                acc = fmaf(s[i], s[i], acc);
                y[i] = fmaf(-O, fabsf(r[i]), fabsf(s[i]));
            }
            float ymax = y[0];
#pragma unroll
            for (int i = 1; i < kE; ++i) ymax = fmaxf(ymax, y[i]);
            if (ballot(!(acc < __builtin_inff()))) {
                // NaN, infinity or a squared difference beyond binary32
                float o = Own;
                const uint32_t mism0 = mism[j];
                float qm;
                uint32_t qs;
                exact_chunk<DT, LOC>(cr, r, atol, rtol, equal_nan, &s_ssd[j][threadIdx.x], mism[j],
                                     amax[j], achunk[j], (uint32_t)chunk, o, s_nf[wave][j], qm, qs);
                if (o > Own) {
                    orel[j] = __float_as_uint(o);
                    if constexpr (LOC)
                        set_idx(&s_idx[wave][j][IX_MAX_REL],
                                ebase + wave_min_u32(qm == o ? slot_offset<DT>(lane, qs) : 0xFFFFFFFFu), lane);
                    publish_rel(&s_rel[j], o, lane);
                }
                if constexpr (LOC) {
                    // the wave's first mismatching chunk (searched after the loop)
                    if (!((fm_found >> j) & 1u) && mism[j] != mism0) {
                        set_idx(&s_idx[wave][j][IX_FIRST_MISMATCH], chunk, lane);
                        fm_found |= 1u << j;
                    }
                }
                continue;
            }
            mism[j] += (uint32_t)kChunk - nmatch;
            if constexpr (LOC) {
                if (!((fm_found >> j) & 1u) && nmatch != (uint32_t)kChunk) {
                    set_idx(&s_idx[wave][j][IX_FIRST_MISMATCH], chunk, lane);
                    fm_found |= 1u << j;
                }
                if (__float_as_uint(tmax) > amax[j]) {
                    amax[j] = __float_as_uint(tmax);
                    achunk[j] = (uint32_t)chunk;
                }
            } else {
                amax[j] = max(amax[j], __float_as_uint(tmax));
            }
            // lanes whose differences are all tiny but not all zero: binary32
            // squares would underflow, so square in binary64
            const bool tiny = (__float_as_uint(tmax) - 1u) < (__float_as_uint(kTiny) - 1u);
            double add = (double)acc;
            if (ballot(tiny)) {
                if (tiny) {
                    double t = 0.0;
#pragma unroll
                    for (int i = 0; i < kE; ++i) t = __builtin_fma((double)s[i], (double)s[i], t);
                    add = t;
                }
            }
            atomicAdd(&s_ssd[j][threadIdx.x], add);
            // the underflow guard as a residual too: 2^-124 - O amin > 0
            // (never while O = 0, where y = d exactly, or for integer O)
            float hz = -__builtin_inff();
            if constexpr (kGuard<DT>)
                hz = fmaf(-O, amin_nz, (O > 0.f && floorf(O) != O) ? 0x1p-124f : -__builtin_inff());
            const bool rel = fmaxf(ymax, hz) > 0.f;
            if (ballot(rel)) {
                float qm = 0.f;
                uint32_t qs = kE;
                if (kGuard<DT> && ballot(hz > 0.f)) {
                    if (rel) qm = rel_quotients<true>(s, r, O, qs);
                } else {
                    if (rel) qm = rel_quotients<false>(s, r, O, qs);
                }
                const float q = wave_max_f(qm);
                if (q > Own) {
                    orel[j] = __float_as_uint(q);
                    if constexpr (LOC)
                        set_idx(&s_idx[wave][j][IX_MAX_REL],
                                ebase + wave_min_u32(qm == q ? slot_offset<DT>(lane, qs) : 0xFFFFFFFFu), lane);
                    publish_rel(&s_rel[j], q, lane);
                }
            }
        }
        if constexpr (FF) {
            // Candidates that failed in this chunk (then set their words) or,
            // by the poll, elsewhere: stop comparing them, keeping what this
            // wave compared (this chunk included).
            ++n_done;
            uint32_t failed = 0u;
#pragma unroll
            for (int j = 0; j < KG; ++j)
                if (mism[j] != 0u) failed |= 1u << j;
            failed &= alive;
            // known failed: by the poll, or by another wave of this work-group
            const uint32_t told = s_told[lane & (KG - 1)];
            const uint32_t seen = (uint32_t)ballot(polled == p.tag || told != 0u) & alive;
            // uniform as far as the compiler can tell too, so that the exit
            // below is a scalar branch and the loop stays uniform
            const uint32_t stop = __builtin_amdgcn_readfirstlane(failed | seen);
            if (stop != 0u) {
                // publish new failures (once per work-group, then once per
                // super-group)
                const uint32_t tell = failed & ~seen;
                if (lane < KG && ((tell >> lane) & 1u)) {
                    if (atomicOr(&s_told[lane], 1u) == 0u &&
                        __hip_atomic_exchange(ff_word(p, j0 + lane, 1 + (stripe >> 4)), p.tag, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT) != p.tag)
                        st_coherent(ff_word(p, j0 + lane, 0), p.tag);
                }
                const double sr = wave_sum_f64(ssr);
                if (lane == 0) {
#pragma unroll
                    for (int j = 0; j < KG; ++j) {
                        if ((stop >> j) & 1u) {
                            s_ssrc[wave][j] = sr;
                            s_nread[wave][j] = n_done * (uint32_t)kChunk;
                        }
                    }
                }
                alive = __builtin_amdgcn_readfirstlane(alive & ~stop);
                if (alive == 0u) break;
            }
        }
    }

    if constexpr (!FF) __builtin_amdgcn_s_setprio(0);

    // Ragged tail: the last numel mod 512 elements, by stripe 0 of each
    // group, one element per thread, exact path (out-of-range lanes and
    // elements 1..7 compare 0 with 0, which changes no statistic).
    uint32_t n_tail = 0u;  // tail elements this wave compared (for every live candidate)
    const uint64_t tfirst = n_chunks * kChunk;
    // positions: candidates whose first mismatch was found in a chunk (the
    // slot holds the chunk number until it is searched, below)
    const uint32_t fm_chunked = fm_found;
    if (stripe == 0) {
        const uint64_t first = tfirst;
        for (uint64_t base = first; base < p.numel; base += kThreads) {
            const uint64_t e = base + threadIdx.x;
            const bool valid = e < p.numel;
            uint32_t rb = 0;
            if (valid) rb = DT == DT_F32 ? ((const uint32_t*)p.ref)[e] : ((const uint16_t*)p.ref)[e];
            if constexpr (FF) n_tail += popc(ballot(valid));
            float r[kE];
            r[0] = widen_bits<DT>(rb);
#pragma unroll
            for (int i = 1; i < kE; ++i) r[i] = 0.f;
            if (__builtin_isfinite(r[0])) ssr = __builtin_fma((double)r[0], (double)r[0], ssr);
#pragma unroll
            for (int j = 0; j < KG; ++j) {
                if (j >= kg) continue;
                if constexpr (FF) {
                    if (!((alive >> j) & 1u)) continue;
                }
                uint32_t cb = 0;
                if (valid)
                    cb = DT == DT_F32 ? ((const __attribute__((address_space(1))) uint32_t*)cand[j])[e]
                                      : ((const __attribute__((address_space(1))) uint16_t*)cand[j])[e];
                if (ballot(cb != rb)) bitdiff |= 1u << j;
                Raw<DT> cr;
#pragma unroll
                for (int w = 0; w < Raw<DT>::kWords; ++w) cr.w[w] = 0u;
                cr.w[0] = cb;
                float o = __uint_as_float(orel[j]);
                const float o0 = o;
                const uint32_t mism0 = mism[j];
                // positions: tail element e is slot 0 of its lane; the max-abs
                // chunk code of the tail is n_chunks + (base - first) / 256
                float qm;
                uint32_t qs;
                exact_chunk<DT, LOC>(cr, r, atol, rtol, equal_nan, &s_ssd[j][threadIdx.x], mism[j],
                                     amax[j], achunk[j], (uint32_t)(n_chunks + (base - first) / kThreads), o,
                                     s_nf[wave][j], qm, qs);
                orel[j] = __float_as_uint(o);
                if constexpr (LOC) {
                    // (the lane's one element is slot 0)
                    if (o > o0) set_idx(&s_idx[wave][j][IX_MAX_REL], wave_min_u64(qm == o ? e : kNone), lane);
                    if (!((fm_found >> j) & 1u) && mism[j] != mism0) {
                        set_idx(&s_idx[wave][j][IX_FIRST_MISMATCH],
                                wave_min_u64(lane_first_mismatch<DT>(cr, r, atol, rtol, equal_nan) < (uint32_t)kE
                                                 ? e
                                                 : kNone),
                                lane);
                        fm_found |= 1u << j;
                    }
                }
            }
        }
    }

    // Positions: the first mismatch of each candidate whose first
    // mismatching chunk of this wave is known, searched in that chunk.
    if constexpr (LOC) {
#pragma unroll
        for (int j = 0; j < KG; ++j) {
            if (j >= kg || !((fm_chunked >> j) & 1u)) continue;
            const uint64_t c = ((uint64_t)__builtin_amdgcn_readfirstlane(
                                   (uint32_t)(s_idx[wave][j][IX_FIRST_MISMATCH] >> 32))
                               << 32) |
                               __builtin_amdgcn_readfirstlane((uint32_t)s_idx[wave][j][IX_FIRST_MISMATCH]);
            const uint64_t cb = c * chunk_bytes<DT>();
            const Raw<DT> cv = load_chunk<DT, false>(uniform_ptr(cand[j] + cb), off);
            const Raw<DT> rv = load_chunk<DT, false>(uniform_ptr(ref + cb), off);
            float rf[kE];
#pragma unroll
            for (int i = 0; i < kE; ++i) rf[i] = elem<DT>(rv, i);
            const uint32_t m =
                wave_min_u32(slot_offset<DT>(lane, lane_first_mismatch<DT>(cv, rf, atol, rtol, equal_nan)));
            set_idx(&s_idx[wave][j][IX_FIRST_MISMATCH], c * kChunk + m, lane);
        }
    }

    // Wave reductions, then the work-group's partials in wave order.
#pragma unroll
    for (int j = 0; j < KG; ++j) {
        if (j >= kg) continue;
        const double sd = wave_sum_f64(s_ssd[j][threadIdx.x]);
        const uint32_t am = wave_max_u32(amax[j]);
        if constexpr (LOC) {
            // the element of the wave's max abs error.  Every element of a
            // chunk lies below every element of a later chunk (and the tail
            // codes follow the chunks in index order), so the smallest index
            // holding the maximum is in the earliest chunk in which a lane
            // first reached it: only the lanes whose first occurrence is in
            // that chunk re-read it -- one chunk, coalesced, however many
            // lanes tie
            uint64_t ai = kNone;
            if (am != 0u) {
                const uint32_t ac = wave_min_u32(amax[j] == am ? achunk[j] : ~0u);
                uint64_t mine = kNone;
                if (amax[j] == am && achunk[j] == ac) {
                    if (ac < n_chunks) {
                        const uint64_t cb = (uint64_t)ac * chunk_bytes<DT>();
                        const Raw<DT> c = load_chunk<DT, false>(uniform_ptr(cand[j] + cb), off);
                        const Raw<DT> rr = load_chunk<DT, false>(uniform_ptr(ref + cb), off);
                        mine = (uint64_t)ac * kChunk + slot_offset<DT>(lane, lane_abs_slot<DT>(c, rr, am));
                    } else {
                        mine = tfirst + (uint64_t)(ac - (uint32_t)n_chunks) * kThreads + threadIdx.x;
                    }
                }
                ai = wave_min_u64(mine);
            }
            if (lane == 0) s_idx[wave][j][IX_MAX_ABS] = ai;
        }
        if (lane == 0) {
            WaveOut& o = s_out[wave][j];
            o.u[PF_MISM] = mism[j];
            o.u[PF_NAN] = s_nf[wave][j].nan;
            o.u[PF_PINF] = s_nf[wave][j].pinf;
            o.u[PF_NINF] = s_nf[wave][j].ninf;
            o.u[PF_MAXABS] = am;
            o.u[PF_MAXREL] = orel[j];
            o.u[PF_BITDIFF] = (bitdiff >> j) & 1u;
            o.ssd = sd;
        }
    }
    {
        const double sr = wave_sum_f64(ssr);
        if (lane == 0) s_ssr[wave] = sr;
        if constexpr (FF) {
            // candidates still compared at the end: everything this wave read
            if (lane == 0) {
#pragma unroll
                for (int j = 0; j < KG; ++j) {
                    if ((alive >> j) & 1u) {
                        s_ssrc[wave][j] = sr;
                        s_nread[wave][j] = n_done * (uint32_t)kChunk + n_tail;
                    }
                }
            }
        }
    }
    __syncthreads();

    const int C = p.blocks_per_group;
    const size_t plane = (size_t)p.n_acc * C;
    const int S = p.n_super;
    const int m = stripe >> 4;
    if (threadIdx.x < kg) {
        const int j = threadIdx.x;
        uint32_t mi = 0, na = 0, pi = 0, ni = 0, ma = 0, mr = 0, bd = 0;
        double sd = 0.0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const WaveOut& o = s_out[w][j];
            mi += o.u[PF_MISM];
            na += o.u[PF_NAN];
            pi += o.u[PF_PINF];
            ni += o.u[PF_NINF];
            ma = max(ma, o.u[PF_MAXABS]);
            mr = max(mr, o.u[PF_MAXREL]);
            bd |= o.u[PF_BITDIFF];
            sd += o.ssd;
        }
        const size_t row = (size_t)(j0 + j) * C + stripe;
        if constexpr (FF) {
            uint32_t nr = 0u;
            double src = 0.0;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                nr += s_nread[w][j];
                src += s_ssrc[w][j];
            }
            st_coherent(&p.part_u32[PF_NREAD * plane + row], nr);
            st_coherent(&p.part_ssrc[row], src);
        }
        if constexpr (LOC) {
            // the smallest index among the waves that hold each maximum
            uint64_t i0 = kNone, i1 = kNone, i2 = kNone;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                i0 = min_u64(i0, s_idx[w][j][IX_FIRST_MISMATCH]);
                if (s_out[w][j].u[PF_MAXABS] == ma) i1 = min_u64(i1, s_idx[w][j][IX_MAX_ABS]);
                if (s_out[w][j].u[PF_MAXREL] == mr) i2 = min_u64(i2, s_idx[w][j][IX_MAX_REL]);
            }
            st_coherent(&p.part_idx[IX_FIRST_MISMATCH * plane + row], i0);
            st_coherent(&p.part_idx[IX_MAX_ABS * plane + row], i1);
            st_coherent(&p.part_idx[IX_MAX_REL * plane + row], i2);
        }
        st_coherent(&p.part_u32[PF_MISM * plane + row], mi);
        st_coherent(&p.part_u32[PF_NAN * plane + row], na);
        st_coherent(&p.part_u32[PF_PINF * plane + row], pi);
        st_coherent(&p.part_u32[PF_NINF * plane + row], ni);
        st_coherent(&p.part_u32[PF_MAXABS * plane + row], ma);
        st_coherent(&p.part_u32[PF_MAXREL * plane + row], mr);
        st_coherent(&p.part_u32[PF_BITDIFF * plane + row], bd);
        st_coherent(&p.part_ssd[row], sd);
    }
    if (threadIdx.x == 0) {
        double sr = 0.0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) sr += s_ssr[w];
        st_coherent(&p.part_ssr[(size_t)g * C + stripe], sr);
    }

    // Two-level finish.  Level 1: the last work-group to arrive in each set
    // of 16 consecutive stripes (a "super-group") combines their partials,
    // one DPP row (16 lanes, one stripe each) per candidate.  Level 2: the
    // last super-group combiner of the candidate group combines the
    // super-group partials (each lane takes super-groups q = lane, lane + 16,
    // ... in order) and writes the records.  A group of at most 16 stripes
    // has one super-group, whose combiner writes the records directly.
    // Fixed orders throughout, so the binary64 sums are the same bits on
    // every call.
    const int msize = min(16, C - 16 * m);
    complete_stores();
    __syncthreads();
    if (threadIdx.x == 0) s_arrival = ticket_arrive(&p.tickets1[(size_t)g * S + m], p.tag);
    __syncthreads();
    if (s_arrival != (uint32_t)msize) {
        if (s_arrival == 0u) report_dirty(p, table_of(p, tab), g, j0, kg);
        return;
    }

    const int jj = threadIdx.x >> 4;
    const int sl = threadIdx.x & 15;
    const CandEntry* table = p.table_inline ? tab.e : p.table;
    {
        const bool have = sl < msize;
        const int s = 16 * m + sl;
        uint64_t mi = 0, na = 0, pi = 0, ni = 0, nr = 0;
        uint32_t ma = 0, mr = 0, bd = 0;
        double sd = 0.0, src = 0.0;
        uint64_t i0 = kNone, i1 = kNone, i2 = kNone;  // positions
        if (jj < kg) {
            const size_t idx = (size_t)(j0 + jj) * C + s;
            if (LOC && have) {
                i0 = ld_coherent(&p.part_idx[IX_FIRST_MISMATCH * plane + idx]);
                i1 = ld_coherent(&p.part_idx[IX_MAX_ABS * plane + idx]);
                i2 = ld_coherent(&p.part_idx[IX_MAX_REL * plane + idx]);
            }
            if (FF && have) {
                nr = ld_coherent(&p.part_u32[PF_NREAD * plane + idx]);
                src = ld_coherent(&p.part_ssrc[idx]);
            }
            if (have) {
                mi = ld_coherent(&p.part_u32[PF_MISM * plane + idx]);
                na = ld_coherent(&p.part_u32[PF_NAN * plane + idx]);
                pi = ld_coherent(&p.part_u32[PF_PINF * plane + idx]);
                ni = ld_coherent(&p.part_u32[PF_NINF * plane + idx]);
                ma = ld_coherent(&p.part_u32[PF_MAXABS * plane + idx]);
                mr = ld_coherent(&p.part_u32[PF_MAXREL * plane + idx]);
                bd = ld_coherent(&p.part_u32[PF_BITDIFF * plane + idx]);
                sd = ld_coherent(&p.part_ssd[idx]);
            }
            mi = row_sum_u64(mi);
            na = row_sum_u64(na);
            pi = row_sum_u64(pi);
            ni = row_sum_u64(ni);
            const uint32_t ma_own = ma, mr_own = mr;
            ma = row_max_u32(ma);
            mr = row_max_u32(mr);
            bd = row_or_u32(bd);
            sd = row_sum_f64(sd);
            if constexpr (LOC) {
                i0 = row_min_u64(i0);
                i1 = row_min_u64(ma_own == ma ? i1 : kNone);
                i2 = row_min_u64(mr_own == mr ? i2 : kNone);
                if (sl == 0 && S > 1) {
                    Part2Idx* q = &p.part2_idx[(size_t)(j0 + jj) * S + m];
                    st_coherent(&q->ix[IX_FIRST_MISMATCH], i0);
                    st_coherent(&q->ix[IX_MAX_ABS], i1);
                    st_coherent(&q->ix[IX_MAX_REL], i2);
                }
            }
            if constexpr (FF) {
                nr = row_sum_u64(nr);
                src = row_sum_f64(src);
                if (sl == 0 && S > 1) {
                    Part2* q = &p.part2[(size_t)(j0 + jj) * S + m];
                    st_coherent(&q->nread, nr);
                    st_coherent(&q->ssr, src);
                }
                if (sl == 0 && S == 1) s_sr1c[jj] = src;
            }
            if (sl == 0 && S > 1) {
                Part2* q = &p.part2[(size_t)(j0 + jj) * S + m];
                st_coherent(&q->mism, mi);
                st_coherent(&q->nan, na);
                st_coherent(&q->pinf, pi);
                st_coherent(&q->ninf, ni);
                st_coherent(&q->maxabs, ma);
                st_coherent(&q->maxrel, mr);
                st_coherent(&q->bitdiff, bd);
                st_coherent(&q->ssd, sd);
            }
        }
        if (jj == 0) {
            double sr = have ? ld_coherent(&p.part_ssr[(size_t)g * C + s]) : 0.0;
            sr = row_sum_f64(sr);
            if (sl == 0) {
                if (S > 1) st_coherent(&p.part2_ssr[(size_t)g * S + m], sr);
                else s_sr1 = sr;
            }
        }
        if (S == 1) {
            // Single-level finish: the group has at most 16 stripes, and this
            // work-group has combined all of them.
            __syncthreads();
            if (jj < kg && sl == 0) {
                if constexpr (FF)
                    write_record(&p.stats[table[j0 + jj].index], nr, mi, na, pi, ni, ma, mr, bd, sd,
                                 s_sr1c[jj]);
                else
                    write_record(&p.stats[table[j0 + jj].index], p.numel, mi, na, pi, ni, ma, mr, bd,
                                 sd, s_sr1);
                if constexpr (LOC) write_loc(&p.loc[table[j0 + jj].index], i0, i1, i2);
            }
            if (g == 0) write_rejected(p, table);
            if (threadIdx.x == 0) st_coherent(&p.tickets1[(size_t)g * S + m], (uint64_t)0);
            if constexpr (FF) clear_ff_words(p, j0, KG);
            return;
        }
    }
    if (threadIdx.x == 0) st_coherent(&p.tickets1[(size_t)g * S + m], (uint64_t)0);

    complete_stores();
    __syncthreads();
    if (threadIdx.x == 0) s_arrival = ticket_arrive(&p.tickets2[g], p.tag);
    __syncthreads();
    if (s_arrival != (uint32_t)S) {
        if (s_arrival == 0u) report_dirty(p, table, g, j0, kg);
        return;
    }

    if (jj < kg) {
        uint64_t mi = 0, na = 0, pi = 0, ni = 0, nr = 0;
        uint32_t ma = 0, mr = 0, bd = 0;
        double sd = 0.0, sr = 0.0, src = 0.0;
        uint64_t i0 = kNone, i1 = kNone, i2 = kNone;  // positions
        const Part2* row = p.part2 + (size_t)(j0 + jj) * S;
        const double* rs = p.part2_ssr + (size_t)g * S;
        // U super-groups per lane in flight (fewer with positions, whose
        // partials are larger: this loop sets the kernel's register peak);
        // either way each lane adds its super-groups in increasing order
        constexpr int U = LOC ? 2 : 4;
        for (int q0 = sl; q0 < S; q0 += 16 * U) {
            Part2 v[U];
            double w[U];
            Part2Idx vi[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = q0 + 16 * u;
                if (FF && q < S) {
                    nr += ld_coherent(&row[q].nread);
                    src += ld_coherent(&row[q].ssr);
                }
                if (q < S) {
                    const Part2* e = &row[q];
                    v[u].mism = ld_coherent(&e->mism);
                    v[u].nan = ld_coherent(&e->nan);
                    v[u].pinf = ld_coherent(&e->pinf);
                    v[u].ninf = ld_coherent(&e->ninf);
                    v[u].maxabs = ld_coherent(&e->maxabs);
                    v[u].maxrel = ld_coherent(&e->maxrel);
                    v[u].bitdiff = ld_coherent(&e->bitdiff);
                    v[u].ssd = ld_coherent(&e->ssd);
                    w[u] = ld_coherent(&rs[q]);
                } else {
                    v[u] = Part2{0, 0, 0, 0, 0u, 0u, 0u, 0u, 0.0, 0, 0.0};
                    w[u] = 0.0;
                }
                if constexpr (LOC) {
                    const Part2Idx* e = &p.part2_idx[(size_t)(j0 + jj) * S + q];
#pragma unroll
                    for (int x = 0; x < IX_COUNT; ++x) vi[u].ix[x] = q < S ? ld_coherent(&e->ix[x]) : kNone;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if constexpr (LOC) {
                    // (value, smallest index) pairs, before the maxima move
                    i0 = min_u64(i0, vi[u].ix[IX_FIRST_MISMATCH]);
                    i1 = v[u].maxabs > ma ? vi[u].ix[IX_MAX_ABS]
                                          : v[u].maxabs == ma ? min_u64(i1, vi[u].ix[IX_MAX_ABS]) : i1;
                    i2 = v[u].maxrel > mr ? vi[u].ix[IX_MAX_REL]
                                          : v[u].maxrel == mr ? min_u64(i2, vi[u].ix[IX_MAX_REL]) : i2;
                }
                mi += v[u].mism;
                na += v[u].nan;
                pi += v[u].pinf;
                ni += v[u].ninf;
                ma = max(ma, v[u].maxabs);
                mr = max(mr, v[u].maxrel);
                bd |= v[u].bitdiff;
                sd += v[u].ssd;
                sr += w[u];
            }
        }
        mi = row_sum_u64(mi);
        na = row_sum_u64(na);
        pi = row_sum_u64(pi);
        ni = row_sum_u64(ni);
        const uint32_t ma_own = ma, mr_own = mr;
        ma = row_max_u32(ma);
        mr = row_max_u32(mr);
        bd = row_or_u32(bd);
        sd = row_sum_f64(sd);
        sr = row_sum_f64(sr);
        if constexpr (LOC) {
            i0 = row_min_u64(i0);
            i1 = row_min_u64(ma_own == ma ? i1 : kNone);
            i2 = row_min_u64(mr_own == mr ? i2 : kNone);
            if (sl == 0) write_loc(&p.loc[table[j0 + jj].index], i0, i1, i2);
        }
        if constexpr (FF) {
            nr = row_sum_u64(nr);
            src = row_sum_f64(src);
            if (sl == 0)
                write_record(&p.stats[table[j0 + jj].index], nr, mi, na, pi, ni, ma, mr, bd, sd, src);
        } else {
            if (sl == 0)
                write_record(&p.stats[table[j0 + jj].index], p.numel, mi, na, pi, ni, ma, mr, bd, sd,
                             sr);
        }
    }
    // Group 0's finisher also writes the rejected candidates' records.
    if (g == 0) write_rejected(p, table);
    // Leave the ticket and the failed words at zero (every work-group of the
    // group has finished reading them): the next call on this workspace then
    // finds them clean even if its tag happens to equal this call's.
    if (threadIdx.x == 0) st_coherent(&p.tickets2[g], (uint64_t)0);
    if constexpr (FF) clear_ff_words(p, j0, KG);
}

// Work-group id -> (candidate group, stripe).  Ids are dealt round robin to
// the 8 XCDs: id -> (XCD, slot), slot -> (group, stripe group), so that the
// groups of one stripe run on one XCD and find the reference stripe in its
// L2.
// FF = false: one persistent round over all groups.
// FF = true: the groups are taken in rounds of p.ff_round groups, each round
// over all stripes, and the grid is sized so that a round fills the device.
// Work-groups are dispatched in id order, so the device works through the
// rounds one after another; the work-groups of a group whose candidates are
// already known to have failed leave at their first poll, and the
// dispatcher fills their place with the next ones.  (With one persistent
// round the work-groups of failed groups would idle while those of the live
// ones did all their work.)  Fewer groups per round re-read the reference
// once more per round; more groups per round balance less well.
// WIDE: the same kernel built for 5 waves per SIMD instead of 4 (only fp32
// with 4 candidates per group, plain launches on large tensors; see
// use_wide_kernel).  LOC: the variant that also finds the positions.
template <int DT, int KG, bool FF, bool WIDE, bool LOC>
__global__ __launch_bounds__(kThreads, WIDE ? 5 : min_waves(DT, KG)) void screen_kernel(
    ScreenParams p, InlineTable tab) {
    int id = blockIdx.x, g0 = 0, R = p.n_groups;
    if constexpr (FF) {
        const int per_round = p.ff_round * p.blocks_per_group;
        const int r = id / per_round;
        g0 = r * p.ff_round;
        id -= r * per_round;
        R = min(p.ff_round, p.n_groups - g0);
    }
    const int xcd = id & 7;
    const int slot = id >> 3;
    screen_part<DT, KG, FF, LOC>(p, tab, g0 + slot % R, (slot / R) * 8 + xcd);
}

__global__ void records_only_kernel(const CandEntry* uploaded, InlineTable tab, int table_inline,
                                    int n_table, uint64_t numel, kb_stats* stats, kb_locate* loc) {
    const CandEntry* table = table_inline ? tab.e : uploaded;
    for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n_table; k += gridDim.x * blockDim.x) {
        if (table[k].index < 0) continue;  // padding
        kb_stats st = {};
        st.status = table[k].status;
        if (st.status == KB_STATUS_OK) {
            st.numel = numel;  // numel == 0 here
            st.bitwise_equal = 1;
        }
        stats[table[k].index] = st;
        if (loc) write_loc(&loc[table[k].index], kNone, kNone, kNone);
    }
}

// Variants: 0 plain, 1 fail-fast, 2 positions.
enum Variant : int { V_PLAIN = 0, V_FF, V_LOC };

template <int DT, int KG, int V>
hipError_t launch_kg(const ScreenPlan& plan, const ScreenParams& p, const InlineTable& tab,
                     hipStream_t stream) {
    constexpr bool FF = V == V_FF, LOC = V == V_LOC;
    const unsigned grid = (unsigned)plan.n_groups * (unsigned)plan.blocks_per_group;
    if constexpr (DT == DT_F32 && KG == 4 && V == V_PLAIN) {
        if (plan.wide) {
            hipLaunchKernelGGL((screen_kernel<DT, KG, false, true, false>), dim3(grid), dim3(kThreads), 0,
                               stream, p, tab);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((screen_kernel<DT, KG, FF, false, LOC>), dim3(grid), dim3(kThreads), 0, stream, p, tab);
    return hipGetLastError();
}

template <int DT, int KG, int V, bool WIDE = false>
int occupancy_kg() {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &n, screen_kernel<DT, KG, V == V_FF, WIDE, V == V_LOC>, kThreads, 0) != hipSuccess)
        return 0;
    return n;
}

template <int DT, int V>
int occupancy_dt(int kg) {
    switch (kg) {
        case 1: return occupancy_kg<DT, 1, V>();
        case 2: return occupancy_kg<DT, 2, V>();
        case 4: return occupancy_kg<DT, 4, V>();
        case 8: return occupancy_kg<DT, 8, V>();
        default: return occupancy_kg<DT, 16, V>();
    }
}

template <int DT, int V>
hipError_t launch_dt(const ScreenPlan& plan, const ScreenParams& p, const InlineTable& tab,
                     hipStream_t stream) {
    switch (plan.kg) {
        case 1: return launch_kg<DT, 1, V>(plan, p, tab, stream);
        case 2: return launch_kg<DT, 2, V>(plan, p, tab, stream);
        case 4: return launch_kg<DT, 4, V>(plan, p, tab, stream);
        case 8: return launch_kg<DT, 8, V>(plan, p, tab, stream);
        default: return launch_kg<DT, 16, V>(plan, p, tab, stream);
    }
}

template <int V>
hipError_t launch_v(const ScreenPlan& plan, const ScreenParams& p, const InlineTable& tab,
                    hipStream_t stream) {
    switch (plan.dtype) {
        case DT_F32: return launch_dt<DT_F32, V>(plan, p, tab, stream);
        case DT_F16: return launch_dt<DT_F16, V>(plan, p, tab, stream);
        default: return launch_dt<DT_BF16, V>(plan, p, tab, stream);
    }
}

template <int V>
int occupancy(int dtype, int kg) {
    return dtype == DT_F32 ? occupancy_dt<DT_F32, V>(kg)
                           : dtype == DT_F16 ? occupancy_dt<DT_F16, V>(kg) : occupancy_dt<DT_BF16, V>(kg);
}

}  // namespace

hipError_t launch_screen(const ScreenPlan& plan, const ScreenParams& p, const InlineTable& tab,
                         bool fail_fast, bool loc, hipStream_t stream) {
    if (fail_fast && loc) return hipErrorInvalidValue;
    return fail_fast ? launch_v<V_FF>(plan, p, tab, stream)
                     : loc ? launch_v<V_LOC>(plan, p, tab, stream) : launch_v<V_PLAIN>(plan, p, tab, stream);
}

__global__ void zero_fill_kernel(uint4* dst, uint64_t n16) {
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16;
         i += (uint64_t)gridDim.x * blockDim.x)
        dst[i] = make_uint4(0u, 0u, 0u, 0u);
}

hipError_t launch_zero_fill(void* dst, size_t n, hipStream_t stream) {
    // the workspace size is always a multiple of 256 bytes
    const uint64_t n16 = n / 16;
    if (n16 == 0) return hipSuccess;
    const uint64_t want = (n16 + 255) / 256;
    const unsigned grid = (unsigned)(want < 4096 ? want : 4096);
    hipLaunchKernelGGL(zero_fill_kernel, dim3(grid), dim3(256), 0, stream, (uint4*)dst, n16);
    return hipGetLastError();
}

int screen_blocks_per_cu(int dtype, int kg, bool fail_fast, bool wide, bool loc) {
    // The occupancy of a kernel does not change during the process.
    static int cache[4][3][5] = {};  // value + 1, 0 = not queried yet
    const int ki = kg == 1 ? 0 : kg == 2 ? 1 : kg == 4 ? 2 : kg == 8 ? 3 : 4;
    const int di = dtype == DT_F32 ? 0 : dtype == DT_F16 ? 1 : 2;
    if (fail_fast && loc) return 0;
    wide = wide && use_wide_kernel(dtype, kg, fail_fast, ~0ull, loc);
    int* slot = &cache[fail_fast ? 1 : wide ? 2 : loc ? 3 : 0][di][ki];
    int v = __atomic_load_n(slot, __ATOMIC_RELAXED) - 1;
    if (v < 0) {
        v = wide ? occupancy_kg<DT_F32, 4, V_PLAIN, true>()
                 : fail_fast ? occupancy<V_FF>(dtype, kg) : loc ? occupancy<V_LOC>(dtype, kg)
                                                                : occupancy<V_PLAIN>(dtype, kg);
        __atomic_store_n(slot, v + 1, __ATOMIC_RELAXED);
    }
    return v;
}

hipError_t launch_records_only(const CandEntry* table, const InlineTable& tab, int table_inline,
                               int n_table, uint64_t numel, kb_stats* stats, kb_locate* loc,
                               hipStream_t stream) {
    const int grid = (n_table + 255) / 256;
    hipLaunchKernelGGL(records_only_kernel, dim3(grid), dim3(256), 0, stream, table, tab,
                       table_inline, n_table, numel, stats, loc);
    return hipGetLastError();
}

}  // namespace kb
