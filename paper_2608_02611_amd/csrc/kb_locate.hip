// kb_locate.hip -- positions of the first mismatch and of the maxima.
//
// The detail a failed candidate's feedback carries (the agent passes the log
// of the failing check to the next generation step, Section 3.4 and the
// prompt template of the appendix): per candidate, the smallest element
// index that does not match, whose |c - r| equals the candidate's max abs
// error, and whose d / |r| equals its max rel error.  The maxima come from
// the records kb_screen wrote, so this is a second, optional pass over the
// candidates one asks about.
//
// A wave scans its chunks in increasing index order and stops looking for a
// position as soon as one of its lanes has found it: every later chunk of
// the wave holds larger indices.  On a failing candidate the first mismatch
// is usually in a wave's first chunk.  Each wave loads two chunks ahead of
// the two it scans.  A cheap, branch-free pass takes per lane the maxima of
// three filters over its elements (the mismatch filter, d against max abs,
// the max-rel filter) and one wave ballot of each; a chunk with a hit is
// evaluated again from the definitions into 8-bit lane masks, and its index
// formed (the lane's lowest set bit, then a wave minimum by DPP).  The wave's finds are merged into
// the output with a 64-bit atomic minimum ("none" is all-ones, which reads
// as -1).  Work-group ids are mapped like the screen's, so that the
// candidates of one stripe run on one XCD and share the reference stripe in
// its L2.
#include "kb_device.hpp"
#include "kb_internal.hpp"

namespace kb {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kE = 8;
constexpr int kChunk = 64 * kE;
constexpr uint64_t kNone = ~0ull;

typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) v4u32* gvec;

template <int DT>
__device__ __forceinline__ float widen_bits(uint32_t bits) {
    if constexpr (DT == DT_F32) return __uint_as_float(bits);
    else if constexpr (DT == DT_F16) return f16_bits_to_f32(bits);
    else return bf16_bits_to_f32(bits);
}

// Storage bits of element i of a lane's chunk and its index within the chunk
// (fp32: elements 4l..4l+3 and 256+4l..256+4l+3; 16-bit: 8l..8l+7; both in
// increasing index order in i).
template <int DT>
struct LaneChunk {
    uint32_t w[DT == DT_F32 ? 8 : 4];
    __device__ __forceinline__ uint32_t bits(int i) const {
        if constexpr (DT == DT_F32) return w[i];
        else return (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu;
    }
    static __device__ __forceinline__ uint32_t offset(int lane, int i) {
        if constexpr (DT == DT_F32) return i < 4 ? 4 * lane + i : 256 + 4 * lane + (i - 4);
        else return 8 * lane + i;
    }
};

// One lane's part of chunk `chunk` of a tensor: base is wave-uniform (scalar
// registers), off = 16 * lane, so a load is a scalar base plus the lane's
// 32-bit offset.  NT marks the loads nontemporal: each candidate byte is
// read once, while the reference chunk is re-read by the work-groups of the
// stripe's other candidates, which run on the same XCD, and should stay in
// its L2.
template <int DT, bool NT = true>
__device__ __forceinline__ LaneChunk<DT> load_lane(const char* base, uint64_t chunk, uint32_t off) {
    LaneChunk<DT> x;
    typedef const __attribute__((address_space(1))) char* gbytes;
    const gbytes c = (gbytes)base + chunk * (DT == DT_F32 ? 2048u : 1024u);
    uint32_t o = off;
    asm volatile("" : "+v"(o));
    const v4u32 a = NT ? __builtin_nontemporal_load((gvec)(c + o)) : *(gvec)(c + o);
    x.w[0] = a.x; x.w[1] = a.y; x.w[2] = a.z; x.w[3] = a.w;
    if constexpr (DT == DT_F32) {
        const v4u32 b = NT ? __builtin_nontemporal_load((gvec)(c + o + 1024u)) : *(gvec)(c + o + 1024u);
        x.w[4] = b.x; x.w[5] = b.y; x.w[6] = b.z; x.w[7] = b.w;
    }
    return x;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
    v = min(v, dpp_u64<DPP_QUAD_XOR1>(v));
    v = min(v, dpp_u64<DPP_QUAD_XOR2>(v));
    v = min(v, dpp_u64<DPP_ROW_HALF_MIRROR>(v));
    v = min(v, dpp_u64<DPP_ROW_MIRROR>(v));
    return min(min(readlane_u64(v, 0), readlane_u64(v, 16)), min(readlane_u64(v, 32), readlane_u64(v, 48)));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) { return ~wave_max_u32(~v); }

// The smallest in-chunk index among the elements of this lane whose bit is
// set in m (bit i = element i of the lane), or all-ones if none.
template <int DT>
__device__ __forceinline__ uint32_t first_in_lane(uint32_t m, int lane) {
    if (m == 0u) return ~0u;
    if constexpr (DT == DT_F32) {
        // elements 0..3 are 4l..4l+3, elements 4..7 are 256+4l..256+4l+3
        return (m & 0xFu) ? 4u * lane + __builtin_ctz(m) : 256u + 4u * lane + __builtin_ctz(m >> 4);
    } else {
        return 8u * lane + __builtin_ctz(m);
    }
}

// The three predicates of one element (the definitions of the screening
// statistics, element by element).
struct Hit {
    bool mism, abs, rel;
};
__device__ __forceinline__ Hit classify(float c, float r, float atol, float rtol, bool equal_nan,
                                        float max_abs, float max_rel, bool want_abs, bool want_rel) {
    const float d = fabsf(c - r);
    const float a = fabsf(r);
    const float tol = __builtin_isfinite(r) ? __fadd_rn(atol, __fmul_rn(rtol, a)) : -1.0f;
    const bool match = (c == r) || (d <= tol) || (equal_nan && __builtin_isnan(c) && __builtin_isnan(r));
    Hit h;
    h.mism = !match;
    h.abs = want_abs && d == max_abs;
    h.rel = false;
    if (want_rel) {
        // fl(d / a) == max_rel needs d / a >= max_rel (1 - 2^-24), hence
        // d - T a > 0 for T = fl(max_rel (1 - 2^-20)): a cheap filter in
        // front of the IEEE division (the fma keeps the sign; an underflow to
        // zero passes).  For max_rel = +inf: a zero reference, an infinite
        // difference or a quotient beyond 2^100; for a tiny max_rel, whose
        // product T might round back up to it, no filter.
        bool cand;
        if (__builtin_isinf(max_rel)) cand = a == 0.f || d == __builtin_inff() || d >= a * 0x1p100f;
        else if (max_rel < 0x1p-100f) cand = true;
        else cand = fmaf(-(max_rel * 0x1.ffffep-1f), a, d) >= 0.f;
        if (cand) h.rel = (d / a) == max_rel;
    }
    return h;
}

// One chunk's cheap pass: per lane, maxima over its elements, then one wave
// ballot per predicate; a nonzero ballot sends the wave to the exact pass.
// Each filter lets through every element the definition accepts (and some
// it rejects), with no branch and no scalar work per element:
//
//  * mismatch (M: still looked for): the NaN-propagating maximum of
//    fl(d - tol).  For finite d and tol, fl(d - tol) > 0 exactly when
//    d > tol (a difference of two binary32 values rounds to zero only when
//    it is zero); not (d <= tol) with an infinite or NaN operand gives +inf
//    or NaN, and so does a reference that is not finite (d is then NaN or
//    infinite, tol infinite or NaN), which the exact pass decides.  So a
//    lane whose maximum is positive or NaN may hold a mismatch, and one
//    whose maximum is <= 0 holds none (d <= tol, a match);
//  * max abs: the maximum of d (NaN ignored) >= max_abs; an element with
//    d == max_abs makes it so;
//  * max rel: the maximum (NaN ignored) of fma(-T, |r|, d) >= 0, with T per
//    candidate (rel_threshold): fl(d / a) == max_rel needs d >= T a.
struct AnyHits {
    uint64_t m, a, r;
};

// T of the max-rel filter.  A finite max_rel >= 2^-100: fl(d / a) ==
// max_rel needs d / a >= max_rel (1 - 2^-24), so d - T a > 0 for T =
// fl(max_rel (1 - 2^-20)) (the fma keeps the sign; an underflow to zero
// passes).  max_rel = +inf: the quotient overflows, or a is zero, or d is
// infinite; each gives d - 2^100 a >= 0 (exact inside the fma) or a NaN
// that the definition rejects too (inf / inf).  max_rel < 2^-100, where T
// might round back up to max_rel: T = 0 lets every element with a finite
// reference through.
__device__ __forceinline__ float rel_threshold(float max_rel) {
    if (__builtin_isinf(max_rel)) return 0x1p100f;
    if (max_rel < 0x1p-100f) return 0.f;
    return max_rel * 0x1.ffffep-1f;
}

template <int DT, bool M>
__device__ __forceinline__ AnyHits cheap_pass(const LaneChunk<DT>& rc, const LaneChunk<DT>& cc, float atol,
                                              float rtol, float max_abs, float T) {
    float ta = 0.f, tr = 0.f;  // (set from the first pair)
#pragma unroll
    for (int i = 0; i < kE; i += 2) {
        float d[2], x[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const float r = widen_bits<DT>(rc.bits(i + j));
            d[j] = fabsf(widen_bits<DT>(cc.bits(i + j)) - r);
            x[j] = fmaf(-T, fabsf(r), d[j]);
        }
        ta = i == 0 ? fmaxf(d[0], d[1]) : fmaxf(ta, fmaxf(d[0], d[1]));
        tr = i == 0 ? fmaxf(x[0], x[1]) : fmaxf(tr, fmaxf(x[0], x[1]));
    }
    AnyHits h;
    h.m = 0u;
    h.a = ballot(ta >= max_abs);
    h.r = ballot(tr >= 0.f);
    if constexpr (M) {
        // (the words pass through an empty asm, so that this pass widens
        // them again instead of keeping the values above live: it runs only
        // until a wave has found its mismatch, and would otherwise set the
        // kernel's register peak)
        LaneChunk<DT> rx = rc, cx = cc;
#pragma unroll
        for (int k = 0; k < (DT == DT_F32 ? 8 : 4); ++k) asm volatile("" : "+v"(rx.w[k]), "+v"(cx.w[k]));
        float tm = 0.f;
#pragma unroll
        for (int i = 0; i < kE; i += 2) {
            float x[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const float r = widen_bits<DT>(rx.bits(i + j));
                x[j] = fabsf(widen_bits<DT>(cx.bits(i + j)) - r) - __fadd_rn(atol, __fmul_rn(rtol, fabsf(r)));
            }
            const float y = __builtin_elementwise_maximum(x[0], x[1]);
            tm = i == 0 ? y : __builtin_elementwise_maximum(tm, y);
        }
        h.m = ballot(!(tm <= 0.f));
    }
    return h;
}

// A pointer made explicitly wave-uniform (held in scalar registers), so that
// a load is a scalar base plus the lane's 32-bit offset.
__device__ __forceinline__ const char* uniform_base(const void* p) {
    const uint64_t v = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (const char*)(((uint64_t)hi << 32) | lo);
}

// Waves per SIMD the kernel is built for: fp32 needs 96 registers for 5;
// bf16 fits 8 either way, and the bound measured faster (its schedule);
// the fp16 build would spill scalar registers under an 8-wave bound, which
// measured slower than its 7 waves.
constexpr int locate_min_waves(int dt) { return dt == DT_F32 ? 5 : dt == DT_BF16 ? 8 : 1; }

template <int DT>
__global__ __launch_bounds__(kThreads, locate_min_waves(DT)) void locate_kernel(LocateParams p, LocTable tab) {
    const int lane = threadIdx.x & 63;
    // (explicitly wave-uniform, so that the chunk index, the loads' bases and
    // the per-chunk choices stay in scalar registers and branches)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int xcd = blockIdx.x & 7;  // p.stripes is a multiple of 8
    const int slot = blockIdx.x >> 3;
    const int k = slot % p.n;
    const int stripe = (slot / p.n) * 8 + xcd;
    const char* cand = uniform_base(tab.e[k].data);
    const char* ref = uniform_base(p.ref);
    const int index = tab.e[k].index;
    // the record's fields, made explicitly wave-uniform (they are loaded by
    // every lane from the same address)
    const float max_abs = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(p.stats[index].max_abs_err)));
    const float max_rel = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(p.stats[index].max_rel_err)));
    const bool has_mism = __builtin_amdgcn_readfirstlane(p.stats[index].mismatches > 0 ? 1 : 0) != 0;
    const bool want_abs = max_abs > 0.f;  // false for 0 and NaN
    const bool want_rel = max_rel > 0.f;
    const bool equal_nan = (p.flags & KB_EQUAL_NAN) != 0;
    const float T = rel_threshold(max_rel);

    // the wave's finds (wave-uniform), all-ones until found; a candidate
    // whose record counts no mismatch has none to look for (the record was
    // written by the screen under the same tolerances and flags)
    uint64_t f_mism = kNone, f_abs = kNone, f_rel = kNone;
    bool need_mism = has_mism, need_abs = want_abs, need_rel = want_rel;
    const uint64_t n_chunks = p.numel / kChunk;
    const uint64_t wstride = (uint64_t)p.stripes * kWaves;
    const uint32_t off = 16u * (uint32_t)lane;
    // One chunk: the cheap pass, and the exact pass when a ballot is set.
    auto scan = [&](uint64_t chunk, const LaneChunk<DT>& rc, const LaneChunk<DT>& cc) {
        // (readfirstlane: the choice of variant is a scalar branch)
        const AnyHits h = __builtin_amdgcn_readfirstlane(need_mism ? 1 : 0)
                              ? cheap_pass<DT, true>(rc, cc, p.atol, p.rtol, max_abs, T)
                              : cheap_pass<DT, false>(rc, cc, p.atol, p.rtol, max_abs, T);
        const uint64_t any_m = h.m, any_a = need_abs ? h.a : 0u, any_r = need_rel ? h.r : 0u;
        if ((any_m | any_a | any_r) == 0) return;
        // Exact pass (rare): the definitions, element by element, into 8-bit
        // lane masks (bit i: element i of this lane qualifies); a position
        // found anywhere in this chunk is below everything later.
        // (the chunk's words pass through an empty asm, so that the widened
        // values of the cheap pass are not kept live for this rare path)
        LaneChunk<DT> rx = rc, cx = cc;
#pragma unroll
        for (int k = 0; k < (DT == DT_F32 ? 8 : 4); ++k) asm volatile("" : "+v"(rx.w[k]), "+v"(cx.w[k]));
        uint32_t mm = 0u, ma = 0u, mr = 0u;
#pragma unroll
        for (int i = 0; i < kE; ++i) {
            const Hit h = classify(widen_bits<DT>(cx.bits(i)), widen_bits<DT>(rx.bits(i)), p.atol, p.rtol,
                                   equal_nan, max_abs, max_rel, any_a != 0, any_r != 0);
            mm |= (uint32_t)h.mism << i;
            ma |= (uint32_t)h.abs << i;
            mr |= (uint32_t)h.rel << i;
        }
        const uint64_t base = chunk * kChunk;
        // (every filter lets through elements that the definitions then
        // reject -- the max-abs one all d above max_abs: a position only if
        // a lane confirmed one)
        if (any_m != 0 && ballot(mm != 0u)) {
            f_mism = base + wave_min_u32(first_in_lane<DT>(mm, lane));
            need_mism = false;
        }
        if (any_a != 0 && ballot(ma != 0u)) {
            f_abs = base + wave_min_u32(first_in_lane<DT>(ma, lane));
            need_abs = false;
        }
        if (any_r != 0 && ballot(mr != 0u)) {
            f_rel = base + wave_min_u32(first_in_lane<DT>(mr, lane));
            need_rel = false;
        }
    };
    // Software pipeline, two chunks deep: the next two chunks of the wave's
    // range are loaded before the current two are scanned, so the scan
    // order (and the early exit) is the wave's chunk order.  A load past the
    // wave's last chunk is redirected to a chunk the wave reads anyway (every
    // index stays inside the tensor), and its data is not scanned.
    uint64_t chunk = (uint64_t)stripe * kWaves + wave;
    if (chunk < n_chunks) {
        // Priority: 3 until the last eighth of the wave's chunk pairs, then
        // 0, so that in the last eighth the waves still behind are issued
        // first (among equal priorities the arbiter favours the oldest
        // wave).  Measured: 64 fp16 candidates of 2^26 elements 10%
        // faster, 16 bf16 of 2^24 and 8 fp32 of 2^27 unchanged, 1024 fp32
        // of 2^18 1.5% slower; the screen's three-step schedule cost the
        // 16 bf16 candidates 7-17% here.
        const uint64_t n_it = (n_chunks - chunk + 2 * wstride - 1) / (2 * wstride);
        const uint64_t drop = n_it * 7 / 8;
        uint64_t n_seen = 0;
        __builtin_amdgcn_s_setprio(3);
        const uint64_t c1 = chunk + wstride < n_chunks ? chunk + wstride : chunk;
        LaneChunk<DT> ra = load_lane<DT, false>(ref, chunk, off);
        LaneChunk<DT> ca = load_lane<DT>(cand, chunk, off);
        LaneChunk<DT> rb = load_lane<DT, false>(ref, c1, off);
        LaneChunk<DT> cb = load_lane<DT>(cand, c1, off);
        for (; chunk < n_chunks && (need_mism || need_abs || need_rel); chunk += 2 * wstride) {
            if (n_seen++ == drop) __builtin_amdgcn_s_setprio(0);
            const uint64_t n0 = chunk + 2 * wstride, n1 = chunk + 3 * wstride;
            const uint64_t l0 = n0 < n_chunks ? n0 : chunk, l1 = n1 < n_chunks ? n1 : chunk;
            const LaneChunk<DT> rn0 = load_lane<DT, false>(ref, l0, off);
            const LaneChunk<DT> cn0 = load_lane<DT>(cand, l0, off);
            const LaneChunk<DT> rn1 = load_lane<DT, false>(ref, l1, off);
            const LaneChunk<DT> cn1 = load_lane<DT>(cand, l1, off);
            scan(chunk, ra, ca);
            if (chunk + wstride < n_chunks && (need_mism || need_abs || need_rel)) scan(chunk + wstride, rb, cb);
            ra = rn0;
            ca = cn0;
            rb = rn1;
            cb = cn1;
        }
    }
    __builtin_amdgcn_s_setprio(0);
    // Ragged tail (numel mod 512 elements): stripe 0, one element per thread.
    if (stripe == 0) {
        for (uint64_t e = n_chunks * kChunk + threadIdx.x; e < p.numel; e += kThreads) {
            const uint32_t rb = DT == DT_F32 ? ((const uint32_t*)p.ref)[e] : ((const uint16_t*)p.ref)[e];
            const uint32_t cb = DT == DT_F32 ? ((const uint32_t*)cand)[e] : ((const uint16_t*)cand)[e];
            const Hit h = classify(widen_bits<DT>(cb), widen_bits<DT>(rb), p.atol, p.rtol, equal_nan,
                                   max_abs, max_rel, want_abs, want_rel);
            if (h.mism && f_mism == kNone) f_mism = e;
            if (h.abs && f_abs == kNone) f_abs = e;
            if (h.rel && f_rel == kNone) f_rel = e;
        }
    }
    f_mism = wave_min_u64(f_mism);
    f_abs = wave_min_u64(f_abs);
    f_rel = wave_min_u64(f_rel);
    if (lane == 0) {
        unsigned long long* o = (unsigned long long*)&p.out[index];
        if (f_mism != kNone) atomicMin(&o[0], (unsigned long long)f_mism);
        if (f_abs != kNone) atomicMin(&o[1], (unsigned long long)f_abs);
        if (f_rel != kNone) atomicMin(&o[2], (unsigned long long)f_rel);
    }
}

__global__ void fill_kernel(uint32_t* dst, uint64_t n, uint32_t value) {
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * blockDim.x)
        dst[i] = value;
}

}  // namespace

hipError_t launch_locate(int dtype, const LocateParams& p, const LocTable& tab, hipStream_t stream) {
    const unsigned grid = (unsigned)p.n * (unsigned)p.stripes;
    switch (dtype) {
        case DT_F32: hipLaunchKernelGGL(locate_kernel<DT_F32>, dim3(grid), dim3(kThreads), 0, stream, p, tab); break;
        case DT_F16: hipLaunchKernelGGL(locate_kernel<DT_F16>, dim3(grid), dim3(kThreads), 0, stream, p, tab); break;
        default: hipLaunchKernelGGL(locate_kernel<DT_BF16>, dim3(grid), dim3(kThreads), 0, stream, p, tab); break;
    }
    return hipGetLastError();
}

int locate_blocks_per_cu(int dtype) {
    // The occupancy of a kernel does not change during the process.
    static int cache[3] = {};  // value + 1, 0 = not queried yet
    const int di = dtype == DT_F32 ? 0 : dtype == DT_F16 ? 1 : 2;
    int v = __atomic_load_n(&cache[di], __ATOMIC_RELAXED) - 1;
    if (v < 0) {
        int n = 0;
        hipError_t e;
        switch (dtype) {
            case DT_F32: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, locate_kernel<DT_F32>, kThreads, 0); break;
            case DT_F16: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, locate_kernel<DT_F16>, kThreads, 0); break;
            default: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, locate_kernel<DT_BF16>, kThreads, 0); break;
        }
        v = e == hipSuccess ? n : 0;
        __atomic_store_n(&cache[di], v + 1, __ATOMIC_RELAXED);
    }
    return v;
}

hipError_t launch_fill_u32(void* dst, uint64_t n_words, uint32_t value, hipStream_t stream) {
    if (n_words == 0) return hipSuccess;
    const uint64_t want = (n_words + 255) / 256;
    const unsigned grid = (unsigned)(want < 1024 ? want : 1024);
    hipLaunchKernelGGL(fill_kernel, dim3(grid), dim3(256), 0, stream, (uint32_t*)dst, n_words, value);
    return hipGetLastError();
}

}  // namespace kb
