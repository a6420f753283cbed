// kb_screen.hip -- batched screening kernel for gfx950.
//
// One pass over the reference and K candidate outputs computing, per
// candidate, the statistics of the Verifier's output check (correctness
// indicator K(p), Sections 3.1 and 3.4): mismatches under
// |c - r| <= atol + rtol*|r|, NaN/+Inf/-Inf counts, bitwise identity, max
// abs error, max rel error and the two squared-error sums of the relative L2
// error.  The work is a streaming reduction bound by HBM bandwidth: no
// contraction, so no MFMA.
//
// Work split.  Candidates that passed the policy gate are cut into groups of
// KG; a work-group owns one candidate group and one stripe of the element
// range, walks its stripe in 16-byte vectors (grid-stride over the group's
// work-groups, so that consecutive work-groups read consecutive memory), loads
// each reference vector once and compares it with the KG candidates' vectors
// while it is in registers.  Work-group ids are mapped so that all candidate
// groups of one stripe run on the same XCD (ids are dealt to the 8 XCDs round
// robin), and a reference stripe fetched for one group is then found in that
// XCD's L2 by the others.
//
// Reduction.  Per lane accumulators -> 64-lane DPP reductions -> LDS combine
// of the work-group's waves in wave order -> per-(work-group, candidate)
// partials in the workspace.  The last work-group of a candidate group to
// finish (an atomic ticket after a release fence) combines the partials of
// its group in a fixed order and writes the kb_stats records; the binary64
// sums are therefore the same bits on every call.
#include "kb_device.hpp"
#include "kb_internal.hpp"

namespace kb {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

template <int DT>
struct Elem {
    static constexpr int kVec = DT == DT_F32 ? 4 : 8;  // elements per 16-byte vector
};

// Per-lane running statistics of one candidate.
struct LaneAcc {
    uint32_t mism, nan, pinf, ninf, bitdiff;
    float max_abs, max_rel;
    double ssd;
};

__device__ __forceinline__ void acc_init(LaneAcc& a) {
    a.mism = a.nan = a.pinf = a.ninf = a.bitdiff = 0u;
    a.max_abs = a.max_rel = 0.f;
    a.ssd = 0.0;
}

// Reference-side values of one element, computed once and used for all KG
// candidates: r, |r|, the tolerance atol + rtol*|r| (two binary32 roundings;
// -1 for a non-finite r, which only c == r can match) and finiteness.
struct RefElem {
    float r, a, tol;
    bool fin;
};

__device__ __forceinline__ RefElem ref_elem(float r, float atol, float rtol) {
    RefElem e;
    e.r = r;
    e.a = fabsf(r);
    e.fin = __builtin_isfinite(r);
    e.tol = e.fin ? __fadd_rn(atol, __fmul_rn(rtol, e.a)) : -1.0f;
    return e;
}

// One (element, candidate) pair, by definition.
__device__ __forceinline__ void acc_elem(LaneAcc& A, float c, const RefElem& R, bool equal_nan) {
    const bool cnan = __builtin_isnan(c);
    A.nan += cnan ? 1u : 0u;
    A.pinf += (c == __builtin_inff()) ? 1u : 0u;
    A.ninf += (c == -__builtin_inff()) ? 1u : 0u;
    const float d = fabsf(__fsub_rn(c, R.r));
    const bool match = (c == R.r) || (d <= R.tol) || (equal_nan && cnan && __builtin_isnan(R.r));
    A.mism += match ? 0u : 1u;
    if (d > A.max_abs) A.max_abs = d;
    const float q = d / R.a;  // IEEE binary32 division (x/0 = inf, 0/0 = NaN)
    if (q > A.max_rel) A.max_rel = q;
    if (R.fin && __builtin_isfinite(c)) A.ssd = __builtin_fma((double)d, (double)d, A.ssd);
}

template <int DT>
__device__ __forceinline__ float widen(uint32_t bits) {
    if constexpr (DT == DT_F32) return __uint_as_float(bits);
    else if constexpr (DT == DT_F16) return f16_bits_to_f32(bits);
    else return bf16_bits_to_f32(bits);
}

// Element i of a 16-byte vector (little-endian halves for 16-bit types).
template <int DT>
__device__ __forceinline__ uint32_t vec_elem_bits(const uint4& v, int i) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if constexpr (DT == DT_F32) return w[i];
    else return (w[i >> 1] >> ((i & 1) * 16)) & 0xFFFFu;
}

template <int DT>
__device__ __forceinline__ uint32_t scalar_bits(const void* base, uint64_t i) {
    if constexpr (DT == DT_F32) return ((const uint32_t*)base)[i];
    else return ((const uint16_t*)base)[i];
}

// Block-wide fixed-order combine helpers (LDS scratch provided by caller).
struct Lds {
    uint32_t u[kWaves][PF_COUNT];
    double ssd[kWaves];
    double ssr[kWaves];
};

template <int DT, int KG>
__global__ __launch_bounds__(kThreads) void screen_kernel(ScreenParams p) {
    constexpr int V = Elem<DT>::kVec;
    __shared__ Lds lds[KG];
    __shared__ uint32_t s_is_last;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    // XCD-aware ids: block ids are dealt to the 8 XCDs round robin; keep one
    // stripe's candidate groups on one XCD.
    const int xcd = blockIdx.x & 7;
    const int slot = blockIdx.x >> 3;
    const int g = slot % p.n_groups;
    const int stripe = (slot / p.n_groups) * 8 + xcd;
    const int j0 = g * KG;
    const int kg = min(KG, p.n_acc - j0);
    const bool equal_nan = (p.flags & KB_EQUAL_NAN) != 0;

    const uint4* cand[KG];
#pragma unroll
    for (int j = 0; j < KG; ++j) cand[j] = (const uint4*)(j < kg ? p.table[j0 + j].data : p.ref);
    const uint4* ref = (const uint4*)p.ref;

    LaneAcc acc[KG];
#pragma unroll
    for (int j = 0; j < KG; ++j) acc_init(acc[j]);
    double ssr = 0.0;

    const uint64_t stride = (uint64_t)p.blocks_per_group * kThreads;
    for (uint64_t v = (uint64_t)stripe * kThreads + threadIdx.x; v < p.n_vec; v += stride) {
        const uint4 rv = ref[v];
        RefElem R[V];
#pragma unroll
        for (int i = 0; i < V; ++i) {
            R[i] = ref_elem(widen<DT>(vec_elem_bits<DT>(rv, i)), p.atol, p.rtol);
            if (R[i].fin) ssr = __builtin_fma((double)R[i].r, (double)R[i].r, ssr);
        }
        uint4 cv[KG];
#pragma unroll
        for (int j = 0; j < KG; ++j)
            if (j < kg) cv[j] = cand[j][v];
#pragma unroll
        for (int j = 0; j < KG; ++j) {
            if (j < kg) {
                acc[j].bitdiff |= (cv[j].x ^ rv.x) | (cv[j].y ^ rv.y) | (cv[j].z ^ rv.z) |
                                  (cv[j].w ^ rv.w);
#pragma unroll
                for (int i = 0; i < V; ++i)
                    acc_elem(acc[j], widen<DT>(vec_elem_bits<DT>(cv[j], i)), R[i], equal_nan);
            }
        }
    }
    // Ragged tail (numel not a multiple of V): stripe 0 of each group.
    if (stripe == 0) {
        const uint64_t first = p.n_vec * V;
        const uint64_t i = first + threadIdx.x;
        if (i < p.numel) {
            const uint32_t rb = scalar_bits<DT>(p.ref, i);
            const RefElem R = ref_elem(widen<DT>(rb), p.atol, p.rtol);
            if (R.fin) ssr = __builtin_fma((double)R.r, (double)R.r, ssr);
#pragma unroll
            for (int j = 0; j < KG; ++j) {
                if (j < kg) {
                    const uint32_t cb = scalar_bits<DT>(p.table[j0 + j].data, i);
                    acc[j].bitdiff |= cb ^ rb;
                    acc_elem(acc[j], widen<DT>(cb), R, equal_nan);
                }
            }
        }
    }

    // Wave reductions, then the work-group's partials in wave order.
#pragma unroll
    for (int j = 0; j < KG; ++j) {
        if (j < kg) {
            const uint32_t m = wave_sum_u32(acc[j].mism);
            const uint32_t na = wave_sum_u32(acc[j].nan);
            const uint32_t pi = wave_sum_u32(acc[j].pinf);
            const uint32_t ni = wave_sum_u32(acc[j].ninf);
            const uint32_t ma = wave_max_u32(__float_as_uint(acc[j].max_abs));
            const uint32_t mr = wave_max_u32(__float_as_uint(acc[j].max_rel));
            const uint32_t bd = wave_or_u32(acc[j].bitdiff);
            const double sd = wave_sum_f64(acc[j].ssd);
            if (lane == 0) {
                lds[j].u[wave][PF_MISM] = m;
                lds[j].u[wave][PF_NAN] = na;
                lds[j].u[wave][PF_PINF] = pi;
                lds[j].u[wave][PF_NINF] = ni;
                lds[j].u[wave][PF_MAXABS] = ma;
                lds[j].u[wave][PF_MAXREL] = mr;
                lds[j].u[wave][PF_BITDIFF] = bd;
                lds[j].ssd[wave] = sd;
            }
        }
    }
    {
        const double sr = wave_sum_f64(ssr);
        if (lane == 0) lds[0].ssr[wave] = sr;
    }
    __syncthreads();

    const int C = p.blocks_per_group;
    if (threadIdx.x < kg) {
        const int j = threadIdx.x;
        const Lds& L = lds[j];
        uint32_t m = 0, na = 0, pi = 0, ni = 0, ma = 0, mr = 0, bd = 0;
        double sd = 0.0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            m += L.u[w][PF_MISM];
            na += L.u[w][PF_NAN];
            pi += L.u[w][PF_PINF];
            ni += L.u[w][PF_NINF];
            ma = max(ma, L.u[w][PF_MAXABS]);
            mr = max(mr, L.u[w][PF_MAXREL]);
            bd |= L.u[w][PF_BITDIFF];
            sd += L.ssd[w];
        }
        const size_t row = (size_t)(j0 + j) * C + stripe;
        const size_t plane = (size_t)p.n_acc * C;
        p.part_u32[PF_MISM * plane + row] = m;
        p.part_u32[PF_NAN * plane + row] = na;
        p.part_u32[PF_PINF * plane + row] = pi;
        p.part_u32[PF_NINF * plane + row] = ni;
        p.part_u32[PF_MAXABS * plane + row] = ma;
        p.part_u32[PF_MAXREL * plane + row] = mr;
        p.part_u32[PF_BITDIFF * plane + row] = bd;
        p.part_ssd[row] = sd;
    }
    if (threadIdx.x == 0) {
        double sr = 0.0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) sr += lds[0].ssr[w];
        p.part_ssr[(size_t)g * C + stripe] = sr;
    }

    // Last work-group of this candidate group finishes it.
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t t = atomicAdd(&p.tickets[g], 1u);
        s_is_last = (t == (uint32_t)C - 1u) ? 1u : 0u;
    }
    __syncthreads();
    if (!s_is_last) return;
    __threadfence();

    // Fixed-order combine over stripes: thread t takes stripes t, t+256, ...
    // in order, then the work-group combines threads in a fixed tree.
    __shared__ double s_red[kWaves];
    __shared__ uint64_t s_cnt[kWaves][4];
    __shared__ uint32_t s_mx[kWaves][3];

    double total_ssr;
    {
        double acc_r = 0.0;
        for (int s = threadIdx.x; s < C; s += kThreads) acc_r += p.part_ssr[(size_t)g * C + s];
        const double w = wave_sum_f64(acc_r);
        if (lane == 0) s_red[wave] = w;
        __syncthreads();
        total_ssr = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
        __syncthreads();
    }

    const size_t plane = (size_t)p.n_acc * C;
    for (int j = 0; j < kg; ++j) {
        const size_t base = (size_t)(j0 + j) * C;
        uint32_t ma = 0, mr = 0, bd = 0;
        uint64_t m64 = 0, na64 = 0, pi64 = 0, ni64 = 0;
        double sd = 0.0;
        for (int s = threadIdx.x; s < C; s += kThreads) {
            m64 += p.part_u32[PF_MISM * plane + base + s];
            na64 += p.part_u32[PF_NAN * plane + base + s];
            pi64 += p.part_u32[PF_PINF * plane + base + s];
            ni64 += p.part_u32[PF_NINF * plane + base + s];
            ma = max(ma, p.part_u32[PF_MAXABS * plane + base + s]);
            mr = max(mr, p.part_u32[PF_MAXREL * plane + base + s]);
            bd |= p.part_u32[PF_BITDIFF * plane + base + s];
            sd += p.part_ssd[base + s];
        }
        const uint64_t wm = wave_sum_u64(m64), wn = wave_sum_u64(na64);
        const uint64_t wp = wave_sum_u64(pi64), wq = wave_sum_u64(ni64);
        const uint32_t wma = wave_max_u32(ma), wmr = wave_max_u32(mr), wbd = wave_or_u32(bd);
        const double wsd = wave_sum_f64(sd);
        if (lane == 0) {
            s_cnt[wave][0] = wm;
            s_cnt[wave][1] = wn;
            s_cnt[wave][2] = wp;
            s_cnt[wave][3] = wq;
            s_mx[wave][0] = wma;
            s_mx[wave][1] = wmr;
            s_mx[wave][2] = wbd;
            s_red[wave] = wsd;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            kb_stats st;
            st.numel = p.numel;
            st.mismatches = (s_cnt[0][0] + s_cnt[1][0]) + (s_cnt[2][0] + s_cnt[3][0]);
            st.nan_count = (s_cnt[0][1] + s_cnt[1][1]) + (s_cnt[2][1] + s_cnt[3][1]);
            st.pos_inf_count = (s_cnt[0][2] + s_cnt[1][2]) + (s_cnt[2][2] + s_cnt[3][2]);
            st.neg_inf_count = (s_cnt[0][3] + s_cnt[1][3]) + (s_cnt[2][3] + s_cnt[3][3]);
            const double ssd_t = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
            st.sum_sq_diff = ssd_t;
            st.sum_sq_ref = total_ssr;
            st.rel_l2 = total_ssr > 0.0 ? sqrt(ssd_t / total_ssr)
                                        : (ssd_t == 0.0 ? 0.0 : __builtin_inf());
            st.max_abs_err = __uint_as_float(max(max(s_mx[0][0], s_mx[1][0]), max(s_mx[2][0], s_mx[3][0])));
            st.max_rel_err = __uint_as_float(max(max(s_mx[0][1], s_mx[1][1]), max(s_mx[2][1], s_mx[3][1])));
            st.bitwise_equal = ((s_mx[0][2] | s_mx[1][2]) | (s_mx[2][2] | s_mx[3][2])) == 0u ? 1 : 0;
            st.status = KB_STATUS_OK;
            p.stats[p.table[j0 + j].index] = st;
        }
        __syncthreads();
    }
    // Group 0's finisher also writes the rejected candidates' records.
    if (g == 0) {
        for (int k = p.n_acc + threadIdx.x; k < p.n_cands; k += kThreads) {
            kb_stats st = {};
            st.status = p.table[k].status;
            p.stats[p.table[k].index] = st;
        }
    }
    // Leave the ticket at zero for the next call on this workspace.
    if (threadIdx.x == 0) p.tickets[g] = 0u;
}

__global__ void records_only_kernel(const CandEntry* table, int n_cands, uint64_t numel,
                                    kb_stats* stats) {
    for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n_cands; k += gridDim.x * blockDim.x) {
        kb_stats st = {};
        st.status = table[k].status;
        if (st.status == KB_STATUS_OK) {
            st.numel = numel;  // numel == 0 here
            st.bitwise_equal = 1;
        }
        stats[table[k].index] = st;
    }
}

template <int DT, int KG>
hipError_t launch_kg(const ScreenPlan& plan, const ScreenParams& p, hipStream_t stream) {
    const unsigned grid = (unsigned)plan.n_groups * (unsigned)plan.blocks_per_group;
    hipLaunchKernelGGL((screen_kernel<DT, KG>), dim3(grid), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

template <int DT>
hipError_t launch_dt(const ScreenPlan& plan, const ScreenParams& p, hipStream_t stream) {
    switch (plan.kg) {
        case 1: return launch_kg<DT, 1>(plan, p, stream);
        case 2: return launch_kg<DT, 2>(plan, p, stream);
        case 4: return launch_kg<DT, 4>(plan, p, stream);
        case 8: return launch_kg<DT, 8>(plan, p, stream);
        default: return launch_kg<DT, 16>(plan, p, stream);
    }
}

}  // namespace

hipError_t launch_screen(const ScreenPlan& plan, const ScreenParams& p, hipStream_t stream) {
    switch (plan.dtype) {
        case DT_F32: return launch_dt<DT_F32>(plan, p, stream);
        case DT_F16: return launch_dt<DT_F16>(plan, p, stream);
        default: return launch_dt<DT_BF16>(plan, p, stream);
    }
}

hipError_t launch_records_only(const CandEntry* table, int n_cands, uint64_t numel,
                               kb_stats* stats, hipStream_t stream) {
    const int grid = (n_cands + 255) / 256;
    hipLaunchKernelGGL(records_only_kernel, dim3(grid), dim3(256), 0, stream, table, n_cands,
                       numel, stats);
    return hipGetLastError();
}

}  // namespace kb
