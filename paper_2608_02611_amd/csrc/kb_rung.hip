// kb_rung.hip -- the rung benchmarker's statistics over timing samples.
//
// A rung times every surviving candidate on the rung's shapes, a number of
// iterations each (Section 3.2: fidelity level and rung budget; Appendix
// A.2: 4, 16 and 60 iterations on three rungs).  From those samples the
// scheduler needs, per (candidate, shape) row, the mean time and the speedup
// over the baseline (Appendix A.5), the quantiles behind the tail ratios of
// Table A.3, and per candidate the latency and the runtime score of Eq. 2.
//
// rows_wave_kernel   rows of at most 64 samples (every rung of the paper):
//                    one wave per row, one sample per lane, a bitonic sort
//                    across the lanes;
// rows_block_kernel  longer rows (up to kRungMaxIter): one work-group per
//                    row, bitonic sort in LDS;
// scores_kernel      one thread per candidate: latency, score, speedups;
// promote_kernel     the promotion decision over the scores.
//
// Every sum runs left to right in binary64, as the definitions read (the
// rows are short, so a sequential sum costs little), and every formula is
// evaluated with explicit roundings in the order written, so the results are
// the same bits as the definition's.
#include "kb_device.hpp"
#include "kb_internal.hpp"
#include "kb_rung.hpp"

namespace kb {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bool sample_ok(double t) { return __builtin_isfinite(t) && t > 0.0; }

// The p-quantile of x sorted ascending (n >= 1): linear interpolation
// between the order statistics around position h = (n - 1) p.
template <class Get>
__device__ __forceinline__ double quantile(Get x, int n, double p) {
    const double h = __dmul_rn((double)(n - 1), p);
    const int k = (int)floor(h);
    if (k >= n - 1) return x(n - 1);
    const double t = __dsub_rn(h, (double)k);
    const double a = x(k), b = x(k + 1);
    return __dadd_rn(a, __dmul_rn(t, __dsub_rn(b, a)));
}

__device__ __forceinline__ void write_row(kb_sample_stats* o, int n, bool valid, double sum,
                                          double q50, double q90, double q95, double q99) {
    kb_sample_stats r;
    const double nan = __builtin_nan("");
    r.n_samples = n;
    r.valid = valid ? 1 : 0;
    r.speedup_vs_base = nan;  // set by scores_kernel
    if (valid) {
        r.mean_us = sum / (double)n;
        r.p50_us = q50;
        r.p90_us = q90;
        r.p95_us = q95;
        r.p99_us = q99;
        r.p90_over_p50 = q90 / q50;
        r.p95_over_p50 = q95 / q50;
        r.p99_over_p50 = q99 / q50;
    } else {
        r.mean_us = r.p50_us = r.p90_us = r.p95_us = r.p99_us = nan;
        r.p90_over_p50 = r.p95_over_p50 = r.p99_over_p50 = nan;
    }
    *o = r;
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, l);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), l);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// One wave per row: lane l holds sample l (+inf past the end), a bitonic
// network over the lane index sorts ascending, and the quantiles read the
// sorted values from their lanes.
__global__ __launch_bounds__(kThreads) void rows_wave_kernel(const double* __restrict__ samples,
                                                              int n_rows, int n,
                                                              kb_sample_stats* __restrict__ rows) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (row >= n_rows) return;  // whole waves
    const double* t = samples + (size_t)row * (size_t)n;
    double v = lane < n ? t[lane] : __builtin_inf();
    const bool valid = __builtin_amdgcn_ballot_w64(lane < n && !sample_ok(v)) == 0;
    // the mean's sum, left to right over the samples
    double sum = 0.0;
    if (valid) {
        for (int i = 0; i < n; ++i) sum = __dadd_rn(sum, readlane_f64(v, i));
    }
    double q50 = 0.0, q90 = 0.0, q95 = 0.0, q99 = 0.0;
    if (valid) {
#pragma unroll
        for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
            for (int j = k >> 1; j > 0; j >>= 1) {
                const double o = __shfl_xor(v, j, 64);
                const bool lower = (lane & j) == 0;
                const bool ascending = (lane & k) == 0;
                v = (lower == ascending) ? fmin(v, o) : fmax(v, o);
            }
        }
        auto x = [&](int i) { return readlane_f64(v, i); };
        q50 = quantile(x, n, 0.5);
        q90 = quantile(x, n, 0.9);
        q95 = quantile(x, n, 0.95);
        q99 = quantile(x, n, 0.99);
    }
    if (lane == 0) write_row(&rows[row], n, valid, sum, q50, q90, q95, q99);
}

// One work-group per row of up to kRungMaxIter samples, sorted in LDS.
__global__ __launch_bounds__(kThreads) void rows_block_kernel(const double* __restrict__ samples,
                                                               int n, int P,
                                                               kb_sample_stats* __restrict__ rows) {
    __shared__ double s[kRungMaxIter];
    __shared__ double s_sum;
    const int row = blockIdx.x;
    const double* t = samples + (size_t)row * (size_t)n;
    int bad = 0;
    for (int i = threadIdx.x; i < P; i += kThreads) {
        const double v = i < n ? t[i] : __builtin_inf();
        bad |= i < n && !sample_ok(v);
        s[i] = v;
    }
    const bool valid = __syncthreads_or(bad) == 0;
    if (!valid) {
        if (threadIdx.x == 0) write_row(&rows[row], n, false, 0.0, 0.0, 0.0, 0.0, 0.0);
        return;
    }
    if (threadIdx.x == 0) {
        // left to right; the loads are batched so that only the adds wait
        double sum = 0.0;
        int i = 0;
        for (; i + 8 <= n; i += 8) {
            double v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = s[i + u];
#pragma unroll
            for (int u = 0; u < 8; ++u) sum = __dadd_rn(sum, v[u]);
        }
        for (; i < n; ++i) sum = __dadd_rn(sum, s[i]);
        s_sum = sum;
    }
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < P / 2; i += kThreads) {
                const int lo = ((i & ~(j - 1)) << 1) | (i & (j - 1));  // j is a power of 2
                const int hi = lo + j;
                const bool ascending = (lo & k) == 0;
                const double a = s[lo], b = s[hi];
                if ((a > b) == ascending) {
                    s[lo] = b;
                    s[hi] = a;
                }
            }
            __syncthreads();
        }
    }
    if (threadIdx.x == 0) {
        auto x = [&](int i) { return s[i]; };
        write_row(&rows[row], n, true, s_sum, quantile(x, n, 0.5), quantile(x, n, 0.9),
                  quantile(x, n, 0.95), quantile(x, n, 0.99));
    }
}

// The latency of candidate c: the mean over shapes of its row means (NaN if
// a row is invalid; `valid` reports it).
__device__ __forceinline__ double latency_of(const kb_sample_stats* rows, int c, int n_shapes,
                                             bool* valid) {
    double sum = 0.0;
    bool ok = true;
    for (int s = 0; s < n_shapes; ++s) {
        const kb_sample_stats& r = rows[(size_t)c * n_shapes + s];
        ok = ok && r.valid != 0;
        sum = __dadd_rn(sum, r.mean_us);
    }
    *valid = ok;
    return ok ? sum / (double)n_shapes : __builtin_nan("");
}

__global__ __launch_bounds__(kThreads) void scores_kernel(RungParams p, kb_sample_stats* rows,
                                                           kb_rung_score* scores) {
    const int c = blockIdx.x * kThreads + threadIdx.x;
    if (c >= p.n_cands) return;
    const double nan = __builtin_nan("");
    bool ok;
    const double lat = latency_of(rows, c, p.n_shapes, &ok);
    double base_lat = nan;
    if (p.base >= 0) {
        bool base_ok;
        base_lat = latency_of(rows, p.base, p.n_shapes, &base_ok);
    }
    kb_rung_score sc;
    sc.valid = ok ? 1 : 0;
    sc.reserved = 0;
    sc.latency_us = lat;
    if (ok) {
        const double lead = 1e6 / (lat > 1.0 ? lat : 1.0);
        // Eq. 2: the latency term plus the one rung term gamma(r) = alpha r + beta b_r
        sc.score = __dadd_rn(lead, __dadd_rn(__dmul_rn(p.alpha, (double)p.rung), __dmul_rn(p.beta, p.budget)));
        sc.speedup_vs_base = base_lat / lat;
    } else {
        sc.score = -__builtin_inf();
        sc.speedup_vs_base = nan;
    }
    scores[c] = sc;
    for (int s = 0; s < p.n_shapes; ++s) {
        kb_sample_stats& r = rows[(size_t)c * p.n_shapes + s];
        const double b = p.base >= 0 ? rows[(size_t)p.base * p.n_shapes + s].mean_us : nan;
        r.speedup_vs_base = r.valid ? b / r.mean_us : nan;
    }
}

// The promotion decision D (Section 3.4): rank by score, ties to the lower
// index, and promote the first ceil(n_eligible num / den) valid non-baseline
// candidates plus a valid baseline.  Ranking is by counting: candidate i's
// rank is the number of candidates that come before it.  One wave per
// candidate: its lanes split the scan over all keys (read from L2), and a
// butterfly sums their counts; no sort or atomic is needed, the ranks are a
// permutation, and `order` is their inverse.
__device__ __forceinline__ double rank_key(const kb_rung_score& s) {
    return s.valid != 0 && s.score == s.score ? s.score : -__builtin_inf();
}

__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

__global__ __launch_bounds__(kThreads) void promote_kernel(const kb_rung_score* __restrict__ scores,
                                                            int n, int base, int num, int den,
                                                            int32_t* __restrict__ rank,
                                                            int32_t* __restrict__ order,
                                                            int32_t* __restrict__ promoted) {
    const int lane = threadIdx.x & 63;
    const int i = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (i >= n) return;  // whole waves
    const double ki = rank_key(scores[i]);
    const bool valid_i = scores[i].valid != 0;
    int before = 0, before_elig = 0, n_elig = 0;
    for (int j = lane; j < n; j += 64) {
        const kb_rung_score sj = scores[j];
        const double kj = rank_key(sj);
        const bool elig = sj.valid != 0 && j != base;
        const bool b = kj > ki || (kj == ki && j < i);
        before += b;
        before_elig += b && elig;
        n_elig += elig;
    }
    before = wave_sum_i32(before);
    before_elig = wave_sum_i32(before_elig);
    n_elig = wave_sum_i32(n_elig);
    if (lane != 0) return;
    const long long keep = ((long long)n_elig * num + den - 1) / den;
    rank[i] = before;
    order[before] = i;
    int p;
    if (i == base) p = valid_i ? 1 : 0;
    else p = valid_i && before_elig < keep ? 1 : 0;
    promoted[i] = p;
}

}  // namespace

hipError_t launch_rung_promote(const kb_rung_score* scores, int n, int base, int num, int den,
                               int32_t* rank, int32_t* order, int32_t* promoted, hipStream_t stream) {
    const int per_block = kThreads / 64;
    hipLaunchKernelGGL(promote_kernel, dim3((n + per_block - 1) / per_block), dim3(kThreads), 0, stream,
                       scores, n, base, num, den, rank, order, promoted);
    return hipGetLastError();
}

hipError_t launch_rung_stats(const RungParams& p, const double* samples, kb_sample_stats* rows,
                             kb_rung_score* scores, hipStream_t stream) {
    const int n_rows = p.n_cands * p.n_shapes;
    if (p.n_iter <= 64) {
        const int per_block = kThreads / 64;
        hipLaunchKernelGGL(rows_wave_kernel, dim3((n_rows + per_block - 1) / per_block), dim3(kThreads),
                           0, stream, samples, n_rows, p.n_iter, rows);
    } else {
        int P = 1;
        while (P < p.n_iter) P <<= 1;
        hipLaunchKernelGGL(rows_block_kernel, dim3(n_rows), dim3(kThreads), 0, stream, samples,
                           p.n_iter, P, rows);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scores_kernel, dim3((p.n_cands + kThreads - 1) / kThreads), dim3(kThreads), 0,
                       stream, p, rows, scores);
    return hipGetLastError();
}

}  // namespace kb
