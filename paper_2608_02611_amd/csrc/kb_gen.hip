// kb_gen.hip -- seeded input generator for gfx950.
//
// Element g of stream (seed, stream_id, sub) is word g mod 4 of Philox4x32-10
// block g / 4 (key = seed, counter = (lo32(b), hi32(b), sub, stream_id)),
// mapped to a uniform value by u = (x >> 8) 2^-24 and fmaf(u, p1 - p0, p0), or
// to a normal value by the Box-Muller transform evaluated in binary64 over the
// word pair of g's half-block.  One thread computes one Philox block and
// stores its (up to) four elements; interior blocks of an offset that is a
// multiple of 4 store with one 16-byte (fp32/u32) or 8-byte (fp16/bf16)
// write.  The work is ALU-bound (ten 32x32->64 multiply rounds per block,
// plus binary64 log/sqrt/sincos per normal pair).
#include "kb_device.hpp"
#include "kb_internal.hpp"

namespace kb {
namespace {

constexpr double kTwoPi = 6.283185307179586476925286766559;  // 2 pi rounded to binary64

__device__ __forceinline__ float u01(uint32_t x) { return (float)(x >> 8) * 0x1p-24f; }

// Box-Muller on one word pair in binary64: the cosine and sine branches
// rho cos(theta), rho sin(theta) with rho = sqrt(-2 ln u1), theta = 2 pi u2.
__device__ __forceinline__ void box_muller64(uint32_t xa, uint32_t xb, double& zc, double& zs) {
    const double u1 = ((double)xa + 1.0) * 0x1p-32;  // (0, 1]
    const double u2 = (double)xb * 0x1p-32;          // [0, 1)
    const double rho = sqrt(-2.0 * log(u1));
    const double theta = kTwoPi * u2;
    double s, c;
    sincos(theta, &s, &c);
    zc = rho * c;
    zs = rho * s;
}

// The same, each branch rounded once to binary32.
__device__ __forceinline__ void box_muller(uint32_t xa, uint32_t xb, float& zc, float& zs) {
    double c, s;
    box_muller64(xa, xb, c, s);
    zc = (float)c;
    zs = (float)s;
}

// binary32 -> binary16 storage as its own rounding.  The value is made
// opaque first: otherwise the compiler may fuse the multiply-add that
// produced it with the conversion into one mixed-precision instruction that
// rounds once, straight to binary16, where the definition rounds to binary32
// and then to binary16 (the two differ when the binary32 result lands on a
// binary16 tie).
__device__ __forceinline__ uint16_t to_f16_bits(float v) {
    asm volatile("" : "+v"(v));
    return f32_to_f16_bits(v);
}

template <int DT>
__device__ __forceinline__ void store_one(void* dst, uint64_t j, float v, uint32_t word) {
    if constexpr (DT == DT_U32) ((uint32_t*)dst)[j] = word;
    else if constexpr (DT == DT_F32) ((float*)dst)[j] = v;
    else if constexpr (DT == DT_F16) ((uint16_t*)dst)[j] = to_f16_bits(v);
    else ((uint16_t*)dst)[j] = f32_to_bf16_bits(v);
}

template <int DT>
__device__ __forceinline__ void store_four(void* dst, uint64_t j, const float v[4], u32x4 w) {
    if constexpr (DT == DT_U32) {
        *(uint4*)((uint32_t*)dst + j) = make_uint4(w.x, w.y, w.z, w.w);
    } else if constexpr (DT == DT_F32) {
        *(float4*)((float*)dst + j) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
        uint32_t h[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            h[i] = DT == DT_F16 ? to_f16_bits(v[i]) : f32_to_bf16_bits(v[i]);
        *(uint2*)((uint16_t*)dst + j) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    }
}

template <int DIST, int DT>
__global__ __launch_bounds__(256) void gen_kernel(void* __restrict__ dst, uint64_t n, float p0,
                                                  float p1, uint32_t k0, uint32_t k1,
                                                  uint32_t stream_id, uint32_t sub,
                                                  uint64_t offset, uint64_t b_first,
                                                  uint64_t n_blocks) {
    const float width = p1 - p0;  // binary32, one rounding
    const uint64_t end = offset + n;
    const uint64_t step = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_blocks; t += step) {
        const uint64_t b = b_first + t;
        const u32x4 w = philox4x32_10({(uint32_t)b, (uint32_t)(b >> 32), sub, stream_id}, k0, k1);
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (DIST == KB_DIST_UNIFORM) {
            v[0] = fmaf(u01(w.x), width, p0);
            v[1] = fmaf(u01(w.y), width, p0);
            v[2] = fmaf(u01(w.z), width, p0);
            v[3] = fmaf(u01(w.w), width, p0);
        } else if constexpr (DIST == KB_DIST_NORMAL) {
            float z[4];
            box_muller(w.x, w.y, z[0], z[1]);
            box_muller(w.z, w.w, z[2], z[3]);
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = fmaf(z[i], p1, p0);
        }
        const uint64_t g0 = 4 * b;
        if (g0 >= offset && g0 + 4 <= end && ((g0 - offset) & 3) == 0) {
            store_four<DT>(dst, g0 - offset, v, w);
        } else {
            const uint32_t words[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint64_t g = g0 + i;
                if (g >= offset && g < end) store_one<DT>(dst, g - offset, v[i], words[i]);
            }
        }
    }
}

template <int DIST, int DT>
hipError_t launch_typed(void* dst, uint64_t n, float p0, float p1, uint64_t seed,
                        uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream) {
    const uint64_t b_first = offset / 4;
    const uint64_t b_last = (offset + n - 1) / 4;
    const uint64_t n_blocks = b_last - b_first + 1;
    const uint64_t want = (n_blocks + 255) / 256;
    const unsigned grid = (unsigned)(want < 16384 ? want : 16384);
    hipLaunchKernelGGL((gen_kernel<DIST, DT>), dim3(grid), dim3(256), 0, stream, dst, n, p0, p1,
                       (uint32_t)seed, (uint32_t)(seed >> 32), stream_id, sub, offset, b_first,
                       n_blocks);
    return hipGetLastError();
}

// Student-t with 3 degrees of freedom of one block's words: the ratio of the
// first binary64 normal to the root of the other three's mean square (a
// chi-square over its degrees of freedom), rounded once to binary32.
__device__ __forceinline__ float student_t3(u32x4 w) {
    double z0, z1, z2, z3;
    box_muller64(w.x, w.y, z0, z1);
    box_muller64(w.z, w.w, z2, z3);
    const double chi2 = (z1 * z1 + z2 * z2) + z3 * z3;
    return (float)(z0 / sqrt(chi2 / 3.0));
}

// An arithmetic result rounded to the storage type (nearest even); a NaN
// result is stored as the type's positive quiet NaN, whatever NaN the
// operation produced (its sign and payload are the platform's choice).
template <int DT>
__device__ __forceinline__ void store_value(void* dst, uint64_t j, float v) {
    const bool nan = __builtin_isnan(v);
    if constexpr (DT == DT_F32) ((uint32_t*)dst)[j] = nan ? 0x7FC00000u : __float_as_uint(v);
    else if constexpr (DT == DT_F16) ((uint16_t*)dst)[j] = nan ? (uint16_t)0x7E00u : to_f16_bits(v);
    else ((uint16_t*)dst)[j] = nan ? (uint16_t)0x7FC0u : f32_to_bf16_bits(v);
}

// The exact binary32 widening of src[j] (kept a separate instruction, so the
// arithmetic after it is plain binary32 arithmetic).
template <int DT>
__device__ __forceinline__ float load_value(const void* src, uint64_t j) {
    float x;
    if constexpr (DT == DT_F32) x = ((const float*)src)[j];
    else if constexpr (DT == DT_F16) x = f16_bits_to_f32(((const uint16_t*)src)[j]);
    else x = bf16_bits_to_f32(((const uint16_t*)src)[j]);
    asm volatile("" : "+v"(x));
    return x;
}

// One thread per element: element g = offset + j is the Student-t of block g.
template <int DT>
__global__ __launch_bounds__(256) void t3_kernel(void* __restrict__ dst, uint64_t n, float p0, float p1,
                                                 uint32_t k0, uint32_t k1, uint32_t stream_id, uint32_t sub,
                                                 uint64_t offset) {
    const uint64_t step = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += step) {
        const uint64_t b = offset + j;
        const u32x4 w = philox4x32_10({(uint32_t)b, (uint32_t)(b >> 32), sub, stream_id}, k0, k1);
        store_value<DT>(dst, j, fmaf(student_t3(w), p1, p0));
    }
}

unsigned elementwise_grid(uint64_t n) {
    const uint64_t want = (n + 255) / 256;
    return (unsigned)(want < 16384 ? want : 16384);
}

template <int DT>
hipError_t launch_t3(void* dst, uint64_t n, float p0, float p1, uint64_t seed, uint32_t stream_id,
                     uint32_t sub, uint64_t offset, hipStream_t stream) {
    hipLaunchKernelGGL((t3_kernel<DT>), dim3(elementwise_grid(n)), dim3(256), 0, stream, dst, n, p0, p1,
                       (uint32_t)seed, (uint32_t)(seed >> 32), stream_id, sub, offset);
    return hipGetLastError();
}

// ------------------------------------------------------------ softmax rows --
// One work-group per row (grid-striding over rows): the logits (the NORMAL
// stream, mean 0, standard deviation sigma) go to dst first, then the row's
// maximum, the binary64 sum of exp(x - max) and the quotients.  The sum is a
// fixed tree (each thread's elements in order, then 64-lane DPP sums, then
// the four waves in order), so it is the same bits on every call.
__device__ __forceinline__ float wave_max_float(float v) {
    v = fmaxf(v, __uint_as_float(dpp_u32<DPP_QUAD_XOR1>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp_u32<DPP_QUAD_XOR2>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp_u32<DPP_ROW_HALF_MIRROR>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp_u32<DPP_ROW_MIRROR>(__float_as_uint(v))));
    const float a = fmaxf(__uint_as_float(readlane_u32(__float_as_uint(v), 0)),
                          __uint_as_float(readlane_u32(__float_as_uint(v), 16)));
    const float b = fmaxf(__uint_as_float(readlane_u32(__float_as_uint(v), 32)),
                          __uint_as_float(readlane_u32(__float_as_uint(v), 48)));
    return fmaxf(a, b);
}

__global__ __launch_bounds__(256) void softmax_rows_kernel(float* __restrict__ dst, uint64_t rows, uint64_t cols,
                                                           float sigma, uint32_t k0, uint32_t k1,
                                                           uint32_t stream_id, uint32_t sub) {
    __shared__ float s_max[4];
    __shared__ double s_sum[4];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (uint64_t row = blockIdx.x; row < rows; row += gridDim.x) {
        float* x = dst + row * cols;
        float m = -__builtin_inff();
        for (uint64_t j = threadIdx.x; j < cols; j += 256) {
            const uint64_t g = row * cols + j;
            const uint64_t b = g >> 2;
            const u32x4 w = philox4x32_10({(uint32_t)b, (uint32_t)(b >> 32), sub, stream_id}, k0, k1);
            const uint32_t k = (uint32_t)(g & 3u);
            float zc, zs;
            if (k < 2) box_muller(w.x, w.y, zc, zs);
            else box_muller(w.z, w.w, zc, zs);
            const float v = fmaf(k & 1u ? zs : zc, sigma, 0.0f);
            x[j] = v;
            m = fmaxf(m, v);
        }
        m = wave_max_float(m);
        if (lane == 0) s_max[wave] = m;
        __syncthreads();
        m = fmaxf(fmaxf(s_max[0], s_max[1]), fmaxf(s_max[2], s_max[3]));
        double s = 0.0;
        for (uint64_t j = threadIdx.x; j < cols; j += 256) s += exp((double)x[j] - (double)m);
        s = wave_sum_f64(s);
        if (lane == 0) s_sum[wave] = s;
        __syncthreads();
        s = ((s_sum[0] + s_sum[1]) + s_sum[2]) + s_sum[3];
        for (uint64_t j = threadIdx.x; j < cols; j += 256) x[j] = (float)(exp((double)x[j] - (double)m) / s);
        __syncthreads();  // s_max / s_sum are reused by the next row
    }
}

// -------------------------------------------------------------- index draws --
// One wave: each round its 64 lanes draw blocks j0 .. j0 + 63 at once, then
// the draws are taken in order, each checked by all lanes against the
// indices accepted so far (in LDS) and appended if new.
__global__ __launch_bounds__(64) void indices_kernel(uint64_t* __restrict__ dst, uint32_t m, uint64_t n,
                                                     uint32_t k0, uint32_t k1, uint32_t stream_id, uint32_t sub) {
    __shared__ uint64_t s_idx[KB_MAX_INDICES];
    const uint32_t lane = threadIdx.x;
    uint32_t have = 0;
    // (at most 2^20 draws: with 2 m <= n each draw is new with probability
    // >= 1/2, so this bound only guarantees the loop ends)
    for (uint64_t j0 = 0; have < m && j0 < (1u << 20); j0 += 64) {
        const uint64_t b = j0 + lane;
        const u32x4 w = philox4x32_10({(uint32_t)b, (uint32_t)(b >> 32), sub, stream_id}, k0, k1);
        const uint64_t mine = (((uint64_t)w.y << 32) | w.x) % n;
        for (int l = 0; l < 64 && have < m; ++l) {
            const uint64_t x = readlane_u64(mine, l);
            bool seen = false;
            for (uint32_t i = lane; i < have; i += 64) seen |= s_idx[i] == x;
            if (__builtin_amdgcn_ballot_w64(seen) == 0) {
                if (lane == 0) s_idx[have] = x;
                ++have;
                __syncthreads();  // the new entry is visible to every lane's next scan
            }
        }
    }
    for (uint32_t i = lane; i < m; i += 64) dst[i] = i < have ? s_idx[i] : ~0ull;
}

// --------------------------------------------------------- planted changes --
// One thread per element (ops 1-5 read word g mod 4 of block g / 4; ops 6-7
// the whole block g, binary32 only).  In place (dst == src) is allowed.
template <int DT, int OP>
__global__ __launch_bounds__(256) void perturb_kernel(void* dst, const void* src, uint64_t n, float a, float b,
                                                      float p, uint32_t k0, uint32_t k1, uint32_t stream_id,
                                                      uint32_t sub, uint64_t offset) {
    const uint64_t step = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += step) {
        const uint64_t g = offset + j;
        if constexpr (OP <= KB_PERTURB_FLIP_LSB_WHERE) {
            const uint64_t blk = g >> 2;
            const u32x4 w = philox4x32_10({(uint32_t)blk, (uint32_t)(blk >> 32), sub, stream_id}, k0, k1);
            const uint32_t k = (uint32_t)(g & 3u);
            const uint32_t word = k == 0 ? w.x : k == 1 ? w.y : k == 2 ? w.z : w.w;
            const float x = load_value<DT>(src, j);
            if constexpr (OP == KB_PERTURB_ADD_UNIFORM) {
                store_value<DT>(dst, j, x + fmaf(u01(word), b - a, a));
            } else if constexpr (OP == KB_PERTURB_REL_UNIFORM) {
                store_value<DT>(dst, j, fmaf(x, fmaf(u01(word), b - a, a), x));
            } else if constexpr (OP == KB_PERTURB_ADD_NORMAL) {
                float zc, zs;
                if (k < 2) box_muller(w.x, w.y, zc, zs);
                else box_muller(w.z, w.w, zc, zs);
                store_value<DT>(dst, j, x + fmaf(k & 1u ? zs : zc, a, 0.0f));
            } else {
                const bool hit = u01(word) < p;
                if constexpr (DT == DT_F32) {
                    const uint32_t bits = ((const uint32_t*)src)[j];
                    if constexpr (OP == KB_PERTURB_SCALE_WHERE) {
                        if (hit) store_value<DT>(dst, j, x * a);
                        else ((uint32_t*)dst)[j] = bits;
                    } else {
                        ((uint32_t*)dst)[j] = hit ? bits ^ 1u : bits;
                    }
                } else {
                    const uint16_t bits = ((const uint16_t*)src)[j];
                    if constexpr (OP == KB_PERTURB_SCALE_WHERE) {
                        if (hit) store_value<DT>(dst, j, x * a);
                        else ((uint16_t*)dst)[j] = bits;
                    } else {
                        ((uint16_t*)dst)[j] = hit ? (uint16_t)(bits ^ 1u) : bits;
                    }
                }
            }
        } else {
            const u32x4 w = philox4x32_10({(uint32_t)g, (uint32_t)(g >> 32), sub, stream_id}, k0, k1);
            const uint32_t bits = ((const uint32_t*)src)[j];
            const float v = u01(w.x);
            uint32_t out = bits;
            if constexpr (OP == KB_PERTURB_SPECIALS) {
                const uint32_t sign = w.y & 0x80000000u;
                if (v < a) out = sign | (w.z & 0x7FFFFFu) | 1u;  // a subnormal of that sign
                else if (v < b) out = sign;                     // a zero
                else if (v < p) out = sign | 0x7F800000u;       // an infinity
            } else {  // KB_PERTURB_ZERO_SUBNORMAL_REL
                const uint32_t mag = bits & 0x7FFFFFFFu;
                if (v < p) {
                    if (mag == 0u) out = bits ^ 0x80000000u;               // flip the zero's sign
                    else if (mag < 0x00800000u) out = bits & 0x80000000u;  // flush the subnormal
                    else if (mag < 0x7F800000u) {                          // a finite normal value
                        const float x = __uint_as_float(bits);
                        out = __float_as_uint(fmaf(x, fmaf(u01(w.y), b - a, a), x));
                    }
                }
            }
            ((uint32_t*)dst)[j] = out;
        }
    }
}

template <int DT, int OP>
hipError_t launch_perturb_op(void* dst, const void* src, uint64_t n, float a, float b, float p, uint64_t seed,
                             uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream) {
    hipLaunchKernelGGL((perturb_kernel<DT, OP>), dim3(elementwise_grid(n)), dim3(256), 0, stream, dst, src, n,
                       a, b, p, (uint32_t)seed, (uint32_t)(seed >> 32), stream_id, sub, offset);
    return hipGetLastError();
}

template <int DT>
hipError_t launch_perturb_dt(void* dst, const void* src, uint64_t n, int op, float a, float b, float p,
                             uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream) {
    switch (op) {
        case KB_PERTURB_ADD_UNIFORM:
            return launch_perturb_op<DT, KB_PERTURB_ADD_UNIFORM>(dst, src, n, a, b, p, seed, stream_id, sub, offset, stream);
        case KB_PERTURB_REL_UNIFORM:
            return launch_perturb_op<DT, KB_PERTURB_REL_UNIFORM>(dst, src, n, a, b, p, seed, stream_id, sub, offset, stream);
        case KB_PERTURB_ADD_NORMAL:
            return launch_perturb_op<DT, KB_PERTURB_ADD_NORMAL>(dst, src, n, a, b, p, seed, stream_id, sub, offset, stream);
        case KB_PERTURB_SCALE_WHERE:
            return launch_perturb_op<DT, KB_PERTURB_SCALE_WHERE>(dst, src, n, a, b, p, seed, stream_id, sub, offset, stream);
        default:
            return launch_perturb_op<DT, KB_PERTURB_FLIP_LSB_WHERE>(dst, src, n, a, b, p, seed, stream_id, sub, offset, stream);
    }
}

// ------------------------------------------------------------------ scatter --
template <int DT>
__global__ __launch_bounds__(256) void scatter_kernel(void* dst, const void* ref, uint64_t n,
                                                      const uint64_t* __restrict__ idx, uint32_t m, int mode) {
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < m; i += gridDim.x * blockDim.x) {
        const uint64_t k = idx[i];
        if (k >= n) continue;
        if constexpr (DT == DT_F32) {
            const uint32_t sign = ((const uint32_t*)ref)[k] & 0x80000000u;
            ((uint32_t*)dst)[k] = mode == KB_SCATTER_NAN ? 0x7FC00000u : (sign | 0x7F800000u);
        } else {
            const uint16_t sign = (uint16_t)(((const uint16_t*)ref)[k] & 0x8000u);
            const uint16_t nan = DT == DT_F16 ? 0x7E00u : 0x7FC0u, inf = DT == DT_F16 ? 0x7C00u : 0x7F80u;
            ((uint16_t*)dst)[k] = mode == KB_SCATTER_NAN ? nan : (uint16_t)(sign | inf);
        }
    }
}

}  // namespace

hipError_t launch_gen_t3(void* dst, int dtype, uint64_t n, float p0, float p1, uint64_t seed,
                         uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream) {
    switch (dtype) {
        case DT_F32: return launch_t3<DT_F32>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
        case DT_F16: return launch_t3<DT_F16>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
        default: return launch_t3<DT_BF16>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
    }
}

hipError_t launch_softmax_rows(float* dst, uint64_t rows, uint64_t cols, float sigma, uint64_t seed,
                               uint32_t stream_id, uint32_t sub, hipStream_t stream) {
    const unsigned grid = (unsigned)(rows < 65536 ? rows : 65536);
    hipLaunchKernelGGL(softmax_rows_kernel, dim3(grid), dim3(256), 0, stream, dst, rows, cols, sigma,
                       (uint32_t)seed, (uint32_t)(seed >> 32), stream_id, sub);
    return hipGetLastError();
}

hipError_t launch_indices(uint64_t* dst, uint32_t m, uint64_t n, uint64_t seed, uint32_t stream_id, uint32_t sub,
                          hipStream_t stream) {
    hipLaunchKernelGGL(indices_kernel, dim3(1), dim3(64), 0, stream, dst, m, n, (uint32_t)seed,
                       (uint32_t)(seed >> 32), stream_id, sub);
    return hipGetLastError();
}

hipError_t launch_perturb(void* dst, const void* src, int dtype, uint64_t n, int op, float a, float b, float p,
                          uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset, hipStream_t stream) {
    if (op == KB_PERTURB_SPECIALS)
        return launch_perturb_op<DT_F32, KB_PERTURB_SPECIALS>(dst, src, n, a, b, p, seed, stream_id, sub, offset, stream);
    if (op == KB_PERTURB_ZERO_SUBNORMAL_REL)
        return launch_perturb_op<DT_F32, KB_PERTURB_ZERO_SUBNORMAL_REL>(dst, src, n, a, b, p, seed, stream_id, sub,
                                                                       offset, stream);
    switch (dtype) {
        case DT_F32: return launch_perturb_dt<DT_F32>(dst, src, n, op, a, b, p, seed, stream_id, sub, offset, stream);
        case DT_F16: return launch_perturb_dt<DT_F16>(dst, src, n, op, a, b, p, seed, stream_id, sub, offset, stream);
        default: return launch_perturb_dt<DT_BF16>(dst, src, n, op, a, b, p, seed, stream_id, sub, offset, stream);
    }
}

hipError_t launch_scatter(void* dst, const void* ref, int dtype, uint64_t n, const uint64_t* idx, uint32_t m,
                          int mode, hipStream_t stream) {
    const unsigned grid = (unsigned)((m + 255) / 256);
    switch (dtype) {
        case DT_F32:
            hipLaunchKernelGGL(scatter_kernel<DT_F32>, dim3(grid), dim3(256), 0, stream, dst, ref, n, idx, m, mode);
            break;
        case DT_F16:
            hipLaunchKernelGGL(scatter_kernel<DT_F16>, dim3(grid), dim3(256), 0, stream, dst, ref, n, idx, m, mode);
            break;
        default:
            hipLaunchKernelGGL(scatter_kernel<DT_BF16>, dim3(grid), dim3(256), 0, stream, dst, ref, n, idx, m, mode);
    }
    return hipGetLastError();
}

hipError_t launch_gen(void* dst, int dtype, uint64_t n, int dist, float p0, float p1,
                      uint64_t seed, uint32_t stream_id, uint32_t sub, uint64_t offset,
                      hipStream_t stream) {
    if (dist == KB_DIST_U32)
        return launch_typed<KB_DIST_U32, DT_U32>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
    if (dist == KB_DIST_UNIFORM) {
        switch (dtype) {
            case DT_F32: return launch_typed<KB_DIST_UNIFORM, DT_F32>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
            case DT_F16: return launch_typed<KB_DIST_UNIFORM, DT_F16>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
            default: return launch_typed<KB_DIST_UNIFORM, DT_BF16>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
        }
    }
    switch (dtype) {
        case DT_F32: return launch_typed<KB_DIST_NORMAL, DT_F32>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
        case DT_F16: return launch_typed<KB_DIST_NORMAL, DT_F16>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
        default: return launch_typed<KB_DIST_NORMAL, DT_BF16>(dst, n, p0, p1, seed, stream_id, sub, offset, stream);
    }
}

}  // namespace kb
