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

// Box-Muller on one word pair: cosine and sine branches, each rounded once
// to binary32 from binary64.
__device__ __forceinline__ void box_muller(uint32_t xa, uint32_t xb, float& zc, float& zs) {
    const double u1 = ((double)xa + 1.0) * 0x1p-32;  // (0, 1]
    const double u2 = (double)xb * 0x1p-32;          // [0, 1)
    const double rho = sqrt(-2.0 * log(u1));
    const double theta = kTwoPi * u2;
    double s, c;
    sincos(theta, &s, &c);
    zc = (float)(rho * c);
    zs = (float)(rho * s);
}

template <int DT>
__device__ __forceinline__ void store_one(void* dst, uint64_t j, float v, uint32_t word) {
    if constexpr (DT == DT_U32) ((uint32_t*)dst)[j] = word;
    else if constexpr (DT == DT_F32) ((float*)dst)[j] = v;
    else if constexpr (DT == DT_F16) ((uint16_t*)dst)[j] = f32_to_f16_bits(v);
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
            h[i] = DT == DT_F16 ? f32_to_f16_bits(v[i]) : f32_to_bf16_bits(v[i]);
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

}  // namespace

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
