// sampling.h -- integer-weight inverse-CDF sampling shared by the token and
// block verification kernels (gfx950).
//
// A probability w becomes the integer weight floor(clamp(w, 0, 1) * 2^40);
// sums of such weights are exact, so every reduction order gives the same
// totals, and a uniform u picks the token whose running weight first exceeds
// T = floor(U * Z / 2^24), U = floor(u * 2^24) clamped to [0, 2^24 - 1].
#pragma once
#include "spire_internal.h"

namespace spire {

constexpr int kTvThreads = 256;
constexpr int kTvWaves = kTvThreads / 64;
constexpr int kTvGroupsPerLane = kTokenPiece / (4 * 64);   // float4 groups per lane (8)
constexpr int kTvSlice = kTokenPiece / kTvThreads;         // entries per select thread (8)

typedef float tv_f32x4 __attribute__((ext_vector_type(4)));

// Integer weight of one entry (w already formed in fp32): negatives and NaN
// weigh 0, values are capped at 1, W = floor(w * 2^40).  Formed from two
// 32-bit conversions: x = 256 w is exact, h = floor(x) its integer part and
// x - h its fraction (both exact in fp32), (x - h) * 2^32 is exact and below
// 2^32, and each conversion truncates, i.e. floors a non-negative value.
__device__ __forceinline__ uint64_t fixed_weight(float w) {
    w = w > 0.f ? w : 0.f;
    w = w < 1.f ? w : 1.f;
    const float x = w * 256.f;
    const float h = floorf(x);
    const uint32_t lo = (uint32_t)((x - h) * 4294967296.f);
    return ((uint64_t)(uint32_t)h << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_sum(uint64_t v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d);
    return v;
}

__device__ __forceinline__ uint64_t wave_incl_scan(uint64_t v, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t o = __shfl_up(v, d);
        if (lane >= d) v += o;
    }
    return v;
}

// Inclusive scan over the 256 threads of the workgroup; *total gets the sum.
__device__ __forceinline__ uint64_t block_incl_scan(uint64_t v, uint64_t *lds4, int lane, int wave,
                                                    uint64_t *total) {
    v = wave_incl_scan(v, lane);
    if (lane == 63) lds4[wave] = v;
    __syncthreads();
    uint64_t add = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kTvWaves; ++w) {
        add += w < wave ? lds4[w] : 0;
        all += lds4[w];
    }
    __syncthreads();
    *total = all;
    return v + add;
}

__device__ __forceinline__ uint64_t block_sum(uint64_t v, uint64_t *lds4, int lane, int wave) {
    v = wave_sum(v);
    if (lane == 0) lds4[wave] = v;
    __syncthreads();
    uint64_t s = 0;
#pragma unroll
    for (int w = 0; w < kTvWaves; ++w) s += lds4[w];
    __syncthreads();
    return s;
}

// T = floor(U * Z / 2^24) without overflow: Z = Zh * 2^24 + Zl.
__device__ __forceinline__ uint64_t sample_threshold(float u, uint64_t Z) {
    uint64_t U;
    if (!(u > 0.f)) U = 0;
    else if (u >= 1.f) U = (1u << 24) - 1;
    else U = (uint64_t)(u * 0x1p24f);  // exact scaling; truncation = floor
    return U * (Z >> 24) + ((U * (Z & 0xFFFFFFu)) >> 24);
}

}  // namespace spire
