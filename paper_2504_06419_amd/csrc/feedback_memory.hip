// feedback_memory.hip -- feedback-memory mixing of the draft's activations (gfx950).
//
// The draft is a Feedback Transformer (paper Sec. 3.3): its attention reads
// memory vectors, one per draft layer i, each a convex mix of the token's
// activations after every layer (layer 0 the embedding):
//     m^i = sum_l exp(w_il) x^l / sum_l exp(w_il).
// x is [L+1, B*d], m is [n_out, B*d].  Every workgroup first turns the n_out
// rows of weights into mixing weights (row maximum subtracted, fp32) in LDS;
// every thread then reads 4 consecutive elements of each layer once and
// produces all n_out outputs from them, so x is read once and m written once.
#include "spire_internal.h"

namespace spire {

constexpr int kFmThreads = 256;

template <int XDT, int MDT, bool VEC>
__global__ __launch_bounds__(kFmThreads) void feedback_memory_kernel(FeedbackArgs a) {
    __shared__ float s_w[kFmMaxOut * kFmMaxLayers];
    if ((int)threadIdx.x < a.n_out) {
        const int i = threadIdx.x;
        float top = -INFINITY;
        for (int l = 0; l < a.Lp1; ++l) top = fmaxf(top, a.w[i * a.Lp1 + l]);
        float sum = 0.f;
        for (int l = 0; l < a.Lp1; ++l) {
            const float e = expf(a.w[i * a.Lp1 + l] - top);
            s_w[i * a.Lp1 + l] = e;
            sum += e;
        }
        const float inv = 1.f / sum;
        for (int l = 0; l < a.Lp1; ++l) s_w[i * a.Lp1 + l] *= inv;
    }
    __syncthreads();
    const int64_t e0 = ((int64_t)blockIdx.x * kFmThreads + threadIdx.x) * 4;
    if (e0 >= a.Bd) return;
    float acc[kFmMaxOut][4];
#pragma unroll
    for (int i = 0; i < kFmMaxOut; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[i][c] = 0.f;
    for (int l = 0; l < a.Lp1; ++l) {
        float xv[4];
        const int64_t base = (int64_t)l * a.Bd + e0;
        if (VEC) {
            if (XDT == SPIRE_F32) {
                const float4 v = *reinterpret_cast<const float4 *>(static_cast<const float *>(a.x) + base);
                xv[0] = v.x; xv[1] = v.y; xv[2] = v.z; xv[3] = v.w;
            } else {
                const uint2 v = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(a.x) + base);
                xv[0] = __uint_as_float(v.x << 16);
                xv[1] = __uint_as_float(v.x & 0xFFFF0000u);
                xv[2] = __uint_as_float(v.y << 16);
                xv[3] = __uint_as_float(v.y & 0xFFFF0000u);
            }
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                xv[c] = 0.f;
                if (e0 + c < a.Bd)
                    xv[c] = XDT == SPIRE_F32 ? static_cast<const float *>(a.x)[base + c]
                                             : bf16_to_f32(static_cast<const uint16_t *>(a.x)[base + c]);
            }
        }
#pragma unroll
        for (int i = 0; i < kFmMaxOut; ++i) {
            if (i < a.n_out) {
                const float wl = s_w[i * a.Lp1 + l];
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[i][c] = fmaf(wl, xv[c], acc[i][c]);
            }
        }
    }
#pragma unroll
    for (int i = 0; i < kFmMaxOut; ++i) {
        if (i >= a.n_out) break;
        const int64_t o = (int64_t)i * a.Bd + e0;
        if (VEC) {
            if (MDT == SPIRE_F32) {
                *reinterpret_cast<float4 *>(static_cast<float *>(a.m) + o) =
                    make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
            } else {
                const uint32_t lo = f32_to_bf16_rne(acc[i][0]) | ((uint32_t)f32_to_bf16_rne(acc[i][1]) << 16);
                const uint32_t hi = f32_to_bf16_rne(acc[i][2]) | ((uint32_t)f32_to_bf16_rne(acc[i][3]) << 16);
                *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(a.m) + o) = make_uint2(lo, hi);
            }
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if (e0 + c >= a.Bd) break;
                if (MDT == SPIRE_F32) static_cast<float *>(a.m)[o + c] = acc[i][c];
                else static_cast<uint16_t *>(a.m)[o + c] = f32_to_bf16_rne(acc[i][c]);
            }
        }
    }
}

template <int XDT, int MDT>
static void launch_fm_dt(const FeedbackArgs &a, bool vec, hipStream_t st) {
    const dim3 grid((unsigned)((a.Bd + 4LL * kFmThreads - 1) / (4LL * kFmThreads))), block(kFmThreads);
    if (vec) hipLaunchKernelGGL((feedback_memory_kernel<XDT, MDT, true>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((feedback_memory_kernel<XDT, MDT, false>), grid, block, 0, st, a);
}

hipError_t launch_feedback_memory(const FeedbackArgs &a, hipStream_t st) {
    // vector loads and stores need B*d % 4 == 0 and 16-byte (f32) / 8-byte (bf16) bases
    const uintptr_t xa = a.x_dtype == SPIRE_F32 ? 15u : 7u, ma = a.m_dtype == SPIRE_F32 ? 15u : 7u;
    const bool vec = (a.Bd % 4) == 0 && ((uintptr_t)a.x & xa) == 0 && ((uintptr_t)a.m & ma) == 0;
    if (a.x_dtype == SPIRE_F32) {
        if (a.m_dtype == SPIRE_F32) launch_fm_dt<SPIRE_F32, SPIRE_F32>(a, vec, st);
        else launch_fm_dt<SPIRE_F32, SPIRE_BF16>(a, vec, st);
    } else {
        if (a.m_dtype == SPIRE_F32) launch_fm_dt<SPIRE_BF16, SPIRE_F32>(a, vec, st);
        else launch_fm_dt<SPIRE_BF16, SPIRE_BF16>(a, vec, st);
    }
    return hipGetLastError();
}

}  // namespace spire
