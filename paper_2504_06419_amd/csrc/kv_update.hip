// kv_update.hip -- KV cache writes around a speculation round (gfx950).
//
//   kv_append       the target's verify pass produced the K/V of the k+1 tokens
//                   of a round (paper Sec. 2); they are appended at positions
//                   n_b .. n_b + T - 1 of each sequence's (paged or contiguous)
//                   cache, rounded to the storage dtype;
//   draft_append    one draft step stores its token at its sink row or ring
//                   slot of the constant-size StreamingLLM cache (Sec. 3.1),
//                   optionally copying the row it overwrites (for a full ring:
//                   the evicted position) into a spill slot;
//   draft_rollback  restores the rows written by rejected draft steps from the
//                   spill slots, latest step first, so the cache holds exactly
//                   what the accepted steps alone would have left.
//
// One wave per (row of D elements); every write stays inside the storage the
// descriptors describe (positions without storage are skipped).
//
// Rounding: bf16 round-to-nearest-even (NaN kept quiet); OCP e4m3fn from the
// fp32 quotient x / scale[h] (IEEE division), nearest with ties to the even
// code, saturating at +-448 (infinities too), NaN -> 0x7F.
#include "spire_internal.h"

namespace spire {

// fp32 -> OCP e4m3fn code, round to nearest even, saturating.
__device__ __forceinline__ uint8_t f32_to_e4m3fn_sat(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t sign = (u >> 24) & 0x80u;
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7F;  // NaN
    const float a = __uint_as_float(u & 0x7fffffffu);
    if (a >= 448.f) return (uint8_t)(sign | 0x7Eu);
    if (a < 0x1p-6f) {
        // subnormal codes m * 2^-9 (m = 8 is the smallest normal, code 0x08)
        const uint32_t m = (uint32_t)__builtin_rintf(a * 512.f);  // exact scaling, ties to even
        return (uint8_t)(sign | m);
    }
    const uint32_t au = __float_as_uint(a);
    int e = (int)(au >> 23) - 127;        // -6 .. 8
    uint32_t m3 = (au >> 20) & 7u;        // top 3 fraction bits
    const uint32_t rem = au & 0xFFFFFu;   // the 20 bits rounded away
    if (rem > 0x80000u || (rem == 0x80000u && (m3 & 1u))) ++m3;
    if (m3 == 8u) {
        m3 = 0;
        ++e;
    }
    return (uint8_t)(sign | ((uint32_t)(e + 7) << 3) | m3);  // a < 448 never reaches 480
}

// One element, converted from the input representation to storage.
__device__ __forceinline__ float load_new(const void *src, int dtype, int64_t i) {
    if (dtype == SPIRE_BF16) return bf16_to_f32(static_cast<const uint16_t *>(src)[i]);
    return static_cast<const float *>(src)[i];
}

__device__ __forceinline__ void store_elem(uint8_t *row, int es, int d, float x, float scale) {
    if (es == 4) reinterpret_cast<float *>(row)[d] = x;
    else if (es == 2) reinterpret_cast<uint16_t *>(row)[d] = f32_to_bf16_rne(x);
    else row[d] = f32_to_e4m3fn_sat(x / scale);
}

__device__ __forceinline__ void copy_row(uint8_t *dst, const uint8_t *src, int bytes, int lane) {
    for (int i = lane; i < bytes; i += 64) dst[i] = src[i];
}

// ---- target append --------------------------------------------------------------

struct AppendArgs {
    KvDev kv;
    const void *k_new, *v_new;  // [B, T, Hkv, D]
    int32_t new_dtype;
    const int32_t *positions;   // [B]
    int32_t B, T, Hkv, D;
};

__global__ __launch_bounds__(256) void kv_append_kernel(AppendArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (b, t, h)
    if (row >= (int64_t)a.B * a.T * a.Hkv) return;
    const int h = (int)(row % a.Hkv);
    const int64_t bt = row / a.Hkv;
    const int t = (int)(bt % a.T);
    const int b = (int)(bt / a.T);
    const int64_t j = (int64_t)a.positions[b] + t;
    if (j < 0) return;
    int64_t blk, tok;
    if (a.kv.page_size > 0) {
        const int64_t idx = j / a.kv.page_size;
        if (idx >= a.kv.max_blocks) return;
        const int page = a.kv.block_table[(int64_t)b * a.kv.max_blocks + idx];
        if (page < 0 || page >= a.kv.num_blocks) return;
        blk = page;
        tok = j - idx * a.kv.page_size;
    } else {
        if (j >= a.kv.capacity) return;
        blk = b;
        tok = j;
    }
    const int es = a.kv.elem;
    const int64_t off = (blk * a.kv.s_blk + (int64_t)h * a.kv.s_head + tok * a.kv.s_tok) * es;
    uint8_t *kr = const_cast<uint8_t *>(a.kv.k) + off;
    uint8_t *vr = const_cast<uint8_t *>(a.kv.v) + off;
    const float ks = es == 1 ? a.kv.k_scale[h] : 1.f;
    const float vs = es == 1 ? a.kv.v_scale[h] : 1.f;
    const int64_t src = row * a.D;
    for (int d = lane; d < a.D; d += 64) {
        store_elem(kr, es, d, load_new(a.k_new, a.new_dtype, src + d), ks);
        store_elem(vr, es, d, load_new(a.v_new, a.new_dtype, src + d), vs);
    }
}

hipError_t launch_kv_append(const KvDev &kv, const void *k_new, const void *v_new, int new_dtype,
                            const int32_t *positions, int B, int T, int Hkv, int D, hipStream_t st) {
    AppendArgs a{kv, k_new, v_new, new_dtype, positions, B, T, Hkv, D};
    const int64_t rows = (int64_t)B * T * Hkv;
    hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, a);
    return hipGetLastError();
}

// ---- draft write and rollback ----------------------------------------------------

struct DraftWriteArgs {
    KvDev sink, ring;
    const void *k_new, *v_new;  // [B, Hkv, D]
    int32_t new_dtype;
    const int32_t *seq_lens;    // [B]: the token is at position m_b - 1
    const int32_t *ring_offset; // [B]
    int32_t B, Hkv, D, S, W;
    uint8_t *spill_k, *spill_v; // [B, Hkv, D] storage elements, or null
    // rollback
    const int32_t *base_lens, *n_accepted;
    int32_t steps;
};

// Row of logical position p of sequence b, KV head h: sink row p < S, else
// ring slot (offset + p - S) mod W; null without storage for p.
__device__ __forceinline__ uint8_t *draft_row_ptr(const DraftWriteArgs &a, int b, int h, int64_t p, bool value) {
    if (p < 0) return nullptr;
    const KvDev &v = p < a.S ? a.sink : a.ring;
    int64_t tok;
    if (p < a.S) {
        tok = p;
    } else {
        if (a.W <= 0) return nullptr;
        int64_t o = a.ring_offset[b] % a.W;
        if (o < 0) o += a.W;
        tok = (o + (p - a.S) % a.W) % a.W;
    }
    const int64_t off = ((int64_t)b * v.s_blk + (int64_t)h * v.s_head + tok * v.s_tok) * v.elem;
    return const_cast<uint8_t *>(value ? v.v : v.k) + off;
}

__global__ __launch_bounds__(256) void draft_append_kernel(DraftWriteArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (b, h)
    if (row >= (int64_t)a.B * a.Hkv) return;
    const int h = (int)(row % a.Hkv), b = (int)(row / a.Hkv);
    const int64_t p = (int64_t)a.seq_lens[b] - 1;
    uint8_t *kr = draft_row_ptr(a, b, h, p, false);
    if (kr == nullptr) return;
    uint8_t *vr = draft_row_ptr(a, b, h, p, true);
    const int es = a.ring.elem;
    const int bytes = a.D * es;
    if (a.spill_k != nullptr) {  // keep what is overwritten
        copy_row(a.spill_k + row * bytes, kr, bytes, lane);
        copy_row(a.spill_v + row * bytes, vr, bytes, lane);
    }
    const bool sink = p < a.S;
    const float ks = es == 1 ? (sink ? a.sink.k_scale : a.ring.k_scale)[h] : 1.f;
    const float vs = es == 1 ? (sink ? a.sink.v_scale : a.ring.v_scale)[h] : 1.f;
    const int64_t src = row * a.D;
    for (int d = lane; d < a.D; d += 64) {
        store_elem(kr, es, d, load_new(a.k_new, a.new_dtype, src + d), ks);
        store_elem(vr, es, d, load_new(a.v_new, a.new_dtype, src + d), vs);
    }
}

__global__ __launch_bounds__(256) void draft_rollback_kernel(DraftWriteArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (b, h)
    if (row >= (int64_t)a.B * a.Hkv) return;
    const int h = (int)(row % a.Hkv), b = (int)(row / a.Hkv);
    const int n = a.n_accepted[b];
    const int bytes = a.D * a.ring.elem;
    const int64_t stride = (int64_t)a.B * a.Hkv * bytes;  // one step of the spill area
    for (int s = a.steps - 1; s > n && s >= 0; --s) {     // latest first
        const int64_t p = (int64_t)a.base_lens[b] + s;
        uint8_t *kr = draft_row_ptr(a, b, h, p, false);
        if (kr == nullptr) continue;
        uint8_t *vr = draft_row_ptr(a, b, h, p, true);
        copy_row(kr, a.spill_k + s * stride + row * bytes, bytes, lane);
        copy_row(vr, a.spill_v + s * stride + row * bytes, bytes, lane);
    }
}

hipError_t launch_draft_append(const KvDev &sink, const KvDev &ring, const void *k_new, const void *v_new,
                               int new_dtype, const int32_t *seq_lens, const int32_t *ring_offset, int B,
                               int Hkv, int D, int S, int W, void *spill_k, void *spill_v, hipStream_t st) {
    DraftWriteArgs a{sink, ring, k_new, v_new, new_dtype, seq_lens, ring_offset, B, Hkv, D, S, W,
                     static_cast<uint8_t *>(spill_k), static_cast<uint8_t *>(spill_v), nullptr, nullptr, 0};
    const int64_t rows = (int64_t)B * Hkv;
    hipLaunchKernelGGL(draft_append_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_draft_rollback(const KvDev &sink, const KvDev &ring, const void *spill_k,
                                 const void *spill_v, const int32_t *base_lens, const int32_t *n_accepted,
                                 int steps, const int32_t *ring_offset, int B, int Hkv, int D, int S, int W,
                                 hipStream_t st) {
    DraftWriteArgs a{sink, ring, nullptr, nullptr, 0, nullptr, ring_offset, B, Hkv, D, S, W,
                     const_cast<uint8_t *>(static_cast<const uint8_t *>(spill_k)),
                     const_cast<uint8_t *>(static_cast<const uint8_t *>(spill_v)), base_lens, n_accepted,
                     steps};
    const int64_t rows = (int64_t)B * Hkv;
    hipLaunchKernelGGL(draft_rollback_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace spire
