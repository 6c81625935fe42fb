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
// Vector paths (D a multiple of 4, inputs, storage and spill rows aligned to
// their 4-element width): one thread per 4 consecutive elements of a row,
// 16 / 8 / 4-byte accesses for f32 / bf16 / fp8 storage, the input loads
// issued before the dependent position -> page -> row chain.  Otherwise one
// wave per row, element by element.  Either way every write stays inside the
// storage the descriptors describe (positions without storage are skipped).
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

// ---- 4-element quads (vector paths) ---------------------------------------------

typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

// elements 4q .. 4q+3 of an input row starting at element i0
__device__ __forceinline__ void load_quad(const void *src, int dtype, int64_t i0, float x[4]) {
    if (dtype == SPIRE_BF16) {
        const u32x2v v = *reinterpret_cast<const u32x2v *>(static_cast<const uint16_t *>(src) + i0);
        x[0] = __uint_as_float(v.x << 16);
        x[1] = __uint_as_float(v.x & 0xFFFF0000u);
        x[2] = __uint_as_float(v.y << 16);
        x[3] = __uint_as_float(v.y & 0xFFFF0000u);
    } else {
        const float4 v = *reinterpret_cast<const float4 *>(static_cast<const float *>(src) + i0);
        x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
    }
}

// store 4 elements at byte `at` (4 * ES-aligned) in the storage representation
template <int ES>
__device__ __forceinline__ void store_quad(uint8_t *at, const float x[4], float scale) {
    if constexpr (ES == 4) {
        *reinterpret_cast<float4 *>(at) = make_float4(x[0], x[1], x[2], x[3]);
    } else if constexpr (ES == 2) {
        u32x2v v;
        v.x = f32_to_bf16_rne(x[0]) | ((uint32_t)f32_to_bf16_rne(x[1]) << 16);
        v.y = f32_to_bf16_rne(x[2]) | ((uint32_t)f32_to_bf16_rne(x[3]) << 16);
        *reinterpret_cast<u32x2v *>(at) = v;
    } else {
        uint32_t v = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) v |= (uint32_t)f32_to_e4m3fn_sat(x[c] / scale) << (8 * c);
        *reinterpret_cast<uint32_t *>(at) = v;
    }
}

template <int ES> struct QuadBits;
template <> struct QuadBits<4> { typedef u32x4v T; };
template <> struct QuadBits<2> { typedef u32x2v T; };
template <> struct QuadBits<1> { typedef uint32_t T; };

template <int ES>
__device__ __forceinline__ void copy_quad(uint8_t *dst, const uint8_t *src) {
    typedef typename QuadBits<ES>::T Q;
    *reinterpret_cast<Q *>(dst) = *reinterpret_cast<const Q *>(src);
}

// true when every row of the view starts on a `bytes` boundary
__device__ __host__ __forceinline__ bool rows_aligned(const KvDev &v, int bytes) {
    const int64_t m = bytes / v.elem;  // stride granularity in elements
    return ((uintptr_t)v.k % bytes) == 0 && ((uintptr_t)v.v % bytes) == 0 && v.s_blk % m == 0 &&
           v.s_head % m == 0 && v.s_tok % m == 0;
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

// (the host launches the vector kernels only when B * T * Hkv * D / 4 < 2^31,
// so the thread's indices fit 32-bit arithmetic)
template <int ES>
__global__ __launch_bounds__(256) void kv_append_vec_kernel(AppendArgs a) {
    const uint32_t nq = (uint32_t)a.D >> 2;
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;  // (b, t, h, quad)
    if (i >= (uint32_t)a.B * a.T * a.Hkv * nq) return;
    const uint32_t row = i / nq;
    const int q = (int)(i - row * nq);
    float kx[4], vx[4];
    load_quad(a.k_new, a.new_dtype, (int64_t)row * a.D + 4 * q, kx);
    load_quad(a.v_new, a.new_dtype, (int64_t)row * a.D + 4 * q, vx);
    const uint32_t bt = row / (uint32_t)a.Hkv;
    const int h = (int)(row - bt * (uint32_t)a.Hkv);
    const uint32_t b32 = bt / (uint32_t)a.T;
    const int t = (int)(bt - b32 * (uint32_t)a.T);
    const int b = (int)b32;
    const int64_t j = (int64_t)a.positions[b] + t;
    if (j < 0) return;
    int64_t blk, tok;
    if (a.kv.page_size > 0) {
        const int ps = a.kv.page_size;
        const int64_t idx = (ps & (ps - 1)) == 0 ? j >> __builtin_ctz((unsigned)ps) : j / ps;
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
    const int64_t off = (blk * a.kv.s_blk + (int64_t)h * a.kv.s_head + tok * a.kv.s_tok) * ES + 4 * ES * q;
    const float ks = ES == 1 ? a.kv.k_scale[h] : 1.f;
    const float vs = ES == 1 ? a.kv.v_scale[h] : 1.f;
    store_quad<ES>(const_cast<uint8_t *>(a.kv.k) + off, kx, ks);
    store_quad<ES>(const_cast<uint8_t *>(a.kv.v) + off, vx, vs);
}

// inputs [B, T or 1, Hkv, D] of `dtype` readable 4 elements at a time
static bool inputs_vec_ok(const void *k_new, const void *v_new, int dtype, int D) {
    const uintptr_t al = dtype == SPIRE_BF16 ? 8u : 16u;
    return D % 4 == 0 && ((uintptr_t)k_new % al) == 0 && ((uintptr_t)v_new % al) == 0;
}

hipError_t launch_kv_append(const KvDev &kv, const void *k_new, const void *v_new, int new_dtype,
                            const int32_t *positions, int B, int T, int Hkv, int D, hipStream_t st) {
    AppendArgs a{kv, k_new, v_new, new_dtype, positions, B, T, Hkv, D};
    const int64_t rows = (int64_t)B * T * Hkv;
    const int es = kv.elem;
    if (inputs_vec_ok(k_new, v_new, new_dtype, D) && rows_aligned(kv, 4 * es) && rows * (D / 4) < (1LL << 31)) {
        const dim3 grid((unsigned)((rows * (D / 4) + 255) / 256));
        if (es == 4) hipLaunchKernelGGL(kv_append_vec_kernel<4>, grid, dim3(256), 0, st, a);
        else if (es == 2) hipLaunchKernelGGL(kv_append_vec_kernel<2>, grid, dim3(256), 0, st, a);
        else hipLaunchKernelGGL(kv_append_vec_kernel<1>, grid, dim3(256), 0, st, a);
    } else {
        hipLaunchKernelGGL(kv_append_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, a);
    }
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

template <int ES>
__global__ __launch_bounds__(256) void draft_append_vec_kernel(DraftWriteArgs a) {
    const uint32_t nq = (uint32_t)a.D >> 2;
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;  // (b, h, quad)
    if (i >= (uint32_t)a.B * a.Hkv * nq) return;
    const uint32_t row = i / nq;
    const int q = (int)(i - row * nq);
    float kx[4], vx[4];
    load_quad(a.k_new, a.new_dtype, (int64_t)row * a.D + 4 * q, kx);
    load_quad(a.v_new, a.new_dtype, (int64_t)row * a.D + 4 * q, vx);
    const uint32_t b32 = row / (uint32_t)a.Hkv;
    const int h = (int)(row - b32 * (uint32_t)a.Hkv), b = (int)b32;
    const int64_t p = (int64_t)a.seq_lens[b] - 1;
    uint8_t *kr = draft_row_ptr(a, b, h, p, false);
    if (kr == nullptr) return;
    uint8_t *vr = draft_row_ptr(a, b, h, p, true);
    const int64_t at = 4 * ES * q;
    if (a.spill_k != nullptr) {  // keep what is overwritten (same thread, same bytes: in order)
        const int64_t sp = (int64_t)row * a.D * ES + at;
        copy_quad<ES>(a.spill_k + sp, kr + at);
        copy_quad<ES>(a.spill_v + sp, vr + at);
    }
    const bool sink = p < a.S;
    const float ks = ES == 1 ? (sink ? a.sink.k_scale : a.ring.k_scale)[h] : 1.f;
    const float vs = ES == 1 ? (sink ? a.sink.v_scale : a.ring.v_scale)[h] : 1.f;
    store_quad<ES>(kr + at, kx, ks);
    store_quad<ES>(vr + at, vx, vs);
}

// Row of position p given the ring offset already reduced to [0, W).
__device__ __forceinline__ uint8_t *draft_row_at(const DraftWriteArgs &a, int b, int h, int64_t p, int64_t o,
                                                 bool value) {
    if (p < 0) return nullptr;
    const KvDev &v = p < a.S ? a.sink : a.ring;
    int64_t tok;
    if (p < a.S) {
        tok = p;
    } else {
        if (a.W <= 0) return nullptr;
        tok = (o + (p - a.S) % a.W) % a.W;
    }
    const int64_t off = ((int64_t)b * v.s_blk + (int64_t)h * v.s_head + tok * v.s_tok) * v.elem;
    return const_cast<uint8_t *>(value ? v.v : v.k) + off;
}

// The spilled quads of up to kRollbackChunk rejected steps are loaded before
// any is stored (the spill area never overlaps the cache), then stored latest
// step first, so steps that share a slot still unwind in order.
constexpr int kRollbackChunk = 8;

template <int ES>
__global__ __launch_bounds__(256) void draft_rollback_vec_kernel(DraftWriteArgs a) {
    typedef typename QuadBits<ES>::T Q;
    const uint32_t nq = (uint32_t)a.D >> 2;
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;  // (b, h, quad)
    if (i >= (uint32_t)a.B * a.Hkv * nq) return;
    const uint32_t row = i / nq;
    const int q = (int)(i - row * nq);
    const uint32_t b32 = row / (uint32_t)a.Hkv;
    const int h = (int)(row - b32 * (uint32_t)a.Hkv), b = (int)b32;
    const int n = a.n_accepted[b];
    const int64_t base = a.base_lens[b];
    int64_t o = 0;
    if (a.W > 0) {
        o = a.ring_offset[b] % a.W;
        if (o < 0) o += a.W;
    }
    const int64_t bytes = (int64_t)a.D * ES;
    const int64_t stride = (int64_t)a.B * a.Hkv * bytes;  // one step of the spill area
    const int64_t at = 4 * ES * q;
    for (int s0 = a.steps - 1; s0 > n && s0 >= 0; s0 -= kRollbackChunk) {
        Q kq[kRollbackChunk], vq[kRollbackChunk];
#pragma unroll
        for (int u = 0; u < kRollbackChunk; ++u) {
            const int s = s0 - u;
            if (s > n && s >= 0) {
                kq[u] = *reinterpret_cast<const Q *>(a.spill_k + s * stride + (int64_t)row * bytes + at);
                vq[u] = *reinterpret_cast<const Q *>(a.spill_v + s * stride + (int64_t)row * bytes + at);
            }
        }
#pragma unroll
        for (int u = 0; u < kRollbackChunk; ++u) {
            const int s = s0 - u;
            if (s > n && s >= 0) {
                uint8_t *kr = draft_row_at(a, b, h, base + s, o, false);
                if (kr == nullptr) continue;
                uint8_t *vr = draft_row_at(a, b, h, base + s, o, true);
                *reinterpret_cast<Q *>(kr + at) = kq[u];
                *reinterpret_cast<Q *>(vr + at) = vq[u];
            }
        }
    }
}

// sinks, ring and spill rows all on 4-element boundaries
static bool draft_vec_ok(const KvDev &sink, const KvDev &ring, const void *spill_k, const void *spill_v, int D) {
    const int bytes = 4 * ring.elem;
    return D % 4 == 0 && rows_aligned(sink, bytes) && rows_aligned(ring, bytes) &&
           ((uintptr_t)spill_k % bytes) == 0 && ((uintptr_t)spill_v % bytes) == 0;
}

hipError_t launch_draft_append(const KvDev &sink, const KvDev &ring, const void *k_new, const void *v_new,
                               int new_dtype, const int32_t *seq_lens, const int32_t *ring_offset, int B,
                               int Hkv, int D, int S, int W, void *spill_k, void *spill_v, hipStream_t st) {
    DraftWriteArgs a{sink, ring, k_new, v_new, new_dtype, seq_lens, ring_offset, B, Hkv, D, S, W,
                     static_cast<uint8_t *>(spill_k), static_cast<uint8_t *>(spill_v), nullptr, nullptr, 0};
    const int64_t rows = (int64_t)B * Hkv;
    const int es = ring.elem;
    if (inputs_vec_ok(k_new, v_new, new_dtype, D) && draft_vec_ok(sink, ring, spill_k, spill_v, D) &&
        rows * (D / 4) < (1LL << 31)) {
        const dim3 grid((unsigned)((rows * (D / 4) + 255) / 256));
        if (es == 4) hipLaunchKernelGGL(draft_append_vec_kernel<4>, grid, dim3(256), 0, st, a);
        else if (es == 2) hipLaunchKernelGGL(draft_append_vec_kernel<2>, grid, dim3(256), 0, st, a);
        else hipLaunchKernelGGL(draft_append_vec_kernel<1>, grid, dim3(256), 0, st, a);
    } else {
        hipLaunchKernelGGL(draft_append_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, a);
    }
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
    const int es = ring.elem;
    if (draft_vec_ok(sink, ring, spill_k, spill_v, D) && rows * (D / 4) < (1LL << 31)) {
        const dim3 grid((unsigned)((rows * (D / 4) + 255) / 256));
        if (es == 4) hipLaunchKernelGGL(draft_rollback_vec_kernel<4>, grid, dim3(256), 0, st, a);
        else if (es == 2) hipLaunchKernelGGL(draft_rollback_vec_kernel<2>, grid, dim3(256), 0, st, a);
        else hipLaunchKernelGGL(draft_rollback_vec_kernel<1>, grid, dim3(256), 0, st, a);
    } else {
        hipLaunchKernelGGL(draft_rollback_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, st, a);
    }
    return hipGetLastError();
}

}  // namespace spire
