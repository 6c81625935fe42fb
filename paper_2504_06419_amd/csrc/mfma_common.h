// mfma_common.h -- building blocks shared by the matrix-core attention kernels
// (register-staged in attn_mfma.hip, LDS-staged in attn_staged.hip).
//
// Register layouts (lane l, n16 = l & 15, j = l >> 4) of one 32-key tile:
//   * MFMA A/B operands: lane l holds row/column n16 and the 8 consecutive
//     reduction indices 8j..8j+7; C: lane l holds rows 4j..4j+3, column n16.
//   * S^T = K Q^T: row m of key group mb is key 16mb + 4(m&3) + (m>>2), so the
//     C output of lane l is keys 16mb + 4i + j (i = 0..3) for row 16nb + n16.
//   * O^T += V^T P^T: the PV reduction index 8j+t is key 4t + j -- exactly the
//     S^T values lane l already holds (t < 4 from mb = 0, t >= 4 from mb = 1),
//     so P never leaves its lane; row m of dim block mb' is head dim 8m + mb',
//     so lane l needs dims 8 n16 .. 8 n16 + 7 of keys 4t + j, transposes those
//     8 keys x 8 dims in registers and owns output dims 32j .. 32j + 31.
//     The LDS-staged fp8 kernel instead reads V^T transposed from LDS: row m
//     of dim block mb' is head dim 16 mb' + m, and lane l owns output dims
//     16 mb' + 4j .. 16 mb' + 4j + 3 of every block mb'.
// fp8 (OCP e4m3fn) K/V are converted in registers (exact): K to bf16 for the
// QK product with the bf16 queries, V to fp16 for the PV product, whose P
// operand then rounds to fp16 (bf16 K/V keep bf16 P); the per-head K scale
// is folded into the softmax scale, the V scale into the final normalisation.
#pragma once

#include <float.h>

#include "spire_internal.h"

namespace spire {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((__vector_size__(16)));
typedef __bf16 bf16x2 __attribute__((__vector_size__(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

enum { MODE_CONTIG = 0, MODE_PAGED = 1, MODE_DRAFT = 2 };

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// 16 bytes per lane HBM -> LDS (global_load_lds_dwordx4): lane L's bytes land
// at l + 16 L.  The compiler does not track this LDS write, so readers wait
// on vmcnt explicitly (wait_vmcnt).  K/V rows are streamed once: the copies
// carry the nontemporal policy (nt), as the register loads do; a plain
// streaming probe read 6.8-7.1 TB/s with it and 5.9 TB/s without.
constexpr int kCpolNT = 2;
__device__ __forceinline__ void dma16(const uint8_t *g, lds_u8 *l) {
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void *>(g),
                                     reinterpret_cast<__attribute__((address_space(3))) void *>(l), 16, 0, kCpolNT);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

constexpr float kRescaleLog2 = 8.f;

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// two OCP e4m3fn bytes (selected half of `x`) -> two bf16 (exact, scale 1)
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t x) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, HI));
}
__device__ __forceinline__ u32x4 fp8x8_to_bf16x8(uint32_t a, uint32_t b) {
    u32x4 r;
    r.x = fp8x2_to_bf16x2<false>(a);
    r.y = fp8x2_to_bf16x2<true>(a);
    r.z = fp8x2_to_bf16x2<false>(b);
    r.w = fp8x2_to_bf16x2<true>(b);
    return r;
}
// the same to fp16: every e4m3fn value (subnormals included, |x| <= 448) is
// exact in fp16
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_to_f16x2(uint32_t x) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(x, 1.0f, HI));
}
__device__ __forceinline__ u32x4 fp8x8_to_f16x8(uint32_t a, uint32_t b) {
    u32x4 r;
    r.x = fp8x2_to_f16x2<false>(a);
    r.y = fp8x2_to_f16x2<true>(a);
    r.z = fp8x2_to_f16x2<false>(b);
    r.w = fp8x2_to_f16x2<true>(b);
    return r;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    bf16x2 v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
    f16x2 v = {(_Float16)lo, (_Float16)hi};
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// The PV product's operand type.  With fp8 K/V it is fp16: the values convert
// exactly and P keeps 11 significant bits (relative rounding error <= 2^-11;
// P <= 2^8 by the lazy reference maximum, far inside fp16's range).  With bf16
// K/V it is bf16, the values' own type (fp16 could not hold every bf16 value).
template <bool F16>
__device__ __forceinline__ uint32_t pack_p(float lo, float hi) {
    return F16 ? pack_f16x2(lo, hi) : pack_bf16x2(lo, hi);
}
template <bool F16>
__device__ __forceinline__ f32x4 mfma_pv(u32x4 a, u32x4 b, f32x4 c) {
    return F16 ? mfma_f16(a, b, c) : mfma_bf16(a, b, c);
}

// K/V rows are streamed once: nontemporal loads (the streaming cache policy)
// keep them from displacing anything in L2 and measurably raise HBM read rate.
__device__ __forceinline__ u32x4 ld16(const uint8_t *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}
__device__ __forceinline__ u32x2 ld8(const uint8_t *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(p));
}

template <bool FP8> struct TileRegs;
template <> struct TileRegs<false> { u32x4 k[2][4]; u32x4 v[8]; };  // bf16
template <> struct TileRegs<true> { u32x4 k[2][2]; u32x2 v[8]; };   // fp8

// Per-segment addressing state (uniform values).
struct SegAddr {
    const uint8_t *kseq, *vseq;      // contiguous/ring: (b, h) base; paged: head offset applied
    const uint8_t *ksink, *vsink;    // draft sinks (b, h) base
    const int32_t *table;            // paged: block table row of b
    int64_t blk_bytes;               // paged: bytes per page
    int64_t tok_bytes, sink_tok_bytes;
    int32_t n;                       // keys of the segment
    int32_t cap;                     // contiguous: rows per sequence
    int32_t ps, num_blocks;          // paged
    int32_t ps_shift;                // paged: log2(ps) when ps is a power of two, else -1
    int32_t nr, rs, W;               // draft: valid ring slots, first slot, window
};

template <bool FP8>
__device__ __forceinline__ void load_k_row(TileRegs<FP8> &T, int mb, const uint8_t *kp) {
    if (FP8) {
#pragma unroll
        for (int u = 0; u < 2; ++u) T.k[mb][u] = ld16(kp + 64 * u);
    } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) T.k[mb][c] = ld16(kp + 64 * c);
    }
}
template <bool FP8>
__device__ __forceinline__ void load_v_row(TileRegs<FP8> &T, int t, const uint8_t *vp) {
    if (FP8)
        *reinterpret_cast<u32x2 *>(&T.v[t]) = ld8(vp);
    else
        *reinterpret_cast<u32x4 *>(&T.v[t]) = ld16(vp);
}

// Draft key space: keys [0, nr) are the valid ring slots starting at slot rs
// (wrapping), keys [nr, nr + ns) the sink rows; keys beyond the segment are
// clamped to a valid row (their scores are masked and values zeroed).
// Branch-free (selects only), so that loads never sit under divergent control flow.
__device__ __forceinline__ const uint8_t *draft_row(const SegAddr &a, int j, bool value) {
    j = j < a.n ? j : (a.nr > 0 ? 0 : a.n - 1);
    // no keys at all (n = 0): ring slot 0 if there is a ring, else sink row 0
    j = j >= 0 ? j : (a.W > 0 ? 0 : a.nr);
    const bool sink = j >= a.nr;
    int s = a.rs + j;
    s = s >= a.W ? s - a.W : s;
    const uint8_t *ring = (value ? a.vseq : a.kseq) + (int64_t)s * a.tok_bytes;
    const uint8_t *snk = (value ? a.vsink : a.ksink) + (int64_t)(j - a.nr) * a.sink_tok_bytes;
    return sink ? snk : ring;
}

// Base byte offset of the contiguous 16-key group starting at key0, or -1 if
// the group is not one contiguous run of rows (only then per-lane addressing).
template <int MODE>
__device__ __forceinline__ int64_t group_base(const SegAddr &a, int key0) {
    if (MODE == MODE_CONTIG) {
        return key0 + 16 <= a.cap ? (int64_t)key0 * a.tok_bytes : -1;
    } else if (MODE == MODE_PAGED) {
        const int kk = key0 < a.n ? key0 : (a.n > 0 ? a.n - 1 : 0);  // n = 0: any valid row
        const uint32_t u = (uint32_t)kk;
        uint32_t idx, rin;
        if (a.ps_shift >= 0) {
            idx = u >> a.ps_shift;
            rin = u & (uint32_t)(a.ps - 1);
        } else {
            idx = u / (uint32_t)a.ps;
            rin = u - idx * (uint32_t)a.ps;
        }
        int page = uload(a.table, (int64_t)idx);
        page = page < 0 ? 0 : (page >= a.num_blocks ? a.num_blocks - 1 : page);
        // 32-bit products: the host routes only pages under 4 GB whose
        // ps rows span under 2 GB to these kernels
        return (int64_t)((uint64_t)(uint32_t)page * (uint32_t)a.blk_bytes) +
               (int64_t)((rin & ~15u) * (uint32_t)a.tok_bytes);
    } else {
        if (key0 + 16 > a.nr) return -1;
        int s = a.rs + key0;
        if (s >= a.W) s -= a.W;
        return s + 16 <= a.W ? (int64_t)s * a.tok_bytes : -1;
    }
}

template <bool FP8, int MODE>
__device__ __forceinline__ void load_tile(TileRegs<FP8> &T, const SegAddr &a, int tile, int lane) {
    const int n16 = lane & 15, j = lane >> 4;
    const int rho = 4 * (n16 & 3) + (n16 >> 2);
    const int key0 = tile * kMfmaTile;
    const int64_t g0 = group_base<MODE>(a, key0);
    const int64_t g1 = group_base<MODE>(a, key0 + 16);
    const int64_t koff = (int64_t)rho * a.tok_bytes + 16 * j;
    const int64_t voff = (int64_t)j * a.tok_bytes + (FP8 ? 8 : 16) * n16;
    if (MODE == MODE_PAGED || (g0 >= 0 && g1 >= 0)) {  // fast path: two contiguous 16-row groups
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) load_k_row<FP8>(T, mb, a.kseq + (mb ? g1 : g0) + koff);
#pragma unroll
        for (int t = 0; t < 8; ++t)
            load_v_row<FP8>(T, t, a.vseq + (t < 4 ? g0 : g1) + (int64_t)(4 * (t & 3)) * a.tok_bytes + voff);
        return;
    }
    // per-lane rows: contiguous tails past the capacity, ring wrap, sinks
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
        const int key = key0 + 16 * mb + rho;
        const uint8_t *kp;
        if (MODE == MODE_DRAFT) {
            kp = draft_row(a, key, false) + 16 * j;
        } else {
            kp = a.kseq + (int64_t)min(key, a.cap - 1) * a.tok_bytes + 16 * j;
        }
        load_k_row<FP8>(T, mb, kp);
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int key = key0 + 4 * t + j;
        const uint8_t *vp;
        if (MODE == MODE_DRAFT) {
            vp = draft_row(a, key, true) + (FP8 ? 8 : 16) * n16;
        } else {
            vp = a.vseq + (int64_t)min(key, a.cap - 1) * a.tok_bytes + (FP8 ? 8 : 16) * n16;
        }
        load_v_row<FP8>(T, t, vp);
    }
}

// Online-softmax state of NB row blocks.  Row sums of P either come from an
// extra MFMA with an all-ones operand (LS = true: no VALU adds, and the sum
// uses the same bf16-rounded P as the output) or from per-lane VALU partial
// sums reduced at the end (LS = false: 4 fewer registers per block, for the
// register-staged kernel, which is at its register limit).
template <int NB, bool LS> struct SoftmaxState {
    f32x4 acc[8][NB];            // O^T blocks
    f32x4 lsum[LS ? NB : 1];     // LS: row sums (every entry of a block equal)
    float l[LS ? 1 : NB];        // !LS: per-lane partial row sums
    float msub[NB];              // reference maximum (base 2), 0 while the row has none
    float thr[NB];               // rescale threshold on raw scores; -inf: no reference yet
    int lim[NB];
};

// Maximum of 8 scores with the NaN-propagating maximum (v_maximum3_f32): the
// IEEE-mode fmaxf would first quiet each matrix-core result with an extra
// instruction.  A NaN score (only from NaN keys inside the visible range)
// never passes the threshold test.
__device__ __forceinline__ float max3n(float a, float b, float c) {
    return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}
__device__ __forceinline__ float max8(f32x4 a, f32x4 b) {
    return __builtin_elementwise_maximum(max3n(a[0], a[1], a[2]),
                                         max3n(a[3], b[0], max3n(b[1], b[2], b[3])));
}

// 1.0 in both halves (bf16, fp16): the A operand whose product with P^T is the row sum
constexpr uint32_t kOnesBF16x2 = 0x3F803F80u;
constexpr uint32_t kOnesF16x2 = 0x3C003C00u;

// 2^x with the hardware instruction: no denormal results (they would stand for
// probabilities below 2^-126 of the row maximum and are dropped).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Query fragments: registers for NB <= 2, LDS (lane-private slots) beyond.
template <int NB, bool QLDS> struct QFrag;
template <int NB> struct QFrag<NB, false> {
    u32x4 r[NB][4];
    __device__ __forceinline__ void put(int nb, int c, u32x4 v, int) { r[nb][c] = v; }
    __device__ __forceinline__ u32x4 get(int nb, int c, int) const { return r[nb][c]; }
};
template <int NB> struct QFrag<NB, true> {
    u32x4 *lds;  // [NB][4][64] of this wave
    __device__ __forceinline__ void put(int nb, int c, u32x4 v, int lane) { lds[(nb * 4 + c) * 64 + lane] = v; }
    __device__ __forceinline__ u32x4 get(int nb, int c, int lane) const { return lds[(nb * 4 + c) * 64 + lane]; }
};

// VTR: T.v[mb] already holds the V^T operand of dim block mb in fp8 (element t
// = key 4t + j of dim 16 mb + n16, from a transposing LDS read); the output
// dims of block mb are then 16 mb .. 16 mb + 15 instead of 8 m + mb.
template <bool FP8, int NB, bool QLDS, bool LS, bool VTR = false>
__device__ __forceinline__ void compute_tile(TileRegs<FP8> &T, const QFrag<NB, QLDS> &qf,
                                             SoftmaxState<NB, LS> &st, int tile, int n, int full_lim,
                                             float sc, int lane) {
    const int j = lane >> 4;
    const int key0 = tile * kMfmaTile;

    // ---- S^T = K Q^T -------------------------------------------------------
    f32x4 s[2][NB];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) s[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        u32x4 kf[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            if (FP8) {
                const u32x4 raw = T.k[mb][c >> 1];
                kf[mb] = (c & 1) ? fp8x8_to_bf16x8(raw.z, raw.w) : fp8x8_to_bf16x8(raw.x, raw.y);
            } else {
                kf[mb] = T.k[mb][c];
            }
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const u32x4 q = qf.get(nb, c, lane);
            s[0][nb] = mfma_bf16(kf[0], q, s[0][nb]);
            s[1][nb] = mfma_bf16(kf[1], q, s[1][nb]);
        }
    }

    // ---- mask (only tiles reaching past a row's last visible key) ----------
    if (key0 + kMfmaTile > full_lim) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (key0 + 16 * mb + 4 * i + j >= st.lim[nb]) s[mb][nb][i] = -INFINITY;
    }

    // ---- online softmax (base 2, scale folded into the exponent) ------------
    // Each row keeps a reference maximum msub that only moves when a score of
    // the tile exceeds it by more than kRescaleLog2 (probabilities stay below
    // 2^kRescaleLog2, far inside the bf16/fp32 range).  The common path only
    // compares lane-local maxima with the row threshold thr = (msub + T) / sc;
    // the cross-lane row maximum and the accumulator rescale run only when
    // some row crosses it (a segment's first tile, rare jumps afterwards).
    float lmax[NB];
    bool over = false;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        lmax[nb] = max8(s[0][nb], s[1][nb]);
        over |= lmax[nb] > st.thr[nb];
    }
    if (__any(over)) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            float mx = fmaxf(lmax[nb], __shfl_xor(lmax[nb], 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            mx *= sc;  // sc > 0
            const float mold = st.thr[nb] == -INFINITY ? -INFINITY : st.msub[nb];
            const float mnew = mx > mold + kRescaleLog2 ? mx : mold;
            const float msub = mnew == -INFINITY ? 0.f : mnew;
            const float alpha = fast_exp2(mold - msub);  // 1 when unchanged, 0 from -inf
            st.msub[nb] = msub;
            // finite once a reference exists (-inf marks "none yet")
            st.thr[nb] = mnew == -INFINITY ? -INFINITY : fmaxf((mnew + kRescaleLog2) / sc, -FLT_MAX);
#pragma unroll
            for (int mb = 0; mb < 8; ++mb) st.acc[mb][nb] *= alpha;
            if constexpr (LS) st.lsum[nb] *= alpha;
            else st.l[nb] *= alpha;
        }
    }
    u32x4 pb[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        float p[2][4];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i) p[mb][i] = fast_exp2(fmaf(s[mb][nb][i], sc, -st.msub[nb]));
        if constexpr (!LS)
            st.l[nb] += ((p[0][0] + p[0][1]) + (p[0][2] + p[0][3])) +
                        ((p[1][0] + p[1][1]) + (p[1][2] + p[1][3]));
        pb[nb].x = pack_p<FP8>(p[0][0], p[0][1]);
        pb[nb].y = pack_p<FP8>(p[0][2], p[0][3]);
        pb[nb].z = pack_p<FP8>(p[1][0], p[1][1]);
        pb[nb].w = pack_p<FP8>(p[1][2], p[1][3]);
    }

    // ---- V: keys beyond the segment end are zeroed (storage there may be anything)
    u32x4 vb[8];
    if constexpr (VTR) {
        static_assert(FP8, "transposed V operands are read for fp8 only");
        if (key0 + kMfmaTile > n) {  // uniform: only a segment's last tile
            // byte t of every operand is key 4t + j
            uint32_t m0 = 0u, m1 = 0u;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                m0 |= (key0 + 4 * t + j < n ? 0xFFu : 0u) << (8 * t);
                m1 |= (key0 + 4 * (t + 4) + j < n ? 0xFFu : 0u) << (8 * t);
            }
#pragma unroll
            for (int mb = 0; mb < 8; ++mb) T.v[mb] = u32x2{T.v[mb].x & m0, T.v[mb].y & m1};
        }
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) vb[mb] = fp8x8_to_f16x8(T.v[mb].x, T.v[mb].y);
    } else {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            if (FP8) {
                const u32x2 raw = *reinterpret_cast<const u32x2 *>(&T.v[t]);
                vb[t] = fp8x8_to_f16x8(raw.x, raw.y);
            } else {
                vb[t] = *reinterpret_cast<const u32x4 *>(&T.v[t]);
            }
        }
        if (key0 + kMfmaTile > n) {  // uniform: only a segment's last tile
#pragma unroll
            for (int t = 0; t < 8; ++t)
                if (key0 + 4 * t + j >= n) vb[t] = u32x4{0u, 0u, 0u, 0u};
        }
    }

    // ---- O^T += V^T P^T, row sums += 1^T P^T ---------------------------------
    // Transpose 8 keys x 8 dims of 16-bit values with byte permutes: element t of
    // operand mb' is dim mb' (half mb'&1 of dword mb'>>1) of key t.
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
        const int w = mb >> 1;
        const uint32_t sel = (mb & 1) ? 0x07060302u : 0x05040100u;
        u32x4 a;
        if constexpr (VTR) {
            a = vb[mb];
        } else {
            a.x = __builtin_amdgcn_perm(vb[1][w], vb[0][w], sel);
            a.y = __builtin_amdgcn_perm(vb[3][w], vb[2][w], sel);
            a.z = __builtin_amdgcn_perm(vb[5][w], vb[4][w], sel);
            a.w = __builtin_amdgcn_perm(vb[7][w], vb[6][w], sel);
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) st.acc[mb][nb] = mfma_pv<FP8>(a, pb[nb], st.acc[mb][nb]);
    }
    if constexpr (LS) {
        constexpr uint32_t one2 = FP8 ? kOnesF16x2 : kOnesBF16x2;
        const u32x4 ones = u32x4{one2, one2, one2, one2};
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) st.lsum[nb] = mfma_pv<FP8>(ones, pb[nb], st.lsum[nb]);
    }
}

// ---- the partition computed inside an attention kernel --------------------------
// Every workgroup of THREADS threads computes the prefix sums of the
// (tiles + phantom positions) of all sequences into s_pre[0..B] (the plan
// kernel's arithmetic); workgroup 0 also stores the key counts and prefix sums
// in the workspace, where the combine reads them.  Ends with a barrier.
template <int THREADS>
__device__ __forceinline__ void plan_in_kernel(const Problem &p, const Plan &pl, int32_t *s_pre,
                                               int32_t *s_sum) {
    const int tid = threadIdx.x, B = p.B;
    const int per = (B + THREADS - 1) / THREADS;
    const int b0 = tid * per;
    const int b1 = b0 + per < B ? b0 + per : B;
    const bool store = blockIdx.x == 0;
    int local = 0;
    for (int b = b0; b < b1; ++b) {
        const int n = effective_keys(p, b);
        if (store) pl.nkeys[b] = n;
        const int span = (n > 0 ? (n + pl.tile - 1) / pl.tile : 1) + pl.seg_cost;
        s_pre[b] = span;
        local += span;
    }
    s_sum[tid] = local;
    __syncthreads();
    for (int off = 1; off < THREADS; off <<= 1) {  // inclusive scan of the per-thread sums
        const int v = tid >= off ? s_sum[tid - off] : 0;
        __syncthreads();
        s_sum[tid] += v;
        __syncthreads();
    }
    int run = s_sum[tid] - local;
    for (int b = b0; b < b1; ++b) {
        const int span = s_pre[b];
        s_pre[b] = run;
        if (store) pl.prefix[b] = run;
        run += span;
    }
    if (tid == THREADS - 1) {
        s_pre[B] = s_sum[THREADS - 1];
        if (store) pl.prefix[B] = s_sum[THREADS - 1];
    }
    __syncthreads();
}

// (segment, tile) holding flattened position x (0 <= x < T) under prefix sums s_pre
__device__ __forceinline__ void locate(const int32_t *s_pre, int B, int units, int64_t x, int &seg, int &tile) {
    int lo = 0, hi = B - 1;  // last b with units * s_pre[b] <= x
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((int64_t)s_pre[mid] * units <= x) lo = mid; else hi = mid - 1;
    }
    const int span = s_pre[lo + 1] - s_pre[lo];
    const int64_t rel = x - (int64_t)s_pre[lo] * units;
    seg = lo * units + (int)(rel / span);
    tile = (int)(rel % span);
}

// ---- per-segment setup and finalisation ---------------------------------------

template <int MODE>
__device__ __forceinline__ SegAddr make_seg_addr(const Problem &p, int b, int h, int n) {
    SegAddr a;
    a.n = n;
    a.tok_bytes = p.kv.s_tok * p.kv.elem;
    a.cap = 0;
    if (MODE == MODE_PAGED) {
        a.kseq = p.kv.k + (int64_t)h * p.kv.s_head * p.kv.elem;
        a.vseq = p.kv.v + (int64_t)h * p.kv.s_head * p.kv.elem;
        a.table = p.kv.block_table + (int64_t)b * p.kv.max_blocks;
        a.blk_bytes = p.kv.s_blk * p.kv.elem;
        a.ps = p.kv.page_size;
        a.ps_shift = (a.ps & (a.ps - 1)) == 0 ? __builtin_ctz(a.ps) : -1;
        a.num_blocks = p.kv.num_blocks;
    } else {
        const int64_t off = ((int64_t)b * p.kv.s_blk + (int64_t)h * p.kv.s_head) * p.kv.elem;
        a.kseq = p.kv.k + off;
        a.vseq = p.kv.v + off;
        a.cap = p.kv.capacity;
    }
    if (MODE == MODE_DRAFT) {
        const int64_t soff = ((int64_t)b * p.sink.s_blk + (int64_t)h * p.sink.s_head) * p.sink.elem;
        a.ksink = p.sink.k + soff;
        a.vsink = p.sink.v + soff;
        a.sink_tok_bytes = p.sink.s_tok * p.sink.elem;
        const int mraw = uload(p.lens, b);
        const int m = mraw < 0 ? 0 : mraw;
        const int ns = m < p.S ? m : p.S;
        a.nr = n - ns;
        a.W = p.W;
        int rs = 0;
        if (p.W > 0 && a.nr < p.W) {  // ring not yet full: start at the oldest valid slot
            int first = m - p.S - p.W;
            first = first < 0 ? 0 : first;
            int o = uload(p.ring_offset, b) % p.W;
            if (o < 0) o += p.W;
            rs = (o + first % p.W) % p.W;
        }
        a.rs = rs;  // a full ring is read in physical slot order
    }
    return a;
}

// Reset the softmax state of row blocks rb0 .. rb0+NB-1.
template <int NB, bool LS>
__device__ __forceinline__ void reset_rows(const Problem &p, int n, int rb0, SoftmaxState<NB, LS> &st,
                                           int lane) {
    const int n16 = lane & 15;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int r = 16 * (rb0 + nb) + n16;
        st.msub[nb] = 0.f;
        st.thr[nb] = -INFINITY;
        if constexpr (LS) st.lsum[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        else st.l[nb] = 0.f;
        st.lim[nb] = r < p.R ? visible_limit(p, n, r) : n;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) st.acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
}

// Load the queries of row blocks rb0 .. rb0+NB-1 (rows 16(rb0+nb) + n16) of
// segment (b, h) as MFMA B operands.
template <bool FP8, int NB, bool QLDS>
__device__ __forceinline__ void load_rows_q(const Problem &p, int b, int h, int rb0,
                                            QFrag<NB, QLDS> &qf, int lane) {
    const int n16 = lane & 15, j = lane >> 4;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int r = 16 * (rb0 + nb) + n16;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int d0 = FP8 ? 64 * (c >> 1) + 16 * j + 8 * (c & 1) : 32 * c + 8 * j;
            u32x4 v = u32x4{0u, 0u, 0u, 0u};
            if (r < p.R) v = *reinterpret_cast<const u32x4 *>(p.q + (row_offset(p, b, h, r) + d0) * 2);
            qf.put(nb, c, v, lane);
        }
    }
}

template <bool FP8, int NB, bool QLDS, bool LS>
__device__ __forceinline__ void begin_rows(const Problem &p, int b, int h, int n, int rb0,
                                           QFrag<NB, QLDS> &qf, SoftmaxState<NB, LS> &st, int lane) {
    reset_rows<NB, LS>(p, n, rb0, st, lane);
    load_rows_q<FP8, NB, QLDS>(p, b, h, rb0, qf, lane);
}

// Write the rows of blocks rb0 .. rb0+NB-1: final output + lse when the worker
// covered the whole segment, else a partial (normalised output, base-2 lse)
// into workspace slot `slot`.
template <bool FP8, int NB, bool LS, bool VTR = false>
__device__ __forceinline__ void end_rows(const Problem &p, const Plan &pl, SoftmaxState<NB, LS> &st,
                                         int b, int h, int rb0, bool whole, int64_t slot, int lane) {
    const int n16 = lane & 15, j = lane >> 4;
    const float vs = FP8 ? uload(p.kv.v_scale, h) : 1.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        float l;
        if constexpr (LS) {
            l = st.lsum[nb][0];  // every entry of the block holds the row sum
        } else {
            l = st.l[nb];
            l += __shfl_xor(l, 16);
            l += __shfl_xor(l, 32);
        }
        const int r = 16 * (rb0 + nb) + n16;
        if (r >= p.R) continue;
        // l == 0: no visible key (zeros, lse -inf); l NaN: a NaN key or a +inf
        // score was visible, and the row is NaN as the definition has it
        const float inv = l > 0.f ? vs / l : (l == 0.f ? 0.f : l);
        const float lse2 = l > 0.f ? st.msub[nb] + log2f(l) : (l == 0.f ? -INFINITY : l);
        if (VTR && whole) {  // lane holds dims 16 mb + 4j .. 16 mb + 4j + 3 of every block mb
            const int64_t off = row_offset(p, b, h, r) + 4 * j;
#pragma unroll
            for (int mb = 0; mb < 8; ++mb) {
                const f32x4 v = st.acc[mb][nb] * inv;
                if (p.out_dtype == SPIRE_BF16)
                    *reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(p.out) + off + 16 * mb) =
                        u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                else
                    *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(p.out) + off + 16 * mb) = v;
            }
            if (j == 0 && p.lse != nullptr) p.lse[lse_index(p, b, h, r)] = lse2 * 0.69314718055994531f;
        } else if (VTR) {
            float *o = pl.part_o + (slot * pl.rows + r) * (int64_t)p.D + 4 * j;
#pragma unroll
            for (int mb = 0; mb < 8; ++mb) *reinterpret_cast<f32x4 *>(o + 16 * mb) = st.acc[mb][nb] * inv;
            if (j == 0) pl.part_lse[slot * pl.rows + r] = lse2;
        } else if (whole) {
            const int64_t off = row_offset(p, b, h, r) + 32 * j;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (p.out_dtype == SPIRE_BF16) {
                    u32x4 o;
                    o.x = pack_bf16x2(st.acc[0][nb][i] * inv, st.acc[1][nb][i] * inv);
                    o.y = pack_bf16x2(st.acc[2][nb][i] * inv, st.acc[3][nb][i] * inv);
                    o.z = pack_bf16x2(st.acc[4][nb][i] * inv, st.acc[5][nb][i] * inv);
                    o.w = pack_bf16x2(st.acc[6][nb][i] * inv, st.acc[7][nb][i] * inv);
                    *reinterpret_cast<u32x4 *>(reinterpret_cast<uint16_t *>(p.out) + off + 8 * i) = o;
                } else {
                    float *o = reinterpret_cast<float *>(p.out) + off + 8 * i;
                    *reinterpret_cast<f32x4 *>(o) = f32x4{st.acc[0][nb][i], st.acc[1][nb][i],
                                                          st.acc[2][nb][i], st.acc[3][nb][i]} * inv;
                    *reinterpret_cast<f32x4 *>(o + 4) = f32x4{st.acc[4][nb][i], st.acc[5][nb][i],
                                                              st.acc[6][nb][i], st.acc[7][nb][i]} * inv;
                }
            }
            if (j == 0 && p.lse != nullptr) p.lse[lse_index(p, b, h, r)] = lse2 * 0.69314718055994531f;
        } else {
            float *o = pl.part_o + (slot * pl.rows + r) * (int64_t)p.D + 32 * j;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                *reinterpret_cast<f32x4 *>(o + 8 * i) = f32x4{st.acc[0][nb][i], st.acc[1][nb][i],
                                                              st.acc[2][nb][i], st.acc[3][nb][i]} * inv;
                *reinterpret_cast<f32x4 *>(o + 8 * i + 4) = f32x4{st.acc[4][nb][i], st.acc[5][nb][i],
                                                                  st.acc[6][nb][i], st.acc[7][nb][i]} * inv;
            }
            if (j == 0) pl.part_lse[slot * pl.rows + r] = lse2;
        }
    }
}

}  // namespace spire
