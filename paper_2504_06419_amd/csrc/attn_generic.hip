// attn_generic.hip -- split-KV partial attention on the vector ALUs.
//
// Serves every request the matrix-core kernel does not take (fp32 K/V or Q,
// head_dim 64, contiguous caches whose capacity is not a multiple of 16, page
// sizes that are not multiples of 16, draft views whose fp8 scales differ) and
// is a second, independently written GPU path for cross-checks.  It keeps fp32
// arithmetic throughout (no bf16 rounding of probabilities).
//
// One wave per workgroup is one worker of the stream-K partition; a unit is
// (KV head h, block of 16 query rows).  Per 64-key tile: lane l scores key
// kb + l against the 16 rows (queries staged in LDS), the row maxima are
// reduced across the wave, probabilities go through LDS, and for the value
// product lane l owns head dims l and l + 64.
#include "spire_internal.h"

namespace spire {

constexpr int RB = kGenericRowBlock;   // 16 rows per unit
constexpr int KT = kGenericTile;       // 64 keys per tile
constexpr int kMaxD = 128;

// OCP e4m3fn byte -> fp32 (independent of the matrix-core path's converter)
__device__ __forceinline__ float e4m3fn_to_f32(uint32_t x) {
    const uint32_t s = (x >> 7) & 1u, e = (x >> 3) & 15u, m = x & 7u;
    float v;
    if (e == 15u && m == 7u) v = __uint_as_float(0x7fc00000u);
    else if (e == 0u) v = (float)m * 0.001953125f;                 // m * 2^-9
    else v = __uint_as_float(((e + 120u) << 23) | (m << 20));       // (1 + m/8) 2^(e-7)
    return s ? -v : v;
}

__device__ __forceinline__ float load_elem(const uint8_t *row, int d, int dtype) {
    if (dtype == SPIRE_F32) return reinterpret_cast<const float *>(row)[d];
    if (dtype == SPIRE_BF16) return bf16_to_f32(reinterpret_cast<const uint16_t *>(row)[d]);
    return e4m3fn_to_f32(row[d]);
}

struct RowRef {
    const uint8_t *k, *v;
    float ks, vs;
};

// Storage row of key j (< n) of segment (b, h); `j` must be a valid key.
__device__ __forceinline__ RowRef key_row(const Problem &p, int b, int h, int j, int ns, int rs) {
    RowRef r;
    if (p.draft) {
        if (j < ns) {
            const KvDev &s = p.sink;
            const int64_t off = ((int64_t)b * s.s_blk + (int64_t)h * s.s_head + (int64_t)j * s.s_tok) * s.elem;
            r.k = s.k + off; r.v = s.v + off;
            r.ks = s.k_scale ? s.k_scale[h] : 1.f;
            r.vs = s.v_scale ? s.v_scale[h] : 1.f;
            return r;
        }
        int slot = rs + (j - ns);
        while (slot >= p.W) slot -= p.W;
        const KvDev &c = p.kv;
        const int64_t off = ((int64_t)b * c.s_blk + (int64_t)h * c.s_head + (int64_t)slot * c.s_tok) * c.elem;
        r.k = c.k + off; r.v = c.v + off;
        r.ks = c.k_scale ? c.k_scale[h] : 1.f;
        r.vs = c.v_scale ? c.v_scale[h] : 1.f;
        return r;
    }
    const KvDev &c = p.kv;
    int64_t blk, tok;
    if (c.page_size > 0) {
        int page = c.block_table[(int64_t)b * c.max_blocks + j / c.page_size];
        page = page < 0 ? 0 : (page >= c.num_blocks ? c.num_blocks - 1 : page);
        blk = page;
        tok = j % c.page_size;
    } else {
        blk = b;
        tok = j;
    }
    const int64_t off = (blk * c.s_blk + (int64_t)h * c.s_head + tok * c.s_tok) * c.elem;
    r.k = c.k + off; r.v = c.v + off;
    r.ks = c.k_scale ? c.k_scale[h] : 1.f;
    r.vs = c.v_scale ? c.v_scale[h] : 1.f;
    return r;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

// One 16-row unit (rows r0 .. r0+15 of KV head h of sequence b, of n keys)
// over tiles [t0, t1): queries in qs, probabilities through ps.  Writes the
// final rows when `whole`, else a partial into workspace slot `slot`.  A value
// is only accumulated for the rows that see its key, so that a non-finite
// value of a key some rows mask reaches only the rows that see it.
__device__ __forceinline__ void generic_unit(const Problem &p, const Plan &pl, int b, int h, int r0, int n,
                                             int ns, int rs, int t0, int t1, bool whole, int64_t slot, int lane,
                                             float (*qs)[kMaxD], float (*ps)[KT]) {
    const int D = p.D;
    __syncthreads();  // previous unit finished reading qs / ps
    for (int idx = lane; idx < RB * D; idx += 64) {
        const int r = idx / D, d = idx - (idx / D) * D;
        float v = 0.f;
        if (r0 + r < p.R) {
            const int64_t off = row_offset(p, b, h, r0 + r) + d;
            v = p.q_dtype == SPIRE_F32 ? reinterpret_cast<const float *>(p.q)[off]
                                       : bf16_to_f32(reinterpret_cast<const uint16_t *>(p.q)[off]);
        }
        qs[r][d] = v;
    }
    __syncthreads();

    float m[RB], l[RB], acc[RB][2];
    int lim[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        m[r] = -INFINITY; l[r] = 0.f; acc[r][0] = 0.f; acc[r][1] = 0.f;
        lim[r] = (r0 + r < p.R) ? visible_limit(p, n, r0 + r) : n;
    }

    for (int t = t0; t < t1 && n > 0; ++t) {
        const int kb = t * KT;
        const int key = kb + lane;
        const int kc = key < n ? key : n - 1;
        const RowRef rr = key_row(p, b, h, kc, ns, rs);
        float s[RB];
#pragma unroll
        for (int r = 0; r < RB; ++r) s[r] = 0.f;
        for (int d = 0; d < D; ++d) {
            const float kx = load_elem(rr.k, d, p.kv_dtype);
#pragma unroll
            for (int r = 0; r < RB; ++r) s[r] += kx * qs[r][d];
        }
        const float sc = p.sm_scale_log2 * rr.ks;
#pragma unroll
        for (int r = 0; r < RB; ++r) {
            float x = key < lim[r] ? s[r] * sc : -INFINITY;
            const float mnew = fmaxf(m[r], wave_max(x));
            const float msub = mnew == -INFINITY ? 0.f : mnew;
            const float alpha = exp2f(m[r] - msub);
            const float pr = exp2f(x - msub);
            m[r] = mnew;
            l[r] = l[r] * alpha + pr;
            acc[r][0] *= alpha;
            acc[r][1] *= alpha;
            ps[r][lane] = pr;
        }
        __syncthreads();
        const int nv = n - kb < KT ? n - kb : KT;
        for (int tk = 0; tk < nv; ++tk) {
            const RowRef vr = key_row(p, b, h, kb + tk, ns, rs);
            const float v0 = load_elem(vr.v, lane, p.kv_dtype) * vr.vs;
            const float v1 = lane + 64 < D ? load_elem(vr.v, lane + 64, p.kv_dtype) * vr.vs : 0.f;
#pragma unroll
            for (int r = 0; r < RB; ++r) {
                if (kb + tk >= lim[r]) continue;  // uniform: masked for this row (0 * inf would be NaN)
                const float pr = ps[r][tk];
                acc[r][0] += pr * v0;
                acc[r][1] += pr * v1;
            }
        }
        __syncthreads();
    }

#pragma unroll
    for (int r = 0; r < RB; ++r) {
        const float L = wave_sum(l[r]);
        if (r0 + r >= p.R) continue;
        // L == 0: no visible key; L NaN: a NaN key or a +inf score was visible
        const float inv = L > 0.f ? 1.f / L : (L == 0.f ? 0.f : L);
        const float lse2 = L > 0.f ? m[r] + log2f(L) : (L == 0.f ? -INFINITY : L);
        if (whole) {
            const int64_t off = row_offset(p, b, h, r0 + r);
#pragma unroll
            for (int dd = 0; dd < 2; ++dd) {
                const int d = lane + 64 * dd;
                if (d >= D) continue;
                const float o = acc[r][dd] * inv;
                if (p.out_dtype == SPIRE_BF16)
                    reinterpret_cast<uint16_t *>(p.out)[off + d] = f32_to_bf16_rne(o);
                else
                    reinterpret_cast<float *>(p.out)[off + d] = o;
            }
            if (lane == 0 && p.lse != nullptr)
                p.lse[lse_index(p, b, h, r0 + r)] = lse2 * 0.69314718055994531f;
        } else {
            float *o = pl.part_o + (slot * pl.rows + r) * (int64_t)D;
#pragma unroll
            for (int dd = 0; dd < 2; ++dd) {
                const int d = lane + 64 * dd;
                if (d < D) o[d] = acc[r][dd] * inv;
            }
            if (lane == 0) pl.part_lse[slot * pl.rows + r] = lse2;
        }
    }
}

__global__ __launch_bounds__(64) void generic_partial_kernel(Problem p, Plan pl) {
    __shared__ float qs[RB][kMaxD];
    __shared__ float ps[RB][KT];
    const int lane = threadIdx.x;
    const int wid = blockIdx.x;
    if (wid >= pl.workers) return;
    const int64_t T = (int64_t)pl.prefix[p.B] * pl.units;
    int64_t pos = worker_begin(wid, T, pl.workers);
    const int64_t end = worker_begin(wid + 1, T, pl.workers);
    if (pos >= end) return;
    const int64_t begin = pos;
    int seg = pl.wstart[2 * wid];
    int tile = pl.wstart[2 * wid + 1];
    const int nrb = pl.units / p.Hkv;

    while (pos < end) {
        const int b = seg / pl.units;
        const int u = seg - b * pl.units;
        const int h = u / nrb;
        const int r0 = (u - h * nrb) * RB;
        const int span = pl.prefix[b + 1] - pl.prefix[b];
        const int tiles_b = span - pl.seg_cost;
        const int64_t left = end - pos;
        const int te = left < (int64_t)(span - tile) ? tile + (int)left : span;
        if (tile >= tiles_b) {  // phantom positions only
            pos += te - tile;
            ++seg;
            tile = 0;
            continue;
        }
        const int t1 = te < tiles_b ? te : tiles_b;
        const int n = pl.nkeys[b];
        int ns = 0, rs = 0;
        if (p.draft) {
            const int m = p.lens[b] < 0 ? 0 : p.lens[b];
            ns = m < p.S ? m : p.S;
            if (p.W > 0) {
                int first = m - p.S - p.W;
                first = first < 0 ? 0 : first;
                int o = p.ring_offset[b] % p.W;
                if (o < 0) o += p.W;
                rs = (n - ns == p.W) ? 0 : (o + first % p.W) % p.W;
            }
        }
        const bool whole = (tile == 0 && t1 == tiles_b);
        const int64_t slot = 2 * (int64_t)wid + (pos == begin ? 0 : 1);
        generic_unit(p, pl, b, h, r0, n, ns, rs, tile, t1, whole, slot, lane, qs, ps);
        pos += te - tile;
        ++seg;
        tile = 0;
    }
}

// ---- non-finite values among the keys only some rows see ------------------------
// Keys [n - k, n) of a verify segment are visible to the later draft rows only.
// In the matrix-core kernels the rows that mask such a key still multiply its
// value by a zero probability, and 0 * inf or 0 * NaN is NaN: a non-finite
// value there (e.g. fp8 0x7F written for a NaN) would reach rows that must not
// see it.  This pass, launched after the combine of a matrix-core verify call,
// checks those few value rows of every (sequence, KV head); a segment holding a
// non-finite one (rare) has all its rows recomputed here by the fp32 unit loop
// above, which only accumulates a value for the rows that see its key, and
// overwritten.  Its cost otherwise is reading k value rows per segment.
__device__ __forceinline__ bool word_nonfinite(uint32_t x, int dtype) {
    if (dtype == SPIRE_F32) return (x & 0x7F800000u) == 0x7F800000u;
    if (dtype == SPIRE_BF16) return (x & 0x7F80u) == 0x7F80u || (x & 0x7F800000u) == 0x7F800000u;
    // e4m3fn: NaN is S.1111.111 (no infinities)
    return (x & 0x7Fu) == 0x7Fu || ((x >> 8) & 0x7Fu) == 0x7Fu || ((x >> 16) & 0x7Fu) == 0x7Fu ||
           ((x >> 24) & 0x7Fu) == 0x7Fu;
}

__global__ __launch_bounds__(64) void tail_fix_kernel(Problem p, Plan pl) {
    __shared__ float qs[RB][kMaxD];
    __shared__ float ps[RB][KT];
    const int lane = threadIdx.x;
    const int b = blockIdx.x / p.Hkv, h = blockIdx.x - (blockIdx.x / p.Hkv) * p.Hkv;
    const int n = effective_keys(p, b);
    const int lo = n - p.k > 0 ? n - p.k : 0;
    if (lo >= n) return;
    // the value rows of keys [lo, n), as 4-byte words (row bytes are a multiple of 16)
    const int words = p.D * p.kv.elem / 4;
    bool bad = false;
    for (int idx = lane; idx < (n - lo) * words; idx += 64) {
        const int key = lo + idx / words, w = idx - (idx / words) * words;
        const RowRef vr = key_row(p, b, h, key, 0, 0);
        bad |= word_nonfinite(reinterpret_cast<const uint32_t *>(vr.v)[w], p.kv_dtype);
    }
    if (!__any(bad)) return;
    const int tiles = (n + KT - 1) / KT;
    for (int r0 = 0; r0 < p.R; r0 += RB) generic_unit(p, pl, b, h, r0, n, 0, 0, 0, tiles, true, 0, lane, qs, ps);
}

hipError_t launch_tail_fix(const Problem &p, const Plan &pl, hipStream_t st) {
    if (p.draft || p.k == 0 || (int64_t)p.B * p.Hkv == 0) return hipSuccess;
    hipLaunchKernelGGL(tail_fix_kernel, dim3((unsigned)(p.B * p.Hkv)), dim3(64), 0, st, p, pl);
    return hipGetLastError();
}

hipError_t launch_generic_partial(const Problem &p, const Plan &pl, hipStream_t st) {
    hipLaunchKernelGGL(generic_partial_kernel, dim3(pl.workers), dim3(64), 0, st, p, pl);
    return hipGetLastError();
}

}  // namespace spire
