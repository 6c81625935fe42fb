// attn_mfma.hip -- split-KV partial attention on CDNA4 matrix cores (gfx950).
//
// One wave is one worker of the stream-K partition (spire_internal.h).  For a
// segment (sequence b, KV head h) it packs all R = (k+1) * g query rows that
// read this KV head -- the k+1 verify tokens (paper Sec. 2) times the g query
// heads of the group -- into 16-row blocks, so that every K/V tile is fetched
// from HBM once and feeds all of them.  Per 32-key tile:
//
//   S^T (keys x rows)  = K Q^T      v_mfma_f32_16x16x32_bf16, A = K, B = Q^T
//   online softmax in base 2 on S^T (row max across the 4 lane groups)
//   O^T (dims x rows) += V^T P^T    v_mfma_f32_16x16x32_bf16, A = V^T, B = P^T
//
// Register layouts (lane l, n16 = l & 15, j = l >> 4):
//   * MFMA A/B operands: lane l holds row/column n16 and the 8 consecutive
//     reduction indices 8j..8j+7; C: lane l holds rows 4j..4j+3, column n16.
//   * S^T row m of key group mb is key 16mb + 4(m&3) + (m>>2), so the C output
//     of lane l is keys 16mb + 4i + j (i = 0..3) for row 16nb + n16.
//   * The PV reduction index 8j+t is key 4t + j: exactly the S^T values lane l
//     already holds (t < 4 from mb = 0, t >= 4 from mb = 1), so P never
//     leaves its lane, and each V load instruction (t fixed) covers 4 whole,
//     consecutive key rows.
//   * PV row m of dim block mb' is head dim 8m + mb', so lane l loads the 8
//     contiguous dims d = 8 n16 .. 8 n16 + 7 of each of its keys, transposes
//     8 keys x 8 dims in registers (byte permutes), and ends up owning the 32
//     contiguous output dims 32j .. 32j + 31 of its row.
//   * K: each load instruction covers 64 contiguous bytes of 16 key rows.
// fp8 (OCP e4m3fn) K/V are converted in registers (exact): K to bf16 for the
// QK product with the bf16 queries, V to fp16 for the PV product, whose P
// operand then rounds to fp16 (bf16 K/V keep bf16 P); the per-head K scale
// is folded into the softmax scale, the V scale into the final normalisation.
//
// This kernel serves up to 32 rows (NB <= 2): the query fragments stay in
// registers and three tiles are kept in registers (two in flight).  More rows
// go to the LDS-staged kernel (attn_staged.hip), which splits them over waves.
#include "mfma_common.h"

namespace spire {

// Tiles [first, last] of one segment through three register buffers, two
// tiles in flight; only tiles of the range are loaded (a buffer is computed
// only after its load).  The stream-K kernel below keeps the same loop
// written out: as a call it compiled to a slightly different schedule.
template <bool FP8, int NB, int MODE>
__device__ __forceinline__ void stream_tiles(const SegAddr &a, const QFrag<NB, false> &qf,
                                             SoftmaxState<NB, false> &st, int first, int last, int n,
                                             int full_lim, float sc, int lane) {
    TileRegs<FP8> A, Bt, C;
    load_tile<FP8, MODE>(A, a, first, lane);
    if (first + 1 <= last) load_tile<FP8, MODE>(Bt, a, first + 1, lane);
    int tt = first;
    while (true) {
        if (tt + 2 <= last) load_tile<FP8, MODE>(C, a, tt + 2, lane);
        compute_tile<FP8, NB>(A, qf, st, tt, n, full_lim, sc, lane);
        if (++tt > last) break;
        if (tt + 2 <= last) load_tile<FP8, MODE>(A, a, tt + 2, lane);
        compute_tile<FP8, NB>(Bt, qf, st, tt, n, full_lim, sc, lane);
        if (++tt > last) break;
        if (tt + 2 <= last) load_tile<FP8, MODE>(Bt, a, tt + 2, lane);
        compute_tile<FP8, NB>(C, qf, st, tt, n, full_lim, sc, lane);
        if (++tt > last) break;
    }
}

template <bool FP8, int NB, int MODE>
__global__ __launch_bounds__(256, 1) void mfma_partial_kernel(Problem p, Plan pl) {
    static_assert(NB >= 1 && NB <= 2, "more than 32 rows go to the LDS-staged kernel");
    __shared__ int32_t s_pre[kPlanMaxB + 1];
    __shared__ int32_t s_sum[64 * kMfmaWavesPerWG];
    // the partition: no separate plan launch (its few microseconds per call
    // were a tenth of a short draft step)
    plan_in_kernel<64 * kMfmaWavesPerWG>(p, pl, s_pre, s_sum);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wid = __builtin_amdgcn_readfirstlane(blockIdx.x * kMfmaWavesPerWG + wave);
    if (wid >= pl.workers) return;
    const int64_t T = (int64_t)s_pre[p.B] * pl.units;
    int64_t pos = worker_begin(wid, T, pl.workers);
    const int64_t end = worker_begin(wid + 1, T, pl.workers);
    if (pos >= end) {
        if (lane == 0) pl.wstart[2 * wid] = -1;
        return;
    }
    int seg, tile;
    locate(s_pre, p.B, pl.units, pos, seg, tile);
    if (lane == 0) {  // recorded like the plan kernel's output
        pl.wstart[2 * wid] = seg;
        pl.wstart[2 * wid + 1] = tile;
    }
    const int64_t begin = pos;

    QFrag<NB, false> qf;

    while (pos < end) {
        const int b = seg / pl.units;
        const int h = seg - b * pl.units;
        const int span = s_pre[b + 1] - s_pre[b];
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
        const int n = effective_keys(p, b);

        const SegAddr a = make_seg_addr<MODE>(p, b, h, n);
        SoftmaxState<NB, false> st;
        begin_rows<FP8, NB, false, false>(p, b, h, n, 0, qf, st, lane);
        const int full_lim = p.draft ? n : n - p.k;
        float sc = p.sm_scale_log2;
        if (FP8) sc *= uload(p.kv.k_scale, h);

        // ---- tiles [tile, t1) ------------------------------------------------------
        if (n > 0) {
            const int last = t1 - 1;
            TileRegs<FP8> A, Bt, C;  // three register buffers, two tiles in flight
            // only tiles of the range are loaded (a buffer is computed only
            // after its load)
            load_tile<FP8, MODE>(A, a, tile, lane);
            if (tile + 1 <= last) load_tile<FP8, MODE>(Bt, a, tile + 1, lane);
            int tt = tile;
            while (true) {
                if (tt + 2 <= last) load_tile<FP8, MODE>(C, a, tt + 2, lane);
                compute_tile<FP8, NB>(A, qf, st, tt, n, full_lim, sc, lane);
                if (++tt > last) break;
                if (tt + 2 <= last) load_tile<FP8, MODE>(A, a, tt + 2, lane);
                compute_tile<FP8, NB>(Bt, qf, st, tt, n, full_lim, sc, lane);
                if (++tt > last) break;
                if (tt + 2 <= last) load_tile<FP8, MODE>(Bt, a, tt + 2, lane);
                compute_tile<FP8, NB>(C, qf, st, tt, n, full_lim, sc, lane);
                if (++tt > last) break;
            }
        }

        const bool whole = (tile == 0 && t1 == tiles_b);
        end_rows<FP8, NB, false>(p, pl, st, b, h, 0, whole, 2 * (int64_t)wid + (pos == begin ? 0 : 1), lane);
        pos += te - tile;
        ++seg;
        tile = 0;
    }
}

// Whole draft segments per workgroup.  A draft segment never holds more than
// S + W keys (paper Sec. 3.1: the constant-size sink + window cache), so when
// the segments number half or a quarter of the device's waves, G = 2 or 4
// waves of one workgroup per segment balance the work as the stream-K
// partition does, without its seams: the waves split the segment's tiles
// evenly (the short sink tile, last in the draft key space, goes to the last
// wave), merge their rows through LDS and write the final rows -- no
// partition, no partial slots, no combine launch.  Rows are merged on the
// base-2 reference maxima: O = sum_w 2^(m_w - M) O_w, l = sum_w 2^(m_w - M) l_w
// with M the largest reference; a wave that saw no finite score holds none
// and weighs zero (its zero or NaN state still propagates).
template <bool FP8, int NB, int G>
__global__ __launch_bounds__(256, 1) void mfma_draft_coop_kernel(Problem p) {
    static_assert(G >= 2 && kMfmaWavesPerWG % G == 0, "waves per segment");
    constexpr int SPW = kMfmaWavesPerWG / G;  // segments per workgroup
    __shared__ f32x4 s_acc[SPW][G - 1][8 * NB][64];
    __shared__ float s_l[SPW][G - 1][NB][64];
    __shared__ float s_m[SPW][G - 1][NB][64];  // reference maximum; -inf: none
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int slot = wave / G, part = wave - (wave / G) * G;
    const int seg = __builtin_amdgcn_readfirstlane((int)blockIdx.x * SPW + slot);
    const bool valid = seg < p.B * p.Hkv;
    const int b = valid ? seg / p.Hkv : 0;
    const int h = valid ? seg - b * p.Hkv : 0;
    SoftmaxState<NB, false> st;
    if (valid) {
        const int n = effective_keys(p, b);
        const int T = (n + kMfmaTile - 1) / kMfmaTile;
        const int t0 = part * T / G, t1 = (part + 1) * T / G;
        const SegAddr a = make_seg_addr<MODE_DRAFT>(p, b, h, n);
        QFrag<NB, false> qf;
        begin_rows<FP8, NB, false, false>(p, b, h, n, 0, qf, st, lane);
        float sc = p.sm_scale_log2;
        if (FP8) sc *= uload(p.kv.k_scale, h);
        if (t0 < t1) stream_tiles<FP8, NB, MODE_DRAFT>(a, qf, st, t0, t1 - 1, n, n, sc, lane);
    }
    if (valid && part > 0) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            float l = st.l[nb];
            l += __shfl_xor(l, 16);
            l += __shfl_xor(l, 32);
            s_l[slot][part - 1][nb][lane] = l;
            s_m[slot][part - 1][nb][lane] = st.thr[nb] == -INFINITY ? -INFINITY : st.msub[nb];
#pragma unroll
            for (int mb = 0; mb < 8; ++mb) s_acc[slot][part - 1][mb * NB + nb][lane] = st.acc[mb][nb];
        }
    }
    __syncthreads();
    if (!valid || part > 0) return;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        float l = st.l[nb];
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        const float m0 = st.thr[nb] == -INFINITY ? -INFINITY : st.msub[nb];
        float M = m0;
#pragma unroll
        for (int w = 0; w < G - 1; ++w) M = fmaxf(M, s_m[slot][w][nb][lane]);
        M = M == -INFINITY ? 0.f : M;
        const float a0 = m0 == -INFINITY ? 0.f : fast_exp2(m0 - M);
        l *= a0;
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) st.acc[mb][nb] *= a0;
#pragma unroll
        for (int w = 0; w < G - 1; ++w) {
            const float mw = s_m[slot][w][nb][lane];
            const float aw = mw == -INFINITY ? 0.f : fast_exp2(mw - M);
            l += s_l[slot][w][nb][lane] * aw;
#pragma unroll
            for (int mb = 0; mb < 8; ++mb) st.acc[mb][nb] += s_acc[slot][w][mb * NB + nb][lane] * aw;
        }
        st.msub[nb] = M;
        // end_rows sums the four lane groups' partial row sums: one holds it all
        st.l[nb] = (lane >> 4) == 0 ? l : 0.f;
    }
    end_rows<FP8, NB, false>(p, Plan{}, st, b, h, 0, true, 0, lane);
}

template <bool FP8, int NB>
static hipError_t launch_coop_nb(const Problem &p, int g, hipStream_t st) {
    const int segs = p.B * p.Hkv;
    const dim3 block(64 * kMfmaWavesPerWG);
    if (g == 4)
        hipLaunchKernelGGL((mfma_draft_coop_kernel<FP8, NB, 4>), dim3(segs), block, 0, st, p);
    else if (g == 2)
        hipLaunchKernelGGL((mfma_draft_coop_kernel<FP8, NB, 2>), dim3((segs + 1) / 2), block, 0, st, p);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_mfma_draft_coop(const Problem &p, int nb, int g, hipStream_t st) {
    const bool fp8 = p.kv_dtype == SPIRE_FP8_E4M3FN;
    if (!p.draft || p.B * p.Hkv <= 0) return hipErrorInvalidValue;
    if (nb == 1) return fp8 ? launch_coop_nb<true, 1>(p, g, st) : launch_coop_nb<false, 1>(p, g, st);
    if (nb == 2) return fp8 ? launch_coop_nb<true, 2>(p, g, st) : launch_coop_nb<false, 2>(p, g, st);
    return hipErrorInvalidValue;
}

template <bool FP8, int NB>
static hipError_t launch_nb(const Problem &p, const Plan &pl, hipStream_t st) {
    const dim3 grid((pl.workers + kMfmaWavesPerWG - 1) / kMfmaWavesPerWG), block(64 * kMfmaWavesPerWG);
    if (p.draft)
        hipLaunchKernelGGL((mfma_partial_kernel<FP8, NB, MODE_DRAFT>), grid, block, 0, st, p, pl);
    else if (p.kv.page_size > 0)
        hipLaunchKernelGGL((mfma_partial_kernel<FP8, NB, MODE_PAGED>), grid, block, 0, st, p, pl);
    else
        hipLaunchKernelGGL((mfma_partial_kernel<FP8, NB, MODE_CONTIG>), grid, block, 0, st, p, pl);
    return hipGetLastError();
}

template <bool FP8>
static hipError_t launch_fp(const Problem &p, const Plan &pl, int nb, hipStream_t st) {
    switch (nb) {
    case 1: return launch_nb<FP8, 1>(p, pl, st);
    case 2: return launch_nb<FP8, 2>(p, pl, st);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_mfma_partial(const Problem &p, const Plan &pl, int nb, hipStream_t st) {
    if (p.kv_dtype == SPIRE_FP8_E4M3FN) return launch_fp<true>(p, pl, nb, st);
    return launch_fp<false>(p, pl, nb, st);
}

}  // namespace spire
