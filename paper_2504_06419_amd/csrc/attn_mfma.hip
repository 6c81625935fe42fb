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
// fp8 (OCP e4m3fn) K/V are converted to bf16 in registers (exact); the
// per-head K scale is folded into the softmax scale, the V scale into the
// final normalisation.
//
// This kernel serves up to 32 rows (NB <= 2): the query fragments stay in
// registers and three tiles are kept in registers (two in flight).  More rows
// go to the LDS-staged kernel (attn_staged.hip), which splits them over waves.
#include "mfma_common.h"

namespace spire {

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
