// plan_combine.hip -- work partition (plan) and split-segment merge (combine).
//
// The plan reads the per-sequence lengths on the device, clamps them to what
// the cache descriptors can address, cuts every sequence into key tiles (plus
// the phantom positions of each segment) and assigns each worker an equal
// share of all positions (see spire_internal.h).  It runs as one workgroup
// ahead of the LDS-staged and generic kernels; the register-staged kernel
// computes the same partition itself (plan_in_kernel, mfma_common.h).
// Everything it produces stays in the caller's workspace.
//
// The combine merges the partial results of a segment that several workers
// shared: with partials (o_p, lse_p) in base 2,
//   M = max_p lse_p,  w_p = 2^(lse_p - M),  out = sum_p w_p o_p / sum_p w_p,
//   lse = (M + log2 sum_p w_p) * ln 2,
// the log-sum-exp identity that makes attention over a union of disjoint key
// sets equal to a weighted merge of attention over each set.  A NaN partial
// (a NaN key or a +inf score in that part) makes the merged row NaN.
#include "spire_internal.h"

namespace spire {

constexpr int kPlanThreads = 1024;

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(Problem p, Plan pl) {
    __shared__ int32_t prefix[kPlanMaxB + 1];
    __shared__ int32_t sums[kPlanThreads];
    const int tid = threadIdx.x;
    const int B = p.B;
    const int per = (B + kPlanThreads - 1) / kPlanThreads;
    const int b0 = tid * per;
    const int b1 = b0 + per < B ? b0 + per : B;
    int local = 0;
    for (int b = b0; b < b1; ++b) {
        const int n = effective_keys(p, b);
        pl.nkeys[b] = n;
        const int tiles = (n > 0 ? (n + pl.tile - 1) / pl.tile : 1) + pl.seg_cost;
        prefix[b] = tiles;  // temporarily the position count
        local += tiles;
    }
    sums[tid] = local;
    __syncthreads();
    for (int off = 1; off < kPlanThreads; off <<= 1) {  // inclusive scan
        const int v = tid >= off ? sums[tid - off] : 0;
        __syncthreads();
        sums[tid] += v;
        __syncthreads();
    }
    int run = sums[tid] - local;
    for (int b = b0; b < b1; ++b) {
        const int tiles = prefix[b];
        prefix[b] = run;
        pl.prefix[b] = run;
        run += tiles;
    }
    if (tid == kPlanThreads - 1) {
        prefix[B] = sums[kPlanThreads - 1];
        pl.prefix[B] = sums[kPlanThreads - 1];
    }
    __syncthreads();
    const int64_t T = (int64_t)prefix[B] * pl.units;
    for (int w = tid; w < pl.workers; w += kPlanThreads) {
        const int64_t x = worker_begin(w, T, pl.workers);
        if (x >= worker_begin(w + 1, T, pl.workers)) {  // empty range
            pl.wstart[2 * w] = -1;
            pl.wstart[2 * w + 1] = 0;
            continue;
        }
        int lo = 0, hi = B - 1;  // last b with units * prefix[b] <= x
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int64_t)prefix[mid] * pl.units <= x) lo = mid; else hi = mid - 1;
        }
        const int tiles = prefix[lo + 1] - prefix[lo];
        const int64_t rel = x - (int64_t)prefix[lo] * pl.units;
        pl.wstart[2 * w] = lo * pl.units + (int)(rel / tiles);
        pl.wstart[2 * w + 1] = (int)(rel % tiles);
    }
}

hipError_t launch_plan(const Problem &p, const Plan &pl, hipStream_t st) {
    if (p.B > kPlanMaxB) return hipErrorInvalidValue;
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, st, p, pl);
    return hipGetLastError();
}

// Merge of the segments several workers shared.  The grid is either one
// workgroup per (segment, row chunk) -- workgroups of segments one worker
// covered return at once -- or, when segments outnumber workers, one per
// (worker w, row chunk): w merges the segment it starts inside of when it is
// the first worker to start inside that segment's tiles (every split segment
// has exactly one such worker), so no workgroup is spent on unsplit segments.
// The segment's rows are split into gridDim.y chunks, one thread per 4 output
// elements.  The partial slot of every worker covering the segment (or -1 for
// a worker with an empty range) is worked out once per workgroup into LDS, so
// the merge loops do no 64-bit divisions.
template <bool PER_WORKER>
__global__ __launch_bounds__(256) void combine_kernel(Problem p, Plan pl) {
    __shared__ int32_t s_slot[kCombineMaxWorkers];
    int seg = blockIdx.x, tile0 = 0;
    if (PER_WORKER) {
        seg = pl.wstart[2 * blockIdx.x];
        if (seg < 0) return;  // empty range
        tile0 = pl.wstart[2 * blockIdx.x + 1];
    }
    const int b = seg / pl.units, u = seg - (seg / pl.units) * pl.units;
    const int span = pl.prefix[b + 1] - pl.prefix[b];  // tiles + phantom positions
    const int tiles = span - pl.seg_cost;
    if (PER_WORKER && (tile0 == 0 || tile0 >= tiles)) return;  // starts at the first tile or past the last
    const int64_t T = (int64_t)pl.prefix[p.B] * pl.units;
    const int64_t start = (int64_t)pl.prefix[b] * pl.units + (int64_t)u * span;
    // the workers whose ranges hold the segment's tiles (phantoms are not read)
    const int64_t wlo = worker_of(start, T, pl.workers);
    const int64_t whi = worker_of(start + tiles - 1, T, pl.workers);
    if (wlo == whi) return;
    // workers wlo+1 .. whi start inside the tiles; the first non-empty one merges
    if (PER_WORKER && worker_begin(blockIdx.x, T, pl.workers) != worker_begin(wlo + 1, T, pl.workers)) return;

    const int nw = (int)(whi - wlo + 1);  // <= workers <= kCombineMaxWorkers
    const int64_t begin_lo = worker_begin(wlo, T, pl.workers);
    for (int i = threadIdx.x; i < nw; i += blockDim.x) {
        const int64_t w = wlo + i;
        // workers with an empty range (more workers than tiles) wrote nothing
        const bool empty = worker_begin(w + 1, T, pl.workers) == worker_begin(w, T, pl.workers);
        s_slot[i] = empty ? -1 : (int)(2 * w + ((i == 0 && begin_lo < start) ? 1 : 0));
    }
    __syncthreads();

    // rows of this unit, and the element of this thread
    const int nrb = pl.units / p.Hkv;  // row blocks per KV head
    const int h = u / nrb;
    const int r0 = (u - h * nrb) * pl.rows;
    const int nrows = p.R - r0 < pl.rows ? p.R - r0 : pl.rows;
    const int d4n = p.D >> 2;
    const int rpc = (pl.rows + gridDim.y - 1) / gridDim.y;  // rows per chunk
    const int rlo = blockIdx.y * rpc;
    const int rhi = rlo + rpc < nrows ? rlo + rpc : nrows;
    for (int idx = threadIdx.x; idx < (rhi - rlo) * d4n; idx += blockDim.x) {
        const int r = rlo + idx / d4n, d4 = idx - (idx / d4n) * d4n;
        // a NaN partial (a NaN key or a +inf score in that part) makes the row NaN
        float M = -INFINITY;
        bool nan = false;
        for (int i = 0; i < nw; ++i) {
            const int slot = s_slot[i];
            if (slot < 0) continue;
            const float lp = pl.part_lse[(int64_t)slot * pl.rows + r];
            if (lp != lp) nan = true;
            else M = fmaxf(M, lp);
        }
        float L = nan ? __builtin_nanf("") : 0.f;
        float4 acc = make_float4(L, L, L, L);
        if (!nan && M != -INFINITY) {
            for (int i = 0; i < nw; ++i) {
                const int slot = s_slot[i];
                if (slot < 0) continue;
                const float lp = pl.part_lse[(int64_t)slot * pl.rows + r];
                const float wgt = lp == -INFINITY ? 0.f : exp2f(lp - M);
                const float4 o = *reinterpret_cast<const float4 *>(
                    pl.part_o + ((int64_t)slot * pl.rows + r) * (int64_t)p.D + 4 * d4);
                L += wgt;
                acc.x += wgt * o.x; acc.y += wgt * o.y; acc.z += wgt * o.z; acc.w += wgt * o.w;
            }
        }
        const float inv = L > 0.f ? 1.f / L : (L == 0.f ? 0.f : L);
        const int64_t off = row_offset(p, b, h, r0 + r) + 4 * d4;
        if (p.out_dtype == SPIRE_BF16) {
            uint16_t *o = reinterpret_cast<uint16_t *>(p.out) + off;
            const uint32_t lo = f32_to_bf16_rne(acc.x * inv) | ((uint32_t)f32_to_bf16_rne(acc.y * inv) << 16);
            const uint32_t hi = f32_to_bf16_rne(acc.z * inv) | ((uint32_t)f32_to_bf16_rne(acc.w * inv) << 16);
            *reinterpret_cast<uint2 *>(o) = make_uint2(lo, hi);
        } else {
            *reinterpret_cast<float4 *>(reinterpret_cast<float *>(p.out) + off) =
                make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
        }
        if (d4 == 0 && p.lse != nullptr)
            p.lse[lse_index(p, b, h, r0 + r)] = L > 0.f ? (M + log2f(L)) * 0.69314718055994531f
                                                         : (L == 0.f ? -INFINITY : L);
    }
}

hipError_t launch_combine(const Problem &p, const Plan &pl, hipStream_t st) {
    if ((int64_t)p.B * pl.units == 0) return hipSuccess;
    if (pl.workers > kCombineMaxWorkers) return hipErrorInvalidValue;
    const int64_t segs = (int64_t)p.B * pl.units;
    const int rpw = 256 / (p.D / 4);  // rows per chunk: one thread per 4 outputs
    const int64_t want = (pl.rows + rpw - 1) / rpw;
    if (segs > pl.workers) {  // at most one split segment per worker start
        hipLaunchKernelGGL(combine_kernel<true>, dim3((unsigned)pl.workers, (unsigned)want), dim3(256), 0, st, p,
                           pl);
    } else {
        // one workgroup per segment, its rows split while that keeps the grid
        // within ~4096 workgroups (more measured slower)
        const int64_t room = segs >= 4096 ? 1 : 4096 / segs;
        hipLaunchKernelGGL(combine_kernel<false>, dim3((unsigned)segs, (unsigned)(want < room ? want : room)),
                           dim3(256), 0, st, p, pl);
    }
    return hipGetLastError();
}

}  // namespace spire
