// spire_internal.h -- shared declarations of the HIP library (not part of the ABI).
//
// Work partition used by every attention kernel ("stream-K" over keys):
//   * the keys of sequence b are cut into tiles of `tile` keys; a sequence
//     with no key still owns one (empty) tile so that its rows get written;
//   * a segment is one (sequence b, unit u) pair, where a unit is one KV head
//     (matrix-core kernels) or one KV head x 16-row block (generic kernel);
//     segment s = b * units + u owns tiles_b + seg_cost consecutive positions:
//     its tiles followed by seg_cost phantom positions that stand for the
//     fixed cost of a segment (queries, output rows, address set-up), so that
//     a worker covering many short segments gets correspondingly fewer tiles;
//     a worker reads no keys for phantom positions;
//   * the flattened positions [0, T), T = units * sum_b (tiles_b + seg_cost),
//     are split into `workers` contiguous ranges of equal length: worker w
//     owns [w*T/workers, (w+1)*T/workers);
//   * a worker that covers a whole segment writes the final rows; otherwise it
//     writes a partial (normalised output + base-2 log-sum-exp) into slot 2w
//     (the segment it starts in) or 2w+1 (the segment it ends in), and the
//     combine kernel merges the partials of each split segment.  (Merging
//     inside the attention kernel by the last worker to finish would need a
//     device-scope release/acquire per split segment, which on a multi-XCD
//     MI355X writes back / invalidates L2 and measured slower than a separate
//     combine launch.)
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/spire.h"

namespace spire {

constexpr int kMaxRows = 128;          // (k+1) * Hq/Hkv
constexpr int kGenericRowBlock = 16;   // rows per unit in the generic kernel
constexpr int kMaxWorkersPerCU = 8;
constexpr int kCombineMaxWorkers = 4096;  // workers one launch may have (the combine's LDS list)

// Device-side description of one K/V view (byte pointers, element strides).
struct KvDev {
    const uint8_t *k;
    const uint8_t *v;
    const int32_t *block_table;
    const float *k_scale;
    const float *v_scale;
    int64_t s_blk, s_head, s_tok;  // elements
    int32_t elem;                  // bytes per element
    int32_t page_size;             // 0 = contiguous
    int32_t max_blocks;
    int32_t num_blocks;
    int32_t capacity;              // contiguous: rows per sequence
};

// Everything an attention kernel needs to know about the request.
struct Problem {
    int32_t draft;          // 0: verify, 1: draft step
    int32_t B, Hq, Hkv, D;
    int32_t k;              // verify: draft tokens; draft: 0
    int32_t g;              // Hq / Hkv
    int32_t R;              // rows per KV head: (k+1) * g
    int32_t S, W;           // draft sinks / window
    float sm_scale_log2;    // sm_scale * log2(e)
    const uint8_t *q;
    int32_t q_dtype;        // SPIRE_F32 / SPIRE_BF16
    int32_t kv_dtype;
    const int32_t *lens;         // verify: kv_lens; draft: seq_lens
    const int32_t *ring_offset;  // draft only
    KvDev kv;               // verify cache, or the draft ring
    KvDev sink;             // draft sinks
    void *out;
    int32_t out_dtype;
    float *lse;
};

// Partition state in the workspace.
struct Plan {
    int32_t *nkeys;     // [B]   keys of each sequence after clamping
    int32_t *prefix;    // [B+1] exclusive prefix sum of tiles + seg_cost per sequence
    int32_t *wstart;    // [2*workers] (segment, tile) where each worker starts
    float *part_lse;    // [2*workers, rows]       base-2 log-sum-exp of a partial
    float *part_o;      // [2*workers, rows, D]    normalised partial output
    int32_t tile;       // keys per tile
    int32_t units;      // segments per sequence
    int32_t rows;       // rows per segment (partials stride)
    int32_t workers;
    int32_t seg_cost;   // phantom positions per segment (see above)
};

// Read-only, wave-uniform metadata (block tables, prefix sums, lengths,
// scales) is read through the constant address space so that it becomes a
// scalar load: those are counted separately from the vector loads of K/V, so
// waiting for a page id never forces waiting for K/V loads already in flight.
template <class T>
__device__ __forceinline__ T uload(const T *p, int64_t i) {
    typedef const T __attribute__((address_space(4))) cT;
    return ((const cT *)p)[i];
}

__device__ __forceinline__ int64_t worker_begin(int64_t w, int64_t T, int64_t workers) {
    return (w * T) / workers;
}
// the worker whose range contains flattened position x (0 <= x < T)
__device__ __forceinline__ int64_t worker_of(int64_t x, int64_t T, int64_t workers) {
    return ((x + 1) * workers - 1) / T;
}

constexpr int kPlanMaxB = 8192;  // sequences per call (the partition's LDS arrays)

// Keys of sequence b the kernels attend to: verify lengths clamped to what
// the cache descriptor can address, draft lengths to the sinks present plus
// the valid ring slots.
__device__ __forceinline__ int effective_keys(const Problem &p, int b) {
    int n = p.lens[b];
    if (!p.draft) {
        int64_t cap = p.kv.page_size > 0 ? (int64_t)p.kv.max_blocks * p.kv.page_size
                                         : (int64_t)p.kv.capacity;
        if (cap > INT32_MAX) cap = INT32_MAX;
        n = n < 0 ? 0 : (n > cap ? (int)cap : n);
    } else {
        const int m = n < 0 ? 0 : n;
        const int ns = m < p.S ? m : p.S;
        int nr = m - p.S;
        nr = nr < 0 ? 0 : (nr > p.W ? p.W : nr);
        n = ns + nr;
    }
    return n;
}

// Row r of KV head h (r in [0, R)) -> element offset of its query/output row
// in [B, k+1, Hq, D]: rows are ordered (draft index i, head in group hg).
__device__ __forceinline__ int64_t row_offset(const Problem &p, int b, int h, int r) {
    const int i = r / p.g, hg = r - (r / p.g) * p.g;
    return (((int64_t)b * (p.k + 1) + i) * p.Hq + (int64_t)h * p.g + hg) * p.D;
}
__device__ __forceinline__ int64_t lse_index(const Problem &p, int b, int h, int r) {
    const int i = r / p.g, hg = r - (r / p.g) * p.g;
    return ((int64_t)b * (p.k + 1) + i) * p.Hq + (int64_t)h * p.g + hg;
}

// Keys visible to row r of a sequence holding n keys: verify rows see
// [0, n - k + i); draft rows see everything the segment holds.
__device__ __forceinline__ int visible_limit(const Problem &p, int n, int r) {
    if (p.draft) return n;
    int i = r / p.g;
    if (i > p.k) i = p.k;
    return n - p.k + i;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t x) {
    return __uint_as_float((uint32_t)x << 16);
}
// round-to-nearest-even fp32 -> bf16 bits (NaN kept quiet)
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// ---- host-side launchers (one per kernel family) ---------------------------
hipError_t launch_plan(const Problem &p, const Plan &pl, hipStream_t st);
hipError_t launch_mfma_partial(const Problem &p, const Plan &pl, int nb, hipStream_t st);
// Draft steps with whole segments per workgroup (g = 2 or 4 waves per segment):
// final rows written directly, no plan and no combine.
hipError_t launch_mfma_draft_coop(const Problem &p, int nb, int g, hipStream_t st);
hipError_t launch_generic_partial(const Problem &p, const Plan &pl, hipStream_t st);
hipError_t launch_staged_partial(const Problem &p, const Plan &pl, int nb, hipStream_t st);
// LDS-staged kernel: waves per worker (a workgroup), waves per SIMD, and the
// workers of a launch (at most 4 per CU, like the register-staged kernel, so
// one workspace size serves both).  fp8 with 5 row blocks (72-80 rows): one
// wave holds every row block (accumulators in VGPRs, query fragments and
// spills in AGPRs), so each fp8 tile is converted once and no workgroup
// barrier orders the stage ring.
constexpr int staged_waves(bool fp8, int nb) { return nb <= 2 || (fp8 && nb == 5) ? 1 : 2; }
constexpr int staged_wps(bool fp8, int nb) { return fp8 && nb > 2 && nb < 5 ? 2 : 1; }
int staged_workers(int cus, int nb, bool fp8);
hipError_t launch_combine(const Problem &p, const Plan &pl, hipStream_t st);
// After a matrix-core verify call: recompute exactly the segments whose values
// at keys [n - k, n) are not all finite (attn_generic.hip).
hipError_t launch_tail_fix(const Problem &p, const Plan &pl, hipStream_t st);
hipError_t launch_hbm_read(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t st);

// ---- token verification (token_verify.hip) -----------------------------------
constexpr int kTokenPiece = 2048;    // vocabulary entries per weights wave
constexpr int kTokenMaxK = 32;
constexpr int kTokenMaxV = 1 << 20;  // keeps integer weight sums below 2^60

struct TokenProblem {
    const float *p;          // [B, k+1, V]
    const float *q;          // [B, k, V] (unused when k == 0)
    const int32_t *draft;    // [B, k]
    const float *u_accept;   // [B, k]
    const float *u_sample;   // [B]
    int32_t B, k, V;
    int32_t npieces;         // ceil(V / kTokenPiece)
    int32_t *n_accepted;     // [B]
    int32_t *out_tokens;     // [B, k+1]
    uint64_t *piece_sum;     // workspace [B, npieces]
    int32_t *nacc;           // workspace [B]: accepted counts (weights -> select)
};
hipError_t launch_token_weights(const TokenProblem &t, hipStream_t st);
hipError_t launch_token_select(const TokenProblem &t, hipStream_t st);
// block verification (block_verify.hip): the same problem, piece_sum holding
// [B, k+1, npieces] (every row's weights), nacc unused
hipError_t launch_block_weights(const TokenProblem &t, hipStream_t st);
hipError_t launch_block_select(const TokenProblem &t, hipStream_t st);

// ---- KV cache updates (kv_update.hip) ------------------------------------------
hipError_t launch_kv_append(const KvDev &kv, const void *k_new, const void *v_new, int new_dtype,
                            const int32_t *positions, int B, int T, int Hkv, int D, hipStream_t st);
hipError_t launch_draft_append(const KvDev &sink, const KvDev &ring, const void *k_new, const void *v_new,
                               int new_dtype, const int32_t *seq_lens, const int32_t *ring_offset, int B,
                               int Hkv, int D, int S, int W, void *spill_k, void *spill_v, hipStream_t st);
hipError_t launch_draft_rollback(const KvDev &sink, const KvDev &ring, const void *spill_k,
                                 const void *spill_v, const int32_t *base_lens, const int32_t *n_accepted,
                                 int steps, const int32_t *ring_offset, int B, int Hkv, int D, int S, int W,
                                 hipStream_t st);

// ---- feedback memory (feedback_memory.hip) ------------------------------------
constexpr int kFmMaxOut = 8;      // memory vectors (draft layers) per call
constexpr int kFmMaxLayers = 64;  // layers mixed (embedding included)
struct FeedbackArgs {
    const void *x;     // [Lp1, B*d]
    const float *w;    // [n_out, Lp1]
    void *m;           // [n_out, B*d]
    int32_t x_dtype, m_dtype;
    int32_t n_out, Lp1;
    int64_t Bd;
};
hipError_t launch_feedback_memory(const FeedbackArgs &a, hipStream_t st);

// MFMA kernel tile size (keys) and its worker count per CU.
constexpr int kMfmaTile = 32;
constexpr int kMfmaWavesPerWG = 4;
constexpr int kGenericTile = 64;

}  // namespace spire
