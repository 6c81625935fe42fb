// attn_staged.hip -- LDS-staged matrix-core partial attention (gfx950).
//
// Same tile math as attn_mfma.hip (mfma_common.h), but K/V tiles travel
// HBM -> LDS with the gfx950 global->LDS DMA loads (global_load_lds_dwordx4),
// which cost no registers while in flight.  That buys two things:
//   * deep pipelines: a ring of NS tile stages per worker keeps NS-1 tiles in
//     flight (fp8 tiles are only 8 KB, so register staging cannot hold
//     enough bytes in flight to cover HBM latency);
//   * room for many query rows: a bf16 worker, or an fp8 one with 3-4 or 6-8
//     row blocks (up to 128 rows, e.g. k = 15 with 8 query heads per KV
//     head), is P = 2 waves of one workgroup that share the stage ring and
//     split the 16-row blocks between them, each keeping its accumulators in
//     registers without spilling.  An fp8 worker with 5 blocks (the 72 rows of
//     k = 8 with 8 query heads per KV head) is one wave with every block: it
//     converts each tile once (two waves would both convert it) and needs no
//     workgroup barrier; measured 3 % faster than 3 + 2 blocks on two waves.
//
// Stage layout (one 32-key tile): the K part is row-major with each row's
// 16-byte chunks permuted (kswz: whole rows per copy instruction, reads free
// of bank conflicts); the V part is row-major (bf16: DMA lane
// L of instruction t = the 16 bytes of key 4t + L/16 lane L needs; fp8: 8 whole
// 128-byte rows per instruction, each row's 16-byte chunks rotated by its key
// group, read back transposed as the V^T operands: no byte permutes, measured
// 1.4-2.1 % faster on the 72-row verify than 8 bytes per key per lane).  With
// P = 2, wave 1 (the one with fewer row blocks) copies whole tiles; a
// workgroup barrier per tile publishes them.  The compiler does not track the DMA -> LDS
// dependency, so the kernel waits on vmcnt explicitly before the barrier.
#include "mfma_common.h"

namespace spire {


template <bool FP8> struct Stage {
    static constexpr int KLOADS = FP8 ? 4 : 8;      // 1 KB DMA instructions for K
    static constexpr int VLOADS = FP8 ? 4 : 8;      // ... and for V
    static constexpr int KBYTES = KLOADS * 1024;
    static constexpr int BYTES = (KLOADS + VLOADS) * 1024;
};

constexpr int kStagedLdsPerCU = 160 * 1024;


// Workgroup barrier of the stage ring.  __syncthreads() carries a release
// fence, for which the compiler waits on every outstanding global->LDS copy
// (vmcnt(0)), draining the whole ring once per tile.  The copies a ring
// barrier publishes were already waited for (wait_vmcnt); what must also be
// complete are the LDS reads of the stage about to be overwritten.  The
// memory clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void ring_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// One 16-byte DMA from a uniform base plus a 32-bit lane offset.  The empty
// asm keeps the offset a 32-bit value at the load (otherwise the compiler
// hoists its widening out of the tile loop, keeps 64-bit offsets in spare
// registers and adds them with vector instructions), so the load takes the
// form with a scalar base and a 32-bit vector offset.
__device__ __forceinline__ void dma16_off(const uint8_t *base, uint32_t off, lds_u8 *l) {
    asm volatile("" : "+v"(off));
    dma16(base + off, l);
}

// K stage layout: row-major, key row r of the tile at r * RB bytes (RB = 128
// fp8, 256 bf16), its 16-byte chunk q at position q ^ kswz(r): each copy
// instruction moves whole rows (8 fp8 / 4 bf16 rows of 1 KB, every 128-byte
// line in one request), and the MFMA-operand reads -- 16 lanes, one per row,
// the same chunk -- still land on distinct banks, with 128 or with 256 bytes
// of banks per cycle.
template <bool FP8> __device__ __forceinline__ int kswz(int r) {
    r &= 15;
    if constexpr (FP8) return ((r >> 2) & 3) | (((r ^ (r >> 1)) & 1) << 2);
    return 4 * (r & 3) + (r >> 2);
}

// Copy the K (PART & 1) and/or V (PART & 2) half of tile `tile` into `st`.
template <bool FP8, int MODE, int PART>
__device__ __forceinline__ void issue_tile(lds_u8 *st, const SegAddr &a, int tile, int lane) {
    using G = Stage<FP8>;
    const int n16 = lane & 15, j = lane >> 4;
    const int key0 = tile * kMfmaTile;
    const int64_t g0 = group_base<MODE>(a, key0);
    const int64_t g1 = group_base<MODE>(a, key0 + 16);
    const bool fast = MODE == MODE_PAGED || (g0 >= 0 && g1 >= 0);
    if (PART & 1) {
        constexpr int CPR = FP8 ? 8 : 16;   // 16-byte chunks per key row
        constexpr int RPI = 64 / CPR;       // rows per copy instruction
#pragma unroll
        for (int x = 0; x < G::KLOADS; ++x) {
            const int r = RPI * x + lane / CPR;
            const int q = (lane % CPR) ^ kswz<FP8>(r);
            if (fast) {  // uniform group base + 32-bit lane offset (the host bounds 16 rows below 2^31 bytes)
                dma16_off(a.kseq + (x < G::KLOADS / 2 ? g0 : g1),
                          (uint32_t)(r & 15) * (uint32_t)a.tok_bytes + (uint32_t)(16 * q), st + x * 1024);
                continue;
            }
            const uint8_t *row;
            if (MODE == MODE_DRAFT) {
                row = draft_row(a, key0 + r, false);
            } else {
                row = a.kseq + (int64_t)min(key0 + r, a.cap - 1) * a.tok_bytes;
            }
            dma16(row + 16 * q, st + x * 1024);
        }
    }
    if (PART & 2) {
#pragma unroll
        for (int x = 0; x < G::VLOADS; ++x) {
            // bf16: key 4x + j, bytes 16 n16;  fp8: key 8x + lane/8, its 16-byte chunk
            // c lands at position (c + kin/4) % 8 of the row (rotation per key
            // group: the transposing reads of 16 lanes then hit distinct banks)
            const int kin = FP8 ? 8 * x + (lane >> 3) : 4 * x + j;
            const int byte = FP8 ? 16 * (((lane & 7) - (kin >> 2)) & 7) : 16 * n16;
            if (fast) {
                dma16_off(a.vseq + (kin < 16 ? g0 : g1), (uint32_t)(kin & 15) * (uint32_t)a.tok_bytes + (uint32_t)byte,
                          st + G::KBYTES + x * 1024);
                continue;
            }
            const uint8_t *row;
            if (MODE == MODE_DRAFT) {
                row = draft_row(a, key0 + kin, true);
            } else {
                row = a.vseq + (int64_t)min(key0 + kin, a.cap - 1) * a.tok_bytes;
            }
            dma16(row + byte, st + G::KBYTES + x * 1024);
        }
    }
}

template <bool FP8>
__device__ __forceinline__ void read_tile(TileRegs<FP8> &T, const lds_u8 *st, int lane) {
    using G = Stage<FP8>;
    const int n16 = lane & 15, j = lane >> 4;
    // MFMA operand (mb, c) of this lane: key row 16 mb + rho, chunk 4 c + j
    constexpr int NK = FP8 ? 2 : 4;
    constexpr int RB = FP8 ? 128 : 256;
    const int rho = 4 * (n16 & 3) + (n16 >> 2);
    const int sw = kswz<FP8>(rho);
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int c = 0; c < NK; ++c)
            T.k[mb][c] = *reinterpret_cast<const __attribute__((address_space(3))) u32x4 *>(
                st + (16 * mb + rho) * RB + 16 * ((4 * c + j) ^ sw));
    if constexpr (FP8) {
        // Transposing reads (ds_read_b64_tr_b8): byte t of lane i of a 16-lane
        // group is byte i % 8 of the 8 bytes lane 2t + i/8 of the group
        // addresses.  Lane s of group j addresses key 4(s/2) + j, dims
        // 16 mb + 8 (s % 2) .. +7, so lane i receives dim 16 mb + i of keys
        // 4t + j, t = 0..7: the V^T operand of dim block mb.
        // Issued as inline assembly: the builtin makes the compiler wait for
        // every outstanding global->LDS copy (vmcnt(0)) before it, draining
        // the stage ring each tile.  The closing wait ties the results, so no
        // use can move above it.
        const int key = 4 * (n16 >> 1) + j, half = n16 & 1;
        const uint32_t row = (uint32_t)(uintptr_t)(st + key * 128 + 8 * half);
        const int rot = key >> 2;
        uint64_t r[8];
#pragma unroll
        for (int mb = 0; mb < 8; ++mb)
            asm volatile("ds_read_b64_tr_b8 %0, %1 offset:%2"
                         : "=v"(r[mb])
                         : "v"(row + 16 * ((mb + rot) & 7)), "i"(G::KBYTES));
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]),
                       "+v"(r[6]), "+v"(r[7]));
#pragma unroll
        for (int mb = 0; mb < 8; ++mb) T.v[mb] = u32x2{(uint32_t)r[mb], (uint32_t)(r[mb] >> 32)};
    } else {
#pragma unroll
        for (int t = 0; t < 8; ++t)
            T.v[t] = *reinterpret_cast<const __attribute__((address_space(3))) u32x4 *>(
                st + G::KBYTES + t * 1024 + lane * 16);
    }
}

// One wave's share of a segment: row blocks rb0 .. rb0+NBW-1 over tiles
// [t0, t1), stage ring shared by the P waves of the workgroup.  COPY says
// which halves of every tile this wave copies into the ring (1 K, 2 V, 3 both,
// 0 none).
template <bool FP8, int NBW, int MODE, int P, int NS, bool QL, int COPY>
__device__ __forceinline__ void run_segment(const Problem &p, const Plan &pl, lds_u8 *ring,
                                            u32x4 *qlds, const SegAddr &a, int b, int h, int n,
                                            int t0, int t1, int rb0, bool whole, int64_t slot,
                                            int lane) {
    using G = Stage<FP8>;
    constexpr int MINE = ((COPY & 1) ? G::KLOADS : 0) + ((COPY & 2) ? G::VLOADS : 0);
    QFrag<NBW, QL> qf;
    if constexpr (QL) qf.lds = qlds;
    SoftmaxState<NBW, true> st;
    begin_rows<FP8, NBW, QL, true>(p, b, h, n, rb0, qf, st, lane);
    const int full_lim = p.draft ? n : n - p.k;
    float sc = p.sm_scale_log2;
    if (FP8) sc *= uload(p.kv.k_scale, h);

    if (n > 0) {
        const int last = t1 - 1;
        auto issue = [&](int stage, int tile) {
            if constexpr (COPY != 0) issue_tile<FP8, MODE, COPY>(ring + stage * G::BYTES, a, tile, lane);
        };
#pragma unroll
        for (int s = 0; s < NS - 1; ++s) issue(s, t0 + s < last ? t0 + s : last);
        int rd = 0, wr = NS - 1;
        for (int tt = t0; tt <= last; ++tt) {
            wait_vmcnt<(NS - 2) * MINE>();  // this wave's copies of tile tt have landed
            ring_barrier();                  // ... and the other waves' parts; tile tt-1 fully read
            issue(wr, tt + NS - 1 < last ? tt + NS - 1 : last);
            wr = wr + 1 == NS ? 0 : wr + 1;
            TileRegs<FP8> T;
            read_tile<FP8>(T, ring + rd * G::BYTES, lane);
            rd = rd + 1 == NS ? 0 : rd + 1;
            compute_tile<FP8, NBW, QL, true, FP8>(T, qf, st, tt, n, full_lim, sc, lane);
        }
        wait_vmcnt<0>();  // no copy may still be landing when the next segment reuses the ring
    }
    end_rows<FP8, NBW, true, FP8>(p, pl, st, b, h, rb0, whole, slot, lane);
}

// WPS waves per SIMD: with two, one wave's scalar, LDS and matrix-core
// instructions issue beside the other's vector instructions (a lone wave
// issues one instruction at a time), at half the registers and LDS each.
template <bool FP8, int NB, int MODE, int P, int WPS>
__global__ __launch_bounds__(64 * P, WPS) void staged_partial_kernel(Problem p, Plan pl) {
    using G = Stage<FP8>;
    constexpr int NB0 = P == 1 ? NB : (NB + 1) / 2;
    constexpr int NB1 = P == 1 ? 1 : NB / 2;
    // Query fragments in LDS free registers for the accumulators.  fp8 stages
    // are half the size of bf16 ones, so that costs few stages: at one wave
    // per SIMD both waves park them; at two, only a wave with three blocks.
    // A single wave with five blocks keeps them in registers (20 KB of LDS
    // would leave only two stages).
    constexpr bool QL0 = FP8 && (P == 1 ? NB0 <= 2 : (WPS == 1 || NB0 > 2));
    constexpr bool QL1 = FP8 && WPS == 1 && P == 2;
    constexpr int QBYTES = ((QL0 ? NB0 : 0) + (QL1 ? NB1 : 0)) * 4 * 64 * 16;
    constexpr int LDS = kStagedLdsPerCU * P / (4 * WPS);  // 4 * WPS / P workgroups per CU
    constexpr int NS = (LDS - QBYTES) / G::BYTES;
    static_assert(NS >= 3, "stage ring too small");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[NS * G::BYTES + QBYTES];
    lds_u8 *ring = (lds_u8 *)smem;
    u32x4 *qsmem = reinterpret_cast<u32x4 *>(smem + NS * G::BYTES);

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wid = blockIdx.x;
    if (wid >= pl.workers) return;
    const int64_t T = (int64_t)uload(pl.prefix, p.B) * pl.units;
    int64_t pos = worker_begin(wid, T, pl.workers);
    const int64_t end = worker_begin(wid + 1, T, pl.workers);
    if (pos >= end) return;
    int seg = uload(pl.wstart, 2 * wid);
    int tile = uload(pl.wstart, 2 * wid + 1);
    const int64_t begin = pos;

    while (pos < end) {
        const int b = seg / pl.units;
        const int h = seg - b * pl.units;
        const int span = uload(pl.prefix, b + 1) - uload(pl.prefix, b);
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
        const int n = uload(pl.nkeys, b);
        const SegAddr a = make_seg_addr<MODE>(p, b, h, n);
        const bool whole = (tile == 0 && t1 == tiles_b);
        const int64_t slot = 2 * (int64_t)wid + (pos == begin ? 0 : 1);
        __syncthreads();  // every wave is done with the ring of the previous segment
        // with two waves, the one with fewer row blocks (wave 1) copies whole
        // tiles, which evens out the work the two waves do between barriers
        if (P == 1)
            run_segment<FP8, NB0, MODE, P, NS, QL0, 3>(p, pl, ring, qsmem, a, b, h, n, tile, t1, 0,
                                                       whole, slot, lane);
        else if (wave == 0)
            run_segment<FP8, NB0, MODE, P, NS, QL0, 0>(p, pl, ring, qsmem, a, b, h, n, tile, t1, 0,
                                                       whole, slot, lane);
        else
            run_segment<FP8, NB1, MODE, P, NS, QL1, 3>(p, pl, ring, qsmem + (QL0 ? NB0 : 0) * 4 * 64, a,
                                                       b, h, n, tile, t1, NB0, whole, slot, lane);
        pos += te - tile;
        ++seg;
        tile = 0;
    }
}

template <bool FP8, int NB, int P>
static hipError_t launch_staged_nb(const Problem &p, const Plan &pl, hipStream_t st) {
    constexpr int WPS = staged_wps(FP8, NB);
    const dim3 grid(pl.workers), block(64 * P);
    if (p.draft)
        hipLaunchKernelGGL((staged_partial_kernel<FP8, NB, MODE_DRAFT, P, WPS>), grid, block, 0, st, p, pl);
    else if (p.kv.page_size > 0)
        hipLaunchKernelGGL((staged_partial_kernel<FP8, NB, MODE_PAGED, P, WPS>), grid, block, 0, st, p, pl);
    else
        hipLaunchKernelGGL((staged_partial_kernel<FP8, NB, MODE_CONTIG, P, WPS>), grid, block, 0, st, p, pl);
    return hipGetLastError();
}

template <bool FP8>
static hipError_t launch_staged_fp(const Problem &p, const Plan &pl, int nb, hipStream_t st) {
    if constexpr (!FP8) {
        // a single bf16 worker would get only 2 stages of 16 KB: the register-
        // staged kernel serves up to 32 rows instead
        if (nb <= 2) return hipErrorInvalidValue;
    }
    switch (nb) {
    case 1: if constexpr (FP8) return launch_staged_nb<FP8, 1, 1>(p, pl, st); else return hipErrorInvalidValue;
    case 2: if constexpr (FP8) return launch_staged_nb<FP8, 2, 1>(p, pl, st); else return hipErrorInvalidValue;
    case 3: return launch_staged_nb<FP8, 3, staged_waves(FP8, 3)>(p, pl, st);
    case 4: return launch_staged_nb<FP8, 4, staged_waves(FP8, 4)>(p, pl, st);
    case 5: return launch_staged_nb<FP8, 5, staged_waves(FP8, 5)>(p, pl, st);
    case 6: return launch_staged_nb<FP8, 6, staged_waves(FP8, 6)>(p, pl, st);
    case 7: return launch_staged_nb<FP8, 7, staged_waves(FP8, 7)>(p, pl, st);
    case 8: return launch_staged_nb<FP8, 8, staged_waves(FP8, 8)>(p, pl, st);
    default: return hipErrorInvalidValue;
    }
}

int staged_workers(int cus, int nb, bool fp8) {
    return cus * 4 * staged_wps(fp8, nb) / staged_waves(fp8, nb);
}

hipError_t launch_staged_partial(const Problem &p, const Plan &pl, int nb, hipStream_t st) {
    if (p.kv_dtype == SPIRE_FP8_E4M3FN) return launch_staged_fp<true>(p, pl, nb, st);
    return launch_staged_fp<false>(p, pl, nb, st);
}

}  // namespace spire
