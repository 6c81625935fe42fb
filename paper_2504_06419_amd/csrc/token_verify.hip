// token_verify.hip -- token verification of a speculation round (gfx950).
//
// After the target's parallel verify pass, each sequence accepts its draft
// tokens x_1..x_k while r_i < p_i(x_i) / q_i(x_i), stops at the first
// rejection, and emits one more token: a correction drawn from
// norm(max(0, p_{n+1} - q_{n+1})) after a rejection, or a bonus drawn from
// p_{k+1} when all k were accepted.  This is the modified rejection sampling
// that makes the accepted tokens follow the target's distribution (paper
// Sec. 1, Sec. 6; Table 1's caption: 1..k+1 tokens per round).
//
// Every decision is exact, so any order of evaluation gives the same tokens:
//   * accept test r * q < p in fp64 (the product of two fp32 numbers is exact);
//   * sampling is an inverse CDF over integer weights W = floor(w * 2^40),
//     w = clamp(p - q, 0, 1) in fp32 (correction) or clamp(p, 0, 1) (bonus),
//     threshold T = floor(U * Z / 2^24) with U = floor(u * 2^24) clamped to
//     [0, 2^24 - 1], token = the smallest x whose running weight exceeds T.
//
// Two launches, both bound by reading the probability rows:
//   weights kernel  every wave owns one 2048-entry piece of the one row its
//                   sequence samples from: it recomputes the accepted count
//                   (k gathers), streams the piece of p (and of q for a
//                   correction) with coalesced 16-byte loads and writes the
//                   piece's weight sum -- no workgroup synchronisation;
//   select kernel   one workgroup per sequence: prefix over the piece sums,
//                   the piece holding the threshold is read again (8 KB of p,
//                   8 KB of q) and searched in registers.  An empty
//                   correction row, which falls back to p, is scanned whole.
#include "sampling.h"

namespace spire {

// Accepted count of sequence b: lane i < k tests draft token i; the first
// rejection ends the prefix (lanes >= k count as rejections).
__device__ __forceinline__ int accepted_count(const TokenProblem &t, int b, int lane) {
    bool reject = true;
    if (lane < t.k) {
        const int x = t.draft[(int64_t)b * t.k + lane];
        if (x >= 0 && x < t.V) {
            const double pv = t.p[((int64_t)b * (t.k + 1) + lane) * t.V + x];
            const double qv = t.q[((int64_t)b * t.k + lane) * t.V + x];
            const double u = t.u_accept[(int64_t)b * t.k + lane];
            reject = !(u * qv < pv);
        }
    }
    const uint64_t m = __ballot(reject);
    return __builtin_ctzll(m);  // k <= 32 < 64: bit k is always set
}

// Weight of entry x of the sampled row: a correction row weighs p - q,
// otherwise p (`qrow` NULL).
__device__ __forceinline__ uint64_t entry_weight(const float *prow, const float *qrow, int x) {
    const float pv = prow[x];
    return fixed_weight(qrow ? pv - qrow[x] : pv);
}

template <bool VEC>
__global__ __launch_bounds__(kTvThreads) void token_weights_kernel(TokenProblem t) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int s = blockIdx.x * kTvWaves + wave;  // piece of the row
    const int b = blockIdx.y;
    if (s >= t.npieces) return;
    const int n = accepted_count(t, b, lane);
    const bool corr = n < t.k;
    const float *prow = t.p + ((int64_t)b * (t.k + 1) + n) * t.V;
    const float *qrow = corr ? t.q + ((int64_t)b * t.k + n) * t.V : nullptr;
    const int x0 = s * kTokenPiece;
    uint64_t sw = 0;
    if (VEC) {
        // coalesced 16-byte loads; V % 4 == 0, so a 4-entry group is wholly in or out
        const tv_f32x4 *p4 = reinterpret_cast<const tv_f32x4 *>(prow + x0);
        const tv_f32x4 *q4 = reinterpret_cast<const tv_f32x4 *>(corr ? qrow + x0 : prow + x0);
        const int groups = min(kTokenPiece, t.V - x0) >> 2;
        tv_f32x4 pv[kTvGroupsPerLane], qv[kTvGroupsPerLane];
        const tv_f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < kTvGroupsPerLane; ++i) {
            const int gi = lane + 64 * i;
            pv[i] = gi < groups ? __builtin_nontemporal_load(p4 + gi) : zero;
            qv[i] = (corr && gi < groups) ? __builtin_nontemporal_load(q4 + gi) : zero;
        }
#pragma unroll
        for (int i = 0; i < kTvGroupsPerLane; ++i) {
            const tv_f32x4 w = pv[i] - qv[i];  // q is zero for a bonus row
            sw += fixed_weight(w.x) + fixed_weight(w.y) + fixed_weight(w.z) + fixed_weight(w.w);
        }
    } else {
        const int cnt = min(kTokenPiece, t.V - x0);
        float pv[kTokenPiece / 64], qv[kTokenPiece / 64];
#pragma unroll
        for (int i = 0; i < kTokenPiece / 64; ++i) {
            const int xi = lane + 64 * i;
            pv[i] = xi < cnt ? prow[x0 + xi] : 0.f;
            qv[i] = (corr && xi < cnt) ? qrow[x0 + xi] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < kTokenPiece / 64; ++i) sw += fixed_weight(pv[i] - qv[i]);
    }
    sw = wave_sum(sw);
    if (lane == 0) {
        t.piece_sum[(int64_t)b * t.npieces + s] = sw;
        if (s == 0) t.nacc[b] = n;
    }
}

// Token in piece entries [x0, x0 + cnt) whose running weight first exceeds R
// (R below the piece's total).  Thread tid owns the contiguous slice of 8
// entries [x0 + 8 tid, ...): its loads are issued at once, its weights stay in
// registers, the block scans the slice sums and the one thread whose slice
// holds R finds the token among its registers.
template <bool VEC>
__device__ __forceinline__ void select_in_piece(const float *prow, const float *qrow, int x0, int cnt,
                                                uint64_t R, uint64_t *s_red, int *s_tok, int lane,
                                                int wave) {
    const int base = kTvSlice * (int)threadIdx.x;
    float pv[kTvSlice], qv[kTvSlice];
    if (VEC) {
        // 16-byte loads; cnt % 4 == 0, so a 4-entry group is wholly in or out
        const tv_f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < kTvSlice / 4; ++i) {
            const bool in = base + 4 * i < cnt;
            const tv_f32x4 a = in ? *reinterpret_cast<const tv_f32x4 *>(prow + x0 + base + 4 * i) : zero;
            const tv_f32x4 c = (in && qrow) ? *reinterpret_cast<const tv_f32x4 *>(qrow + x0 + base + 4 * i)
                                            : zero;
            pv[4 * i] = a.x; pv[4 * i + 1] = a.y; pv[4 * i + 2] = a.z; pv[4 * i + 3] = a.w;
            qv[4 * i] = c.x; qv[4 * i + 1] = c.y; qv[4 * i + 2] = c.z; qv[4 * i + 3] = c.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < kTvSlice; ++i) {
            const bool in = base + i < cnt;
            pv[i] = in ? prow[x0 + base + i] : 0.f;
            qv[i] = (in && qrow) ? qrow[x0 + base + i] : 0.f;
        }
    }
    uint64_t w[kTvSlice];
    uint64_t s = 0;
#pragma unroll
    for (int i = 0; i < kTvSlice; ++i) {
        w[i] = fixed_weight(pv[i] - qv[i]);  // q is zero for a bonus row; entries past cnt weigh 0
        s += w[i];
    }
    uint64_t total;
    const uint64_t ti = block_incl_scan(s, s_red, lane, wave, &total);
    const uint64_t te = ti - s;
    if (te <= R && R < ti) {  // exactly one thread
        uint64_t run = te;
        int found = -1;
#pragma unroll
        for (int i = 0; i < kTvSlice; ++i) {
            run += w[i];
            if (found < 0 && run > R) found = i;
        }
        *s_tok = x0 + base + found;
    }
}

// Token in entries [x0, x1) of a row whose running weight first exceeds R
// (R below the range's total), for ranges of any length (the whole-row
// fallback): every thread owns a contiguous slice, the block scans the slice
// sums, and the one thread whose slice holds R walks it again.
__device__ __forceinline__ void select_in_range(const float *prow, const float *qrow, int x0, int x1,
                                                uint64_t R, uint64_t *s_red, int *s_tok, int lane,
                                                int wave) {
    const int per = (x1 - x0 + kTvThreads - 1) / kTvThreads;
    const int a = min(x0 + per * (int)threadIdx.x, x1), e = min(a + per, x1);
    uint64_t s = 0;
    for (int x = a; x < e; ++x) s += entry_weight(prow, qrow, x);
    uint64_t total;
    const uint64_t ti = block_incl_scan(s, s_red, lane, wave, &total);
    const uint64_t te = ti - s;
    if (te <= R && R < ti) {  // exactly one thread
        uint64_t run = te;
        int x = a;
        for (; x < e; ++x) {
            run += entry_weight(prow, qrow, x);
            if (run > R) break;
        }
        *s_tok = x;
    }
}

template <bool VEC>
__global__ __launch_bounds__(kTvThreads) void token_select_kernel(TokenProblem t) {
    __shared__ uint64_t s_red[kTvWaves];
    __shared__ int s_piece, s_tok;
    __shared__ uint64_t s_rem;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    if (tid == 0) s_tok = -1;
    const int n = uload(t.nacc, b);  // recorded by the weights kernel (0 <= n <= k)
    const bool corr = n < t.k;
    const uint64_t *ps = t.piece_sum + (int64_t)b * t.npieces;
    const float *prow = t.p + ((int64_t)b * (t.k + 1) + n) * t.V;
    const float *qrow = corr ? t.q + ((int64_t)b * t.k + n) * t.V : nullptr;

    // total weight of the row (npieces <= 512: at most two sums per thread)
    uint64_t mine = 0;
    for (int i = tid; i < t.npieces; i += kTvThreads) mine += ps[i];
    const uint64_t Z = block_sum(mine, s_red, lane, wave);
    if (Z != 0) {
        const uint64_t T = sample_threshold(t.u_sample[b], Z);
        // piece holding the threshold: the first whose running sum exceeds T
        uint64_t carry = 0;
        for (int base = 0; base < t.npieces; base += kTvThreads) {
            const int i = base + tid;
            const uint64_t v = i < t.npieces ? ps[i] : 0;
            uint64_t total;
            const uint64_t incl = block_incl_scan(v, s_red, lane, wave, &total) + carry;
            const uint64_t excl = incl - v;
            if (i < t.npieces && excl <= T && T < incl) {  // exactly one thread
                s_piece = i;
                s_rem = T - excl;
            }
            carry += total;
        }
        __syncthreads();
        const int c = s_piece;
        select_in_piece<VEC>(prow, qrow, c * kTokenPiece, min(kTokenPiece, t.V - c * kTokenPiece), s_rem,
                             s_red, &s_tok, lane, wave);
    } else if (corr) {
        // empty correction row (p <= q everywhere at this resolution): draw
        // from p of the same row, scanning the whole row
        const int per = (t.V + kTvThreads - 1) / kTvThreads;
        const int a = min(per * tid, t.V), e = min(a + per, t.V);
        uint64_t s = 0;
        for (int x = a; x < e; ++x) s += entry_weight(prow, nullptr, x);
        const uint64_t Zp = block_sum(s, s_red, lane, wave);
        if (Zp != 0)
            select_in_range(prow, nullptr, 0, t.V, sample_threshold(t.u_sample[b], Zp), s_red, &s_tok,
                            lane, wave);
    }
    __syncthreads();
    if (tid <= t.k) {
        int v = -1;
        if (tid < n) v = t.draft[(int64_t)b * t.k + tid];
        else if (tid == n) v = s_tok;
        t.out_tokens[(int64_t)b * (t.k + 1) + tid] = v;
    }
    if (tid == 0) t.n_accepted[b] = n;
}

// 16-byte loads need every row 16-byte aligned: V % 4 == 0 and aligned bases
static bool token_vec(const TokenProblem &t) {
    return (t.V % 4) == 0 && ((uintptr_t)t.p & 15u) == 0 && ((uintptr_t)t.q & 15u) == 0;
}

hipError_t launch_token_weights(const TokenProblem &t, hipStream_t st) {
    const dim3 grid((t.npieces + kTvWaves - 1) / kTvWaves, t.B), block(kTvThreads);
    if (token_vec(t)) hipLaunchKernelGGL(token_weights_kernel<true>, grid, block, 0, st, t);
    else hipLaunchKernelGGL(token_weights_kernel<false>, grid, block, 0, st, t);
    return hipGetLastError();
}

hipError_t launch_token_select(const TokenProblem &t, hipStream_t st) {
    if (token_vec(t)) hipLaunchKernelGGL(token_select_kernel<true>, dim3(t.B), dim3(kTvThreads), 0, st, t);
    else hipLaunchKernelGGL(token_select_kernel<false>, dim3(t.B), dim3(kTvThreads), 0, st, t);
    return hipGetLastError();
}

}  // namespace spire
