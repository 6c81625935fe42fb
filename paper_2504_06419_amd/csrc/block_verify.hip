// block_verify.hip -- block verification of a speculation round (gfx950).
//
// The alternative to token verification that the paper names (Sec. 6): the
// draft block is judged as a whole.  With P_i the target's row i and Q_i the
// draft's row i of sequence b, x_1..x_k its draft tokens:
//   p_0 = 1,  p_i = min(p_{i-1} P_{i-1}(x_i) / Q_{i-1}(x_i), 1)
//   h_i = s_i / (s_i + 1 - p_i),  s_i = sum_x max(p_i P_i(x) - Q_i(x), 0)  (i < k),
//   h_k = p_k;
// walking down from i = k, the first i with u_i < h_i is the number of
// accepted tokens tau (0 when none: h_0 = 1), and one token is drawn from the
// residual max(p_tau P_tau - Q_tau, 0) (tau < k) or from P_k (tau = k).
//
// Every decision is taken exactly as the header states, so any evaluation
// order gives the same tokens: p_i in fp64 (fixed order of the fold), residual
// entries p32 * P - Q with each operation rounded in fp32 (no fused
// multiply-add), the integer weights and threshold of token verification
// (sampling.h), s_i as exact integer sums, h_i and the comparison in fp64.
//
// Two launches, both bound by reading the probability rows (block
// verification needs every row's residual mass, token verification one row):
//   weights kernel  grid (pieces, k+1 rows, B): every wave owns one 2048-entry
//                   piece of one row, recomputes p_i (k gathers, an in-order
//                   fold across lanes) and writes the piece's weight sum;
//   select kernel   one workgroup per sequence: row sums from the piece sums,
//                   the walk, then the threshold's piece is read again and
//                   searched as in token verification.  An empty residual
//                   row, which draws from P instead, is scanned whole.
#include "sampling.h"

namespace spire {

// p_0 .. p_k of sequence b: lane j < k gathers x_{j+1}, P_j(x), Q_j(x); the
// fold runs lane by lane in order and every lane computes the same values.
// Returns p_lane on lanes 0..k (and p_k beyond).
__device__ __forceinline__ double block_prefix_weights(const TokenProblem &t, int b, int lane) {
    double P = 0.0, Q = 0.0;
    int ok = 0;
    if (lane < t.k) {
        const int x = t.draft[(int64_t)b * t.k + lane];
        if (x >= 0 && x < t.V) {
            P = (double)t.p[((int64_t)b * (t.k + 1) + lane) * t.V + x];
            Q = (double)t.q[((int64_t)b * t.k + lane) * t.V + x];
            ok = (P > 0.0 && Q >= 0.0) ? 1 : 0;  // NaN fails both
        }
    }
    double pw = 1.0, mine = 1.0;
    for (int j = 0; j < t.k; ++j) {
        const double Pj = __shfl(P, j), Qj = __shfl(Q, j);
        const int okj = __shfl(ok, j);
        if (pw > 0.0 && okj) {
            const double v = __dmul_rn(pw, Pj);
            pw = v >= Qj ? 1.0 : __ddiv_rn(v, Qj);
        } else {
            pw = 0.0;
        }
        if (lane == j + 1) mine = pw;
    }
    return lane > t.k ? pw : mine;
}

// Weight of one entry of row i: residual p32 * P - Q (Q given) or P.
__device__ __forceinline__ uint64_t block_weight(float scale, float pv, const float *qrow, int x) {
    return fixed_weight(qrow ? __fsub_rn(__fmul_rn(scale, pv), qrow[x]) : pv);
}

// h_i = S / (S + (1 - p) 2^40) in fp64, S converted with one rounding (its
// high and low 32-bit halves are exact in fp64, their sum is rounded once);
// 1 when the denominator is 0.
__device__ __forceinline__ double stop_probability(uint64_t S, double p) {
    const double Sd = __dadd_rn((double)(uint32_t)(S >> 32) * 4294967296.0, (double)(uint32_t)S);
    const double den = __dadd_rn(Sd, __dmul_rn(__dsub_rn(1.0, p), 1099511627776.0));
    return den > 0.0 ? __ddiv_rn(Sd, den) : 1.0;
}

template <bool VEC>
__global__ __launch_bounds__(kTvThreads) void block_weights_kernel(TokenProblem t) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int s = blockIdx.x * kTvWaves + wave;  // piece of the row
    const int i = blockIdx.y;                    // row 0..k
    const int b = blockIdx.z;
    if (s >= t.npieces) return;
    const bool resid = i < t.k;
    const double pw = block_prefix_weights(t, b, lane);
    const float scale = (float)__shfl(pw, i);  // p_i rounded to fp32
    const float *prow = t.p + ((int64_t)b * (t.k + 1) + i) * t.V;
    const float *qrow = resid ? t.q + ((int64_t)b * t.k + i) * t.V : nullptr;
    const int x0 = s * kTokenPiece;
    uint64_t sw = 0;
    if (VEC) {
        // coalesced 16-byte loads; V % 4 == 0, so a 4-entry group is wholly in or out
        const tv_f32x4 *p4 = reinterpret_cast<const tv_f32x4 *>(prow + x0);
        const tv_f32x4 *q4 = reinterpret_cast<const tv_f32x4 *>(resid ? qrow + x0 : prow + x0);
        const int groups = min(kTokenPiece, t.V - x0) >> 2;
        tv_f32x4 pv[kTvGroupsPerLane], qv[kTvGroupsPerLane];
        const tv_f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int g = 0; g < kTvGroupsPerLane; ++g) {
            const int gi = lane + 64 * g;
            pv[g] = gi < groups ? __builtin_nontemporal_load(p4 + gi) : zero;
            qv[g] = (resid && gi < groups) ? __builtin_nontemporal_load(q4 + gi) : zero;
        }
#pragma unroll
        for (int g = 0; g < kTvGroupsPerLane; ++g) {
            if (resid) {
#pragma unroll
                for (int e = 0; e < 4; ++e) sw += fixed_weight(__fsub_rn(__fmul_rn(scale, pv[g][e]), qv[g][e]));
            } else {
                sw += fixed_weight(pv[g].x) + fixed_weight(pv[g].y) + fixed_weight(pv[g].z) + fixed_weight(pv[g].w);
            }
        }
    } else {
        const int cnt = min(kTokenPiece, t.V - x0);
#pragma unroll 4
        for (int e = 0; e < kTokenPiece / 64; ++e) {
            const int xi = lane + 64 * e;
            if (xi < cnt) sw += block_weight(scale, prow[x0 + xi], qrow, x0 + xi);
        }
    }
    sw = wave_sum(sw);
    if (lane == 0) t.piece_sum[((int64_t)b * (t.k + 1) + i) * t.npieces + s] = sw;
}

// Token in piece entries [x0, x0 + cnt) whose running weight first exceeds R
// (R below the piece's total); as token verification's search, with the
// weights of a block verification row.
template <bool VEC>
__device__ __forceinline__ void block_select_in_piece(const float *prow, const float *qrow, float scale, int x0,
                                                      int cnt, uint64_t R, uint64_t *s_red, int *s_tok,
                                                      int lane, int wave) {
    const int base = kTvSlice * (int)threadIdx.x;
    float pv[kTvSlice], qv[kTvSlice];
    if (VEC) {
        const tv_f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int g = 0; g < kTvSlice / 4; ++g) {
            const bool in = base + 4 * g < cnt;
            const tv_f32x4 a = in ? *reinterpret_cast<const tv_f32x4 *>(prow + x0 + base + 4 * g) : zero;
            const tv_f32x4 c = (in && qrow) ? *reinterpret_cast<const tv_f32x4 *>(qrow + x0 + base + 4 * g)
                                            : zero;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                pv[4 * g + e] = a[e];
                qv[4 * g + e] = c[e];
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < kTvSlice; ++e) {
            const bool in = base + e < cnt;
            pv[e] = in ? prow[x0 + base + e] : 0.f;
            qv[e] = (in && qrow) ? qrow[x0 + base + e] : 0.f;
        }
    }
    uint64_t w[kTvSlice];
    uint64_t sum = 0;
#pragma unroll
    for (int e = 0; e < kTvSlice; ++e) {
        // entries past cnt hold 0 and weigh 0 either way
        w[e] = fixed_weight(qrow ? __fsub_rn(__fmul_rn(scale, pv[e]), qv[e]) : pv[e]);
        sum += w[e];
    }
    uint64_t total;
    const uint64_t ti = block_incl_scan(sum, s_red, lane, wave, &total);
    const uint64_t te = ti - sum;
    if (te <= R && R < ti) {  // exactly one thread
        uint64_t run = te;
        int found = -1;
#pragma unroll
        for (int e = 0; e < kTvSlice; ++e) {
            run += w[e];
            if (found < 0 && run > R) found = e;
        }
        *s_tok = x0 + base + found;
    }
}

// Token of P_row drawn with u over the whole row (an empty residual row's
// fallback): every thread owns a contiguous slice, the block scans the slice
// sums, the thread whose slice holds the threshold walks it again.
__device__ __forceinline__ void block_select_from_p(const float *prow, int V, float u, uint64_t *s_red,
                                                    int *s_tok, int lane, int wave) {
    const int per = (V + kTvThreads - 1) / kTvThreads;
    const int a = min(per * (int)threadIdx.x, V), e = min(a + per, V);
    uint64_t sum = 0;
    for (int x = a; x < e; ++x) sum += fixed_weight(prow[x]);
    uint64_t Z;
    const uint64_t ti = block_incl_scan(sum, s_red, lane, wave, &Z);
    if (Z == 0) return;  // a row of P without mass: -1
    const uint64_t R = sample_threshold(u, Z);
    const uint64_t te = ti - sum;
    if (te <= R && R < ti) {
        uint64_t run = te;
        int x = a;
        for (; x < e; ++x) {
            run += fixed_weight(prow[x]);
            if (run > R) break;
        }
        *s_tok = x;
    }
}

template <bool VEC>
__global__ __launch_bounds__(kTvThreads) void block_select_kernel(TokenProblem t) {
    __shared__ uint64_t s_red[kTvWaves];
    __shared__ int s_piece, s_tok;
    __shared__ uint64_t s_rem;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int tid = threadIdx.x;
    const int b = blockIdx.x;
    const int K = t.k;
    if (tid == 0) s_tok = -1;
    const double pw = block_prefix_weights(t, b, lane);  // p_lane on lanes 0..k

    // sum of one row's weights from its piece sums (npieces <= 512)
    auto row_sum = [&](int i) -> uint64_t {
        const uint64_t *ps = t.piece_sum + ((int64_t)b * (K + 1) + i) * t.npieces;
        uint64_t mine = 0;
        for (int c = tid; c < t.npieces; c += kTvThreads) mine += ps[c];
        return block_sum(mine, s_red, lane, wave);
    };

    // the walk: every thread takes the same decisions
    int tau = 0;
    for (int i = K; i >= 1; --i) {
        const double pi = __shfl(pw, i);
        const double h = i == K ? pi : stop_probability(row_sum(i), pi);
        if ((double)t.u_accept[(int64_t)b * K + i - 1] < h) {
            tau = i;
            break;
        }
    }

    const bool resid = tau < K;
    const float scale = (float)__shfl(pw, tau);
    const float *prow = t.p + ((int64_t)b * (K + 1) + tau) * t.V;
    const float *qrow = resid ? t.q + ((int64_t)b * K + tau) * t.V : nullptr;
    const uint64_t Z = row_sum(tau);
    const uint64_t *ps = t.piece_sum + ((int64_t)b * (K + 1) + tau) * t.npieces;
    if (Z != 0) {
        const uint64_t T = sample_threshold(t.u_sample[b], Z);
        // piece holding the threshold: the first whose running sum exceeds T
        uint64_t carry = 0;
        for (int base = 0; base < t.npieces; base += kTvThreads) {
            const int c = base + tid;
            const uint64_t v = c < t.npieces ? ps[c] : 0;
            uint64_t total;
            const uint64_t incl = block_incl_scan(v, s_red, lane, wave, &total) + carry;
            const uint64_t excl = incl - v;
            if (c < t.npieces && excl <= T && T < incl) {  // exactly one thread
                s_piece = c;
                s_rem = T - excl;
            }
            carry += total;
        }
        __syncthreads();
        const int c = s_piece;
        block_select_in_piece<VEC>(prow, qrow, scale, c * kTokenPiece, min(kTokenPiece, t.V - c * kTokenPiece),
                                   s_rem, s_red, &s_tok, lane, wave);
    } else if (resid) {
        // empty residual row: draw from P of the same row
        block_select_from_p(prow, t.V, t.u_sample[b], s_red, &s_tok, lane, wave);
    }
    __syncthreads();
    if (tid <= K) {
        int v = -1;
        if (tid < tau) v = t.draft[(int64_t)b * K + tid];
        else if (tid == tau) v = s_tok;
        t.out_tokens[(int64_t)b * (K + 1) + tid] = v;
    }
    if (tid == 0) t.n_accepted[b] = tau;
}

// 16-byte loads need every row 16-byte aligned: V % 4 == 0 and aligned bases
static bool block_vec(const TokenProblem &t) {
    return (t.V % 4) == 0 && ((uintptr_t)t.p & 15u) == 0 && (t.k == 0 || ((uintptr_t)t.q & 15u) == 0);
}

hipError_t launch_block_weights(const TokenProblem &t, hipStream_t st) {
    const dim3 grid((t.npieces + kTvWaves - 1) / kTvWaves, t.k + 1, t.B), block(kTvThreads);
    if (block_vec(t)) hipLaunchKernelGGL(block_weights_kernel<true>, grid, block, 0, st, t);
    else hipLaunchKernelGGL(block_weights_kernel<false>, grid, block, 0, st, t);
    return hipGetLastError();
}

hipError_t launch_block_select(const TokenProblem &t, hipStream_t st) {
    if (block_vec(t)) hipLaunchKernelGGL(block_select_kernel<true>, dim3(t.B), dim3(kTvThreads), 0, st, t);
    else hipLaunchKernelGGL(block_select_kernel<false>, dim3(t.B), dim3(kTvThreads), 0, st, t);
    return hipGetLastError();
}

}  // namespace spire
