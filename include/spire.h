/*
 * spire.h -- C ABI of the speculative-round attention library for MI355X (gfx950).
 *
 * A speculation round (paper Sec. 2) runs the draft model k times on one token
 * and then the target model once on k+1 tokens in parallel; in the
 * large-batch, long-context regime the paper targets (Sec. 1, Sec. 3.1) the
 * cost of each of those forward passes is dominated by reading the KV cache
 * inside attention.  This library computes exactly that attention:
 *
 *   spire_verify_attn        -- target verification (Sec. 2, t_verify): k+1
 *                               queries per sequence, causal among themselves,
 *                               over the sequence's whole variable-length,
 *                               grouped-query KV cache (contiguous or paged).
 *   spire_draft_sparse_attn  -- one draft step (Sec. 3.1, Sec. 4): one query per
 *                               sequence over S attention-sink tokens plus a
 *                               sliding window of the W most recent positions
 *                               kept in a ring buffer (StreamingLLM mask).
 *
 * Attention definition used by both (the paper does not spell it out): for each
 * visible key j, s_j = sm_scale * <q, K_j>; out = sum_j softmax(s)_j V_j and
 * lse = ln sum_j exp(s_j).  Query head h reads KV head h / (Hq / Hkv).  A row
 * with no visible key returns zeros and lse = -inf.
 *
 * Conventions for every entry point
 *  - All data pointers are DEVICE pointers (memory of the current HIP device);
 *    the spire_kv descriptor itself is a HOST struct read during the call.
 *  - Every buffer is borrowed: the library never allocates device memory,
 *    never frees, and keeps no pointer after the call returns.  Scratch memory
 *    comes from the caller's `workspace` (sized by *_workspace_size).
 *  - Work is enqueued on `stream` and the call returns without synchronising;
 *    the caller keeps every buffer alive until the stream has passed it.
 *  - Calls that share one workspace must be ordered on one stream.
 *  - Arguments are validated on the host before anything is enqueued; invalid
 *    input returns a status and enqueues nothing.  Device-resident values
 *    (lengths, block tables, ring offsets) are clamped on the device to what
 *    the descriptors allow, so no value of them can make a kernel read outside
 *    the described storage.
 *  - Results are deterministic: the same inputs give bitwise identical output
 *    (fixed work partition, no floating-point atomics).
 *  - On a non-OK status spire_last_error() returns a message for the calling
 *    thread.
 *  - The library holds no mutable state besides a per-device cache of the
 *    compute-unit count: calls from several host threads, each with its own
 *    workspace, need no locking.
 */
#ifndef SPIRE_H
#define SPIRE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPIRE_VERSION 1

typedef enum spire_dtype {
    SPIRE_F32 = 0,        /* IEEE binary32 */
    SPIRE_BF16 = 1,       /* bfloat16 (upper half of binary32) */
    SPIRE_FP8_E4M3FN = 2  /* OCP 8-bit e4m3fn (bias 7, no inf, max 448), KV only */
} spire_dtype;

typedef enum spire_status {
    SPIRE_OK = 0,
    SPIRE_ERR_INVALID_ARG = 1,  /* null pointer, negative size, bad stride, ... */
    SPIRE_ERR_UNSUPPORTED = 2,  /* valid request outside what the kernels implement */
    SPIRE_ERR_WORKSPACE = 3,    /* workspace missing or smaller than *_workspace_size */
    SPIRE_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed */
} spire_status;

/*
 * A K/V cache view.  Element (blk, h, t, d) of K lives at
 *   k + (blk * s_blk + h * s_head + t * s_tok + d) * sizeof(dtype)
 * and likewise for V (same strides).  d is contiguous and each row of D
 * elements must start 16-byte aligned (strides multiples of 16 bytes).
 *   contiguous (page_size == 0): blk = sequence index b, t = key index j,
 *     j < capacity; `capacity` is the number of token rows per sequence.
 *   paged (page_size > 0): blk = block_table[b * max_blocks + j / page_size],
 *     t = j % page_size; page ids are clamped to [0, num_blocks).
 * fp8 storage needs per-KV-head dequantisation scales: the value of a stored
 * byte is decode(byte) * k_scale[h] (keys) or * v_scale[h] (values); the
 * scales must be finite and > 0 (device data: not checked).
 */
typedef struct spire_kv {
    const void *k;               /* device */
    const void *v;               /* device */
    const int32_t *block_table;  /* device [B, max_blocks] int32, paged only (else NULL) */
    const float *k_scale;        /* device [Hkv] fp32, fp8 only (else NULL) */
    const float *v_scale;        /* device [Hkv] fp32, fp8 only (else NULL) */
    int64_t s_blk;               /* element strides (not bytes) */
    int64_t s_head;
    int64_t s_tok;
    int32_t dtype;               /* spire_dtype */
    int32_t page_size;           /* 0 = contiguous; paged: tokens per page */
    int32_t max_blocks;          /* paged: columns of block_table */
    int32_t num_blocks;          /* paged: physical pages addressable in k / v */
    int32_t capacity;            /* contiguous: token rows per sequence */
    int32_t reserved;            /* must be 0 */
} spire_kv;

/* Bytes of workspace spire_verify_attn needs for these sizes on the current
 * device (0 on invalid sizes). */
size_t spire_verify_workspace_size(int32_t B, int32_t Hq, int32_t Hkv, int32_t D, int32_t k);

/*
 * Target verification attention (paper Sec. 2: the target forward pass on the
 * k+1 tokens of a round in parallel).
 *   q        [B, k+1, Hq, D] contiguous, q_dtype SPIRE_F32 or SPIRE_BF16;
 *            row i of sequence b is the last accepted token (i = 0) or draft
 *            token i.
 *   kv       cache of every sequence; the k+1 tokens being verified have been
 *            appended already, so sequence b holds n_b = kv_lens[b] keys.
 *   kv_lens  [B] int32: n_b; query i sees keys [0, n_b - k + i) (bottom-right
 *            causal mask).  n_b >= k+1 for a full result; smaller values are
 *            legal (rows with no visible key return zeros, lse = -inf); values
 *            above the cache capacity are clamped to it.
 *   sizes    0 <= B <= 8192, Hkv >= 1, Hq % Hkv == 0, D in {64, 128},
 *            0 <= k <= 15, (k+1) * Hq / Hkv <= 128 (SPIRE_ERR_UNSUPPORTED
 *            beyond these limits).
 *   sm_scale softmax scale (usually 1/sqrt(D)); finite and > 0, else
 *            SPIRE_ERR_INVALID_ARG.
 *   out      [B, k+1, Hq, D] contiguous, out_dtype SPIRE_F32 or SPIRE_BF16.
 *   lse      [B, k+1, Hq] fp32 natural-log sum-exp, or NULL.
 *   workspace >= spire_verify_workspace_size(B, Hq, Hkv, D, k) bytes of device
 *            memory, 256-byte aligned; its contents need no initialisation.
 * Supported storage: KV f32, bf16 or fp8 (fp8 needs k_scale and v_scale).
 * Non-finite values in the visible keys act as in the definition: a NaN key,
 * or a key whose score is +inf, makes the rows that see it NaN (output and
 * lse); a NaN or infinite value makes the output elements of its dimension
 * NaN or infinite in the rows that see it; a score of -inf weighs zero, so a
 * row whose visible scores are all -inf is an empty row.  Storage outside a
 * row's visible keys never influences that row, whatever it holds -- also
 * keys [n_b - k + i, n_b), which only later rows see.
 */
spire_status spire_verify_attn(const void *q, int32_t q_dtype, const spire_kv *kv,
                               const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                               int32_t D, int32_t k, float sm_scale, void *out,
                               int32_t out_dtype, float *lse, void *workspace,
                               size_t workspace_bytes, hipStream_t stream);

/*
 * spire_verify_attn for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * arguments without a workspace, the same kernels and results.  Its scratch
 * memory (the work partition and the partial results of split segments) is an
 * 80 MiB array of the library in device memory, one per device, held from the
 * library's load until the process ends; the first call on a device looks up
 * that device's copy.  A call whose scratch need, spire_verify_workspace_size
 * of the kernel it takes, exceeds it returns SPIRE_ERR_UNSUPPORTED and
 * enqueues nothing (on a 256-CU MI355X at head_dim 128 that is fp8 K/V with 80
 * rows per KV head, (k+1) * Hq / Hkv = 80; the 72 rows of k = 8 with 8 query
 * heads per KV head need 72.6 MiB).
 * The call allocates and frees nothing.  Every call on a device shares its
 * array: calls that may overlap on one device (several streams or host
 * threads) race and must be ordered by the caller; calls in order on one
 * stream are safe.  The array needs no clearing between calls.
 */
spire_status spire_verify_attn_noalloc(const void *q, int32_t q_dtype, const spire_kv *kv,
                                       const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                                       int32_t D, int32_t k, float sm_scale, void *out,
                                       int32_t out_dtype, float *lse, hipStream_t stream);

/* Bytes of workspace spire_draft_sparse_attn needs (0 on invalid sizes). */
size_t spire_draft_workspace_size(int32_t B, int32_t Hq, int32_t Hkv, int32_t D);

/*
 * One draft step of static sparse attention (paper Sec. 3.1 and Sec. 4: a
 * StreamingLLM mask of S sink tokens plus a window of W positions keeps the
 * draft KV cache at constant size).
 *   q        [B, Hq, D] contiguous: one query per sequence (f32 or bf16).
 *   sink     contiguous view (page_size 0, capacity >= S): row p < S holds
 *            logical position p.
 *   ring     contiguous view (page_size 0, capacity >= W) of W slots: logical
 *            position p >= S lives in slot (ring_offset[b] + p - S) mod W.
 *            sink and ring have the same dtype (fp8: each view's own scales).
 *            The sink view may have NULL k/v when S == 0, the ring view when
 *            W == 0 (they are never read then).
 *   seq_lens [B] int32: m_b, the number of logical positions including the
 *            query's own token (the caller has written it to the cache).
 *            Visible positions: [0, min(S, m_b)) U [max(S, m_b - W), m_b),
 *            each counted once.  m_b <= 0 gives zeros and lse = -inf.
 *   ring_offset [B] int32, reduced modulo W on the device.
 *   sizes    S >= 0, W >= 0, S + W >= 1, other sizes as for verify with k = 0.
 *   out      [B, Hq, D]; lse [B, Hq] or NULL; workspace as for verify.
 * Non-finite values in visible positions act as for verify.
 */
spire_status spire_draft_sparse_attn(const void *q, int32_t q_dtype, const spire_kv *sink,
                                     const spire_kv *ring, const int32_t *seq_lens,
                                     const int32_t *ring_offset, int32_t B, int32_t Hq,
                                     int32_t Hkv, int32_t D, int32_t S, int32_t W, float sm_scale,
                                     void *out, int32_t out_dtype, float *lse, void *workspace,
                                     size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace spire_token_verify needs (0 on invalid sizes). */
size_t spire_token_verify_workspace_size(int32_t B, int32_t k, int32_t V);

/*
 * Token verification of one speculation round: the modified rejection
 * sampling that follows the target's verify pass and makes the accepted
 * tokens follow the target's distribution (paper Sec. 1 and Sec. 6; Table 1:
 * a round emits 1..k+1 tokens, 0..k accepted before the first rejection).
 * For each sequence b:
 *   n = the number of leading draft tokens x_i (i < k) with
 *       u_accept[b,i] * q(b,i,x_i) < p(b,i,x_i)   (accept with probability
 *       min(1, p/q); the product is formed exactly in fp64; a token outside
 *       [0, V) or a NaN is a rejection);
 *   the emitted token is drawn with u_sample[b] from the correction
 *   distribution norm(max(0, p(b,n,.) - q(b,n,.))) when n < k, else from the
 *   bonus distribution p(b,k,.).
 * Sampling is an inverse CDF over integer weights W(x) = floor(w(x) * 2^40),
 * w = clamp(p - q, 0, 1) rounded to fp32 (correction) or clamp(p, 0, 1)
 * (bonus), NaN weighing 0: with Z = sum W and U = floor(u * 2^24) clamped to
 * [0, 2^24 - 1], the token is the smallest x whose running weight exceeds
 * floor(U * Z / 2^24).  A token of zero weight is never drawn; a correction
 * row with Z = 0 draws from p(b,n,.) instead; a row of p with Z = 0 emits -1.
 * Results do not depend on the order of any summation (integer arithmetic).
 *   p_target     [B, k+1, V] fp32 target probabilities; row i scores the
 *                token after the last accepted token and draft tokens 1..i.
 *   q_draft      [B, k, V] fp32 draft probabilities (NULL allowed if k == 0).
 *   draft_tokens [B, k] int32 x_1..x_k;  u_accept [B, k] fp32;  u_sample [B]
 *                fp32 -- uniforms in [0, 1) supplied by the caller.
 *   sizes        0 <= B <= 65535, 0 <= k <= 32, 1 <= V <= 2^20.
 *   n_accepted   [B] int32 out: n.
 *   out_tokens   [B, k+1] int32 out: the n accepted draft tokens, the emitted
 *                token, then -1.
 *   workspace    >= spire_token_verify_workspace_size(B, k, V) bytes, 256-byte
 *                aligned, contents need no initialisation.
 * All arrays are contiguous device memory, 4-byte aligned.
 */
spire_status spire_token_verify(const float *p_target, const float *q_draft,
                                const int32_t *draft_tokens, const float *u_accept,
                                const float *u_sample, int32_t B, int32_t k, int32_t V,
                                int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace spire_block_verify needs (0 on invalid sizes). */
size_t spire_block_verify_workspace_size(int32_t B, int32_t k, int32_t V);

/*
 * Block verification of one speculation round: the alternative to token
 * verification the paper names (Sec. 6: its results should hold with block
 * verification too); the draft block is judged as a whole.  Arguments,
 * sizes, outputs and the sampling of the emitted token are those of
 * spire_token_verify; the accepted count n is defined instead by, for each
 * sequence b with p(i,.) = p_target[b,i,.], q(i,.) = q_draft[b,i,.]:
 *   w_0 = 1;  w_i = 1 if t >= q(i-1, x_i), else t / q(i-1, x_i), with
 *             t = w_{i-1} * p(i-1, x_i)                 (i = 1..k, fp64),
 *             and w_i = 0 when w_{i-1} = 0, x_i is outside [0, V), p(i-1, x_i)
 *             is not > 0 or q(i-1, x_i) is not >= 0 (NaN included);
 *   residual row i < k: r_i(x) = w32 * p(i, x) - q(i, x), w32 = w_i rounded
 *             to fp32, both operations rounded in fp32 (no fused multiply-add),
 *             turned into integer weights as for token verification; S_i =
 *             the sum of row i's weights;
 *   h_i = S / (S + (1 - w_i) * 2^40) in fp64 with S = S_i rounded once to
 *             fp64 (h_i = 1 if the denominator is 0), for i < k;  h_k = w_k;
 *   n = the largest i in 1..k with u_accept[b, i-1] < h_i, or 0.
 * The emitted token is drawn with u_sample[b] from row n's residual weights
 * when n < k (from p(n,.) if they sum to 0), else from p(k,.).  Emitted tokens
 * follow the target's distribution, and on average at least as many are
 * accepted as by token verification.  Reads every row of p and q.
 *   workspace  >= spire_block_verify_workspace_size(B, k, V) bytes, 256-byte
 *              aligned, contents need no initialisation.
 */
spire_status spire_block_verify(const float *p_target, const float *q_draft,
                                const int32_t *draft_tokens, const float *u_accept,
                                const float *u_sample, int32_t B, int32_t k, int32_t V,
                                int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                size_t workspace_bytes, hipStream_t stream);

/*
 * Append the K/V of newly verified tokens to the target cache (paper Sec. 2:
 * the target's forward pass on the k+1 tokens of a round produces their K/V).
 *   kv        destination view (paged or contiguous, as for spire_verify_attn);
 *             its k / v storage is WRITTEN (the descriptor's const only means
 *             the struct is not modified).  fp8 storage needs k_scale / v_scale.
 *   k_new, v_new  [B, T, Hkv, D] contiguous, new_dtype SPIRE_F32 or SPIRE_BF16.
 *   positions [B] int32: token t of sequence b goes to cache position
 *             positions[b] + t (usually the length before the append).  A
 *             position without storage (negative, at or beyond the contiguous
 *             capacity, a block beyond max_blocks or a page id outside
 *             [0, num_blocks)) is skipped, so no value makes the kernel write
 *             outside the described storage.
 * Rounding to storage: f32 keeps the value (bf16 input widened exactly);
 * bf16 rounds to nearest even (NaN stays a quiet NaN); fp8 stores the OCP
 * e4m3fn code nearest to value / scale[h] (fp32 division; ties to the even
 * code; magnitudes beyond 448 and infinities saturate to +-448; NaN -> 0x7F).
 * Pages of the new positions must already be in block_table (page
 * allocation belongs to the caller).  Sizes: B >= 0, T >= 0, Hkv >= 1,
 * 1 <= D <= 1024.  No workspace.
 */
spire_status spire_kv_append(const spire_kv *kv, const void *k_new, const void *v_new,
                             int32_t new_dtype, const int32_t *positions, int32_t B, int32_t Hkv,
                             int32_t D, int32_t T, hipStream_t stream);

/*
 * One draft step's write into the constant-size StreamingLLM cache (paper
 * Sec. 3.1): the token at logical position p = seq_lens[b] - 1 is stored in
 * sink row p (p < S) or ring slot (ring_offset[b] + p - S) mod W, rounded as
 * for spire_kv_append (sink and ring have one dtype; fp8 uses each view's own
 * scales).  seq_lens is the m_b of the draft attention that follows.
 *   k_new, v_new  [B, Hkv, D] contiguous, SPIRE_F32 or SPIRE_BF16.
 *   spill_k, spill_v  [B, Hkv, D] in the storage dtype, or both NULL: before
 *             writing, the row being overwritten is copied there (for a full
 *             ring, p >= S + W, that is the evicted position p - W).  Keep
 *             one spill area per step of the round for spire_draft_rollback.
 * A sequence with p < 0, or p >= S without a window (W == 0), writes nothing.
 */
spire_status spire_draft_append(const spire_kv *sink, const spire_kv *ring, const void *k_new,
                                const void *v_new, int32_t new_dtype, const int32_t *seq_lens,
                                const int32_t *ring_offset, int32_t B, int32_t Hkv, int32_t D,
                                int32_t S, int32_t W, void *spill_k, void *spill_v,
                                hipStream_t stream);

/*
 * Undo the draft writes of rejected steps after token verification.  Step s
 * of the round (s = 0 .. steps-1) wrote logical position base_lens[b] + s and
 * kept the overwritten row in spill[s] (spill_k / spill_v are
 * [steps, B, Hkv, D] in the storage dtype).  With n_accepted[b] = n, steps
 * s > n wrote rejected tokens: their rows get the spilled bytes back, latest
 * step first, so afterwards sink and ring hold exactly the bytes that steps
 * 0 .. n alone would have left (also when steps of one round share a slot).
 */
spire_status spire_draft_rollback(const spire_kv *sink, const spire_kv *ring, const void *spill_k,
                                  const void *spill_v, const int32_t *base_lens,
                                  const int32_t *n_accepted, int32_t steps,
                                  const int32_t *ring_offset, int32_t B, int32_t Hkv, int32_t D,
                                  int32_t S, int32_t W, hipStream_t stream);

/*
 * Feedback-memory mixing of the draft (paper Sec. 3.3): the draft is a Feedback
 * Transformer whose attention reads memory vectors, one per draft layer i,
 * each a convex mix of the token's activations after every layer (layer 0 is
 * the embedding):
 *     m[i] = sum_l exp(w[i][l]) x[l] / sum_l exp(w[i][l]).
 *   x        [layers, B, d] contiguous, x_dtype SPIRE_F32 or SPIRE_BF16: the
 *            activations of the step's tokens after each layer.
 *   w        [n_out, layers] fp32 device array of the learnable weights
 *            (any finite values; the row maximum is subtracted before exp).
 *   m        [n_out, B, d] contiguous, m_dtype SPIRE_F32 or SPIRE_BF16 (RNE).
 *   sizes    1 <= n_out <= 8, 1 <= layers <= 64, B >= 0, d >= 0.
 * Arithmetic in fp32 (mixing weights and accumulation).  No workspace.
 */
spire_status spire_feedback_memory(const void *x, int32_t x_dtype, const float *w, int32_t n_out,
                                   int32_t layers, int32_t B, int32_t d, void *m, int32_t m_dtype,
                                   hipStream_t stream);

/*
 * Streaming-read probe (a measurement aid, not a step of the method): reads
 * the `bytes` bytes at device pointer `buf` once with 16-byte nontemporal
 * loads, as a plain streaming kernel does, and writes an XOR fold of what it
 * read to the device array `sink` of `sink_words` words, which must be at
 * least SPIRE_HBM_PROBE_SINK_WORDS (else SPIRE_ERR_INVALID_ARG); the first
 * SPIRE_HBM_PROBE_SINK_WORDS words are written, and their XOR equals the XOR
 * of every 32-bit word of the buffer.  Its duration gives
 * the HBM read rate this device reaches in practice, the ceiling the
 * attention kernels are compared against beside the 8 TB/s specification.
 *   buf   16-byte aligned, bytes a multiple of 16 (0 is allowed: nothing read,
 *         the sink still written);
 *   sink  4-byte aligned.
 * Asynchronous on `stream`; allocates nothing.
 */
#define SPIRE_HBM_PROBE_SINK_WORDS 2048
spire_status spire_hbm_read_probe(const void *buf, size_t bytes, uint32_t *sink, size_t sink_words,
                                  hipStream_t stream);

/* Human-readable name of a status code (static string, never NULL); any
 * value is accepted, unknown ones give "SPIRE_ERR_UNKNOWN". */
const char *spire_status_string(int32_t status);

/* Detail message of the last non-OK status returned on the calling thread
 * (thread-local static storage, "" if none). */
const char *spire_last_error(void);

/* SPIRE_VERSION of the built library. */
int32_t spire_version(void);

/*
 * Per-call options of the entry points that launch several kernels
 * (spire_verify_attn_ex, spire_draft_sparse_attn_ex, spire_token_verify_ex,
 * spire_block_verify_ex).
 * A NULL pointer, or a zero-initialised struct, means the defaults; the
 * library reads the struct and writes the host arrays it points to only
 * during the call and keeps nothing afterwards, so calls stay reentrant.
 *   kernel        attention family (the token and block verification entry
 *                 points ignore it):
 *                 0 automatic -- the matrix-core kernels where dtype and shape
 *                 allow (LDS-staged above 32 rows per KV head, register-staged
 *                 otherwise), the generic vector kernel for the rest;
 *                 a draft step whose B * Hkv segments number half or a
 *                 quarter of the device's waves (4 per compute unit; at least
 *                 15/16 of them filled) gives each segment 2 or 4 waves of one
 *                 workgroup and launches no plan or combine;
 *                 1 always the generic vector kernel; 2 prefer the
 *                 register-staged kernel (at most 32 rows) with the stream-K
 *                 partition of every call; 3 prefer the LDS-staged one (bf16
 *                 K/V only above 32 rows); each where its limits allow.
 *                 Results agree within the stated tolerances; the choice
 *                 exists for measurement and cross-checks.
 *   max_launches  capacity of the two arrays below; 0 records nothing.
 *   events        host array [2 * max_launches] of events the CALLER created
 *                 (hipEventCreate, timing enabled) on the stream's device:
 *                 events[2i] is recorded on `stream` right before the i-th
 *                 kernel the call launches, events[2i + 1] right after it.
 *                 Launches beyond max_launches are not recorded.
 *   kernel_ids    host array [max_launches] or NULL: the id of each recorded
 *                 launch -- 0 plan, 1 verify partial attention, 2 draft
 *                 partial attention, 3 combine, 4 token verification weights,
 *                 5 token verification select, 11 the check of the values of
 *                 keys [n - k, n) after a matrix-core verify call, 12 block
 *                 verification weights, 13 block verification select.
 *   n_launches    host int32 or NULL: set to the number of kernels the call
 *                 launched (0 when it returned before launching).
 *   reserved      must be 0.
 * Invalid options return SPIRE_ERR_INVALID_ARG before anything is enqueued.
 */
typedef struct spire_launch_opts {
    int32_t kernel;
    int32_t max_launches;
    hipEvent_t *events;
    int32_t *kernel_ids;
    int32_t *n_launches;
    int32_t reserved;
} spire_launch_opts;

spire_status spire_verify_attn_ex(const void *q, int32_t q_dtype, const spire_kv *kv,
                                  const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                                  int32_t D, int32_t k, float sm_scale, void *out,
                                  int32_t out_dtype, float *lse, void *workspace,
                                  size_t workspace_bytes, hipStream_t stream,
                                  const spire_launch_opts *opts);
spire_status spire_draft_sparse_attn_ex(const void *q, int32_t q_dtype, const spire_kv *sink,
                                        const spire_kv *ring, const int32_t *seq_lens,
                                        const int32_t *ring_offset, int32_t B, int32_t Hq,
                                        int32_t Hkv, int32_t D, int32_t S, int32_t W, float sm_scale,
                                        void *out, int32_t out_dtype, float *lse, void *workspace,
                                        size_t workspace_bytes, hipStream_t stream,
                                        const spire_launch_opts *opts);
spire_status spire_token_verify_ex(const float *p_target, const float *q_draft,
                                   const int32_t *draft_tokens, const float *u_accept,
                                   const float *u_sample, int32_t B, int32_t k, int32_t V,
                                   int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream,
                                   const spire_launch_opts *opts);
spire_status spire_block_verify_ex(const float *p_target, const float *q_draft,
                                   const int32_t *draft_tokens, const float *u_accept,
                                   const float *u_sample, int32_t B, int32_t k, int32_t V,
                                   int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream,
                                   const spire_launch_opts *opts);

#ifdef __cplusplus
}
#endif

#endif /* SPIRE_H */
