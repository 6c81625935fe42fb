/*
 * spire_oracle.c -- plain fp64 CPU oracle for speculative-round attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
 * the benchmark's CPU-baseline leg load this library.  It shares no code,
 * header, table or helper with the HIP library: it decodes the stored bytes
 * itself, walks the cache layouts itself and evaluates the attention
 * definition directly, with no blocking, no online softmax and no reordering.
 *
 * What it computes (the paper never writes out the attention formula, its
 * scale, grouped heads, paging or dtypes; those follow the problem statement
 * of the library and are listed as readings in the design notes):
 *
 *  verify  -- Sec. 2 defines t_verify as one target forward pass on the k+1
 *             tokens of a round (the last accepted token plus k drafts) in
 *             parallel.  Query i (0..k) of sequence b attends causally: with
 *             n_b keys in the cache (the k+1 new tokens already appended) it
 *             sees keys [0, n_b - k + i).
 *  draft   -- Sec. 3.1 and Sec. 4: the draft model's KV cache is sparse, read
 *             through a StreamingLLM mask of S attention-sink tokens plus a
 *             sliding window of the W most recent positions, so its size does
 *             not grow with the context.  With m_b logical positions (the
 *             query's own token included) the visible set is
 *             [0, min(S, m_b))  U  [max(S, m_b - W), m_b).
 *
 *  For every visible key j:  s_j = sm_scale * sum_d q_d * K_j,d   (fp64)
 *  two-pass softmax:         M = max_j s_j,  w_j = exp(s_j - M),  L = sum w_j
 *  output:                   o_d = sum_j w_j * V_j,d / L,   lse = M + ln L
 *  Grouped-query attention:  query head h reads KV head h / (Hq / Hkv).
 *  A row with no visible key outputs zeros and lse = -inf.  A visible key whose
 *  score is -inf weighs zero (exp(-inf) = 0), so a row whose visible scores are
 *  all -inf is such an empty row too; a NaN score (a NaN key, or +inf met by
 *  -inf in the dot product) or a score of +inf makes the row NaN.
 *
 * Storage decoding (own implementation):
 *   f32   as stored;
 *   bf16  the 16 stored bits are the high half of an IEEE binary32;
 *   fp8   OCP 8-bit e4m3fn: sign bit 7, exponent bits 6..3 (bias 7), mantissa
 *         bits 2..0; exponent 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN;
 *         no infinities; the decoded value is multiplied by the per-KV-head
 *         scale (k_scale[h] for keys, v_scale[h] for values).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_F32 = 0, OR_BF16 = 1, OR_FP8 = 2 };

typedef struct {
    const void *k, *v;
    int32_t dtype;
    int64_t s_blk, s_head, s_tok;  /* element strides; the head-dim index is contiguous */
    int32_t page_size;             /* 0: block index = sequence index, token = key index */
    const int32_t *block_table;    /* [B, max_blocks] when page_size > 0 */
    int32_t max_blocks;
    const float *k_scale, *v_scale;/* [Hkv], fp8 only */
} oracle_kv;

/* ---- decoders -------------------------------------------------------- */
static double dec_bf16(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double dec_e4m3fn(uint8_t x)
{
    int sign = (x >> 7) & 1;
    int e = (x >> 3) & 0xF;
    int m = x & 0x7;
    double mag;
    if (e == 0xF && m == 0x7)
        return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, -6);
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -mag : mag;
}

static double load_elem(const void *base, int dtype, int64_t idx)
{
    switch (dtype) {
    case OR_F32: return (double)((const float *)base)[idx];
    case OR_BF16: return dec_bf16(((const uint16_t *)base)[idx]);
    case OR_FP8: return dec_e4m3fn(((const uint8_t *)base)[idx]);
    default: return NAN;
    }
}

double spire_oracle_decode(int dtype, const void *base, int64_t idx)
{
    return load_elem(base, dtype, idx);
}

int spire_oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* element offset of (key j of sequence b, kv head h, dim 0) */
static int64_t key_offset(const oracle_kv *kv, int b, int64_t j, int h)
{
    int64_t blk, tok;
    if (kv->page_size > 0) {
        blk = kv->block_table[(int64_t)b * kv->max_blocks + j / kv->page_size];
        tok = j % kv->page_size;
    } else {
        blk = b;
        tok = j;
    }
    return blk * kv->s_blk + (int64_t)h * kv->s_head + tok * kv->s_tok;
}

/* One query row over an explicit list of visible keys: keys[t] is the storage
 * offset of visible key t inside `src[t]` (0: first view, 1: second view). */
static void attend_row(const double *q, int D, double sm_scale,
                       const oracle_kv *const *views, const int *src, const int64_t *keys,
                       int64_t nvis, int h, double *scores, double *out, double *lse)
{
    int64_t t;
    int d;
    if (nvis <= 0) {
        for (d = 0; d < D; ++d) out[d] = 0.0;
        *lse = -INFINITY;
        return;
    }
    /* pass 1: scores and their maximum (a NaN score is noted, not compared) */
    double M = -INFINITY;
    int nan_score = 0;
    for (t = 0; t < nvis; ++t) {
        const oracle_kv *kv = views[src[t]];
        double ks = (kv->dtype == OR_FP8) ? (double)kv->k_scale[h] : 1.0;
        double dot = 0.0;
        for (d = 0; d < D; ++d)
            dot += q[d] * (load_elem(kv->k, kv->dtype, keys[t] + d) * ks);
        scores[t] = sm_scale * dot;
        if (isnan(scores[t])) nan_score = 1;
        else if (scores[t] > M) M = scores[t];
    }
    /* A score of -inf weighs zero, as a masked key does, so a row whose visible
     * scores are all -inf is an empty row: zeros and lse = -inf.  A NaN score
     * makes the whole row NaN (pass 2 below computes exactly that). */
    if (M == -INFINITY && !nan_score) {
        for (d = 0; d < D; ++d) out[d] = 0.0;
        *lse = -INFINITY;
        return;
    }
    /* pass 2: weights, normaliser and weighted sum of values */
    double L = 0.0;
    for (d = 0; d < D; ++d) out[d] = 0.0;
    for (t = 0; t < nvis; ++t) {
        const oracle_kv *kv = views[src[t]];
        double vs = (kv->dtype == OR_FP8) ? (double)kv->v_scale[h] : 1.0;
        double w = exp(scores[t] - M);
        L += w;
        for (d = 0; d < D; ++d)
            out[d] += w * (load_elem(kv->v, kv->dtype, keys[t] + d) * vs);
    }
    for (d = 0; d < D; ++d) out[d] /= L;
    *lse = M + log(L);
}

/*
 * Verify attention.  q: [B, k+1, Hq, D] (q_dtype f32 or bf16); output rows are
 * the selected sequences seq_ids[0..nsel) (all B in order when seq_ids is
 * NULL): out [nsel, k+1, Hq, D] fp64, lse [nsel, k+1, Hq] fp64.
 */
int spire_oracle_verify(const void *q, int q_dtype, const oracle_kv *kv, const int32_t *kv_lens,
                        const int32_t *seq_ids, int nsel, int Hq, int Hkv, int D, int k,
                        double sm_scale, double *out, double *lse)
{
    if (Hkv <= 0 || Hq % Hkv != 0 || D <= 0 || k < 0) return 1;
    const int g = Hq / Hkv;
    const int nq = k + 1;
    int64_t task;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(|| : bad)
    for (task = 0; task < (int64_t)nsel * Hkv; ++task) {
        const int r = (int)(task / Hkv), hk = (int)(task % Hkv);
        const int b = seq_ids ? seq_ids[r] : r;
        const int64_t n = kv_lens[b];
        const oracle_kv *views[1] = {kv};
        double *qrow = malloc(sizeof(double) * D);
        double *scores = malloc(sizeof(double) * (n > 0 ? n : 1));
        int64_t *keys = malloc(sizeof(int64_t) * (n > 0 ? n : 1));
        int *src = calloc((size_t)(n > 0 ? n : 1), sizeof(int));
        if (!qrow || !scores || !keys || !src) {
            bad = 1;
        } else {
            for (int64_t j = 0; j < n; ++j) keys[j] = key_offset(kv, b, j, hk);
            for (int i = 0; i < nq; ++i) {
                int64_t visible = n - k + i;  /* bottom-right causal mask */
                if (visible > n) visible = n;
                for (int hg = 0; hg < g; ++hg) {
                    const int h = hk * g + hg;
                    const int64_t qoff = (((int64_t)b * nq + i) * Hq + h) * D;
                    const int64_t ooff = (((int64_t)r * nq + i) * Hq + h) * D;
                    for (int d = 0; d < D; ++d) qrow[d] = load_elem(q, q_dtype, qoff + d);
                    attend_row(qrow, D, sm_scale, views, src, keys, visible, hk, scores,
                               out + ooff, lse + ((int64_t)r * nq + i) * Hq + h);
                }
            }
        }
        free(qrow); free(scores); free(keys); free(src);
    }
    return bad ? 2 : 0;
}

/*
 * Draft sparse attention for one draft step.  q: [B, Hq, D]; sink rows live in
 * `sink` (row p = logical position p < S), ring slots in `ring` (slot
 * (ring_offset_b + p - S) mod W holds position p >= S).  The visible set is
 * the union of the sinks and the window, each position counted once.
 */
int spire_oracle_draft(const void *q, int q_dtype, const oracle_kv *sink, const oracle_kv *ring,
                       const int32_t *seq_lens, const int32_t *ring_offset,
                       const int32_t *seq_ids, int nsel, int Hq, int Hkv, int D, int S, int W,
                       double sm_scale, double *out, double *lse)
{
    if (Hkv <= 0 || Hq % Hkv != 0 || D <= 0 || S < 0 || W < 0) return 1;
    const int g = Hq / Hkv;
    const int cap = S + W;
    int64_t task;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(|| : bad)
    for (task = 0; task < (int64_t)nsel * Hkv; ++task) {
        const int r = (int)(task / Hkv), hk = (int)(task % Hkv);
        const int b = seq_ids ? seq_ids[r] : r;
        const int64_t m = seq_lens[b];
        const oracle_kv *views[2] = {sink, ring};
        double *qrow = malloc(sizeof(double) * D);
        double *scores = malloc(sizeof(double) * (cap > 0 ? cap : 1));
        int64_t *keys = malloc(sizeof(int64_t) * (cap > 0 ? cap : 1));
        int *src = malloc(sizeof(int) * (cap > 0 ? cap : 1));
        if (!qrow || !scores || !keys || !src) {
            bad = 1;
        } else {
            int64_t nvis = 0;
            int64_t sink_end = m < S ? m : S;
            int64_t win_begin = m - W > S ? m - W : S;
            for (int64_t p = 0; p < sink_end; ++p) {          /* attention sinks */
                keys[nvis] = key_offset(sink, b, p, hk);
                src[nvis++] = 0;
            }
            for (int64_t p = win_begin; p < m; ++p) {         /* sliding window */
                int64_t slot = ((int64_t)ring_offset[b] + p - S) % W;
                if (slot < 0) slot += W;
                keys[nvis] = key_offset(ring, b, slot, hk);
                src[nvis++] = 1;
            }
            for (int hg = 0; hg < g; ++hg) {
                const int h = hk * g + hg;
                const int64_t qoff = ((int64_t)b * Hq + h) * D;
                const int64_t ooff = ((int64_t)r * Hq + h) * D;
                for (int d = 0; d < D; ++d) qrow[d] = load_elem(q, q_dtype, qoff + d);
                attend_row(qrow, D, sm_scale, views, src, keys, nvis, hk, scores, out + ooff,
                           lse + (int64_t)r * Hq + h);
            }
        }
        free(qrow); free(scores); free(keys); free(src);
    }
    return bad ? 2 : 0;
}
