/*
 * occam_oracle.c -- plain fp64 CPU oracle for OccamToken's register-anchored
 * relative evidence test (arXiv 2605.29657).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference that the HIP path is
 * checked against.  Only the tests, the smoke check and the benchmark's CPU
 * baseline leg may load it.  It shares no code, header, table or helper with
 * the GPU library, and the GPU library never calls it.
 *
 * Everything is computed in double precision with straightforward loops, in
 * the order the paper states the method:
 *
 *   1. attention logits of each anchor row against [registers ; visual] keys,
 *      scaled by 1/sqrt(d_h)                       (Sec. 3.1, Eq. (1))
 *   2. row softmax, then the mean over attention heads
 *                                                  (Eq. (1); Appendix "Stage-I
 *                                                   pruning": the vision map is
 *                                                   averaged over heads)
 *   3. anchor-row reduction: a single CLS row is taken as is (Eq. EQ:CLS);
 *      text rows are reduced by max for visual tokens and by mean for the
 *      register                                    (Eq. text_scoring);
 *      mutual scoring takes the mean over the rows for every key
 *                                                  (Eq. mutual_scoring)
 *   4. threshold tau = lambda * s(r)               (Eqs. stage1_threshold_appendix,
 *                                                   stage2_set_appendix)
 *   5. keep visual tokens with s(v) >= tau; the register is never a candidate
 *                                                  (Eqs. stage1, stage2, framework)
 *   6. ascending list of survivors per sample, packed over the batch, and a
 *      byte copy of their rows (the pruned sequence [S; T] of Algorithm 1)
 *
 * and the two threshold variants of the component ablation (Appendix, Table
 * tab:qwen_compact_component_ablation): a mean-based threshold, lambda times
 * the mean score of the sample's visual tokens, and a fixed budget, the K
 * highest-scoring visual tokens of every sample.
 *
 * Readings where the paper is silent (all listed in the design notes):
 *   - several registers: s(r) is the mean over the R register scores (MAX and
 *     SUM are offered as alternatives);
 *   - Stage II heads: the head mean is taken before the max/mean over text rows;
 *   - the softmax runs over the R+N keys given, unless the caller supplies the
 *     per-(row, head) log-sum-exp of a larger key set;
 *   - grouped-query attention: query head h reads key head h / (H / Hkv).
 *
 * Layouts (token-major, packed over a ragged batch):
 *   q[(q_off[b] + t) * H * d + h * d + e]          anchor rows of sample b
 *   k[(k_off[b] + s) * Hkv * d + g * d + e]        s in [0,R) registers,
 *                                                  s in [R, R+N_b) visual
 *   scores[k_off[b] + s]
 *   candidate prefix co_b = k_off[b] - R * b (visual tokens before sample b)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

#define ORACLE_REG_MEAN 0
#define ORACLE_REG_MAX 1
#define ORACLE_REG_SUM 2
#define ORACLE_REF_CAND_MEAN 3   /* mean over the visual tokens (the ablation's mean threshold) */
#define ORACLE_ROWS_MAX 0
#define ORACLE_ROWS_MEAN 1

/* bfloat16 is the upper half of an IEEE binary32; widening is exact. */
static double bf16_to_double(uint16_t bits)
{
    uint32_t w = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

static double load_elem(const void *base, int dtype, int64_t i)
{
    if (dtype == ORACLE_BF16)
        return bf16_to_double(((const uint16_t *)base)[i]);
    return (double)((const float *)base)[i];
}

/* Exposed so a test can compare the decoder with an independent one. */
double oracle_bf16_to_double(uint16_t bits) { return bf16_to_double(bits); }

/*
 * Steps 1-3: scores of every key of every sample.
 * scale     : softmax temperature; the paper's value is 1/sqrt(d).
 * row_lse   : optional natural-log normaliser per (anchor row, head),
 *             laid out [(q_off[b] + t) * H + h]; NULL = softmax over the keys
 *             given.
 * Returns 0, or -1 on a shape error.
 */
int oracle_scores(int B, int H, int Hkv, int d, int R,
                  const int64_t *q_off, const int64_t *k_off,
                  int dtype, const void *q, const void *k,
                  double scale, const double *row_lse, int row_reduce, double *scores)
{
    if (B < 0 || H < 1 || Hkv < 1 || H % Hkv != 0 || d < 1 || R < 1)
        return -1;
    if (row_reduce != ORACLE_ROWS_MAX && row_reduce != ORACLE_ROWS_MEAN)
        return -1;
    for (int b = 0; b < B; ++b)
        if (q_off[b + 1] - q_off[b] < 1 || k_off[b + 1] - k_off[b] < R)
            return -1;

    const int group = H / Hkv;
    int err = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t T = q_off[b + 1] - q_off[b];
        const int64_t S = k_off[b + 1] - k_off[b];
        /* abar[t][s]: head-mean attention of anchor row t to key s. */
        double *abar = (double *)calloc((size_t)(T * S), sizeof(double));
        if (!abar)
            return -1;
        /* Anchor rows are independent: one row per OpenMP task. */
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t t = 0; t < T; ++t) {
            double *logit = (double *)malloc(sizeof(double) * (size_t)S);
            double *qrow = (double *)malloc(sizeof(double) * (size_t)d);
            if (!logit || !qrow) {
#pragma omp atomic write
                err = 1;
                free(logit); free(qrow);
                continue;
            }
            const int64_t qrow_idx = q_off[b] + t;
            double *arow = abar + t * S;
            for (int h = 0; h < H; ++h) {
                const int g = h / group; /* key head read by query head h */
                for (int e = 0; e < d; ++e)
                    qrow[e] = load_elem(q, dtype, (qrow_idx * H + h) * d + e);
                /* Step 1: l_s = scale * <q_t, k_s> (Eq. (1)). */
                for (int64_t s = 0; s < S; ++s) {
                    const int64_t krow = k_off[b] + s;
                    double dot = 0.0;
                    for (int e = 0; e < d; ++e)
                        dot += qrow[e] * load_elem(k, dtype, (krow * Hkv + g) * d + e);
                    logit[s] = scale * dot;
                }
                /* Step 2: A_s = softmax(l)_s over the S keys (Eq. (1)), or
                 * exp(l_s - lse) with a caller-supplied normaliser; the head
                 * mean accumulates A / H. */
                if (row_lse) {
                    const double lse = row_lse[qrow_idx * H + h];
                    for (int64_t s = 0; s < S; ++s)
                        arow[s] += exp(logit[s] - lse) / (double)H;
                } else {
                    double m = logit[0];
                    for (int64_t s = 1; s < S; ++s)
                        if (logit[s] > m) m = logit[s];
                    double z = 0.0;
                    for (int64_t s = 0; s < S; ++s)
                        z += exp(logit[s] - m);
                    for (int64_t s = 0; s < S; ++s)
                        arow[s] += (exp(logit[s] - m) / z) / (double)H;
                }
            }
            free(logit);
            free(qrow);
        }
        /* Step 3: visual score = max over anchor rows of the head-mean map;
         * register score = mean over anchor rows (Eq. text_scoring).  In the
         * mutual-scoring form every key takes the mean over the anchor rows, the
         * average attention it receives from all of them (Eq. mutual_scoring).
         * With one anchor row all of these are the CLS row itself (Eq. EQ:CLS). */
        double *out = scores + k_off[b];
        for (int64_t s = 0; s < S; ++s) {
            if (s < R || row_reduce == ORACLE_ROWS_MEAN) {
                double acc = 0.0;
                for (int64_t t = 0; t < T; ++t)
                    acc += abar[t * S + s];
                out[s] = acc / (double)T;
            } else {
                double mx = abar[s];
                for (int64_t t = 1; t < T; ++t)
                    if (abar[t * S + s] > mx) mx = abar[t * S + s];
                out[s] = mx;
            }
        }
        free(abar);
    }
    return err ? -1 : 0;
}

/*
 * Step 4: tau_b = lambda * s_b(r), with s_b(r) the mean (or max, or sum) of
 * the R register scores of sample b.
 */
int oracle_threshold(int B, int R, const int64_t *k_off, const double *scores,
                     double lambda, int reduce, double *tau)
{
    if (B < 0 || R < 1 || !(lambda >= 0.0) || isinf(lambda))
        return -1;
    if (reduce != ORACLE_REG_MEAN && reduce != ORACLE_REG_MAX && reduce != ORACLE_REG_SUM &&
        reduce != ORACLE_REF_CAND_MEAN)
        return -1;
    for (int b = 0; b < B; ++b) {
        const double *reg = scores + k_off[b];
        double sr;
        if (reduce == ORACLE_REF_CAND_MEAN) {
            /* Mean-based threshold: the reference is the mean visual score (0 without
             * visual tokens, where no decision is taken). */
            const int64_t N = k_off[b + 1] - k_off[b] - R;
            sr = 0.0;
            for (int64_t v = 0; v < N; ++v)
                sr += reg[R + v];
            if (N > 0)
                sr /= (double)N;
        } else if (reduce == ORACLE_REG_MAX) {
            sr = reg[0];
            for (int r = 1; r < R; ++r)
                if (reg[r] > sr) sr = reg[r];
        } else {
            sr = 0.0;
            for (int r = 0; r < R; ++r)
                sr += reg[r];
            if (reduce == ORACLE_REG_MEAN)
                sr /= (double)R;
        }
        tau[b] = lambda * sr;
    }
    return 0;
}

/*
 * Step 5: keep visual token v of sample b iff scores[k_off[b] + R + v] >= tau[b].
 * kept_idx is packed over the batch: sample b's survivors, ascending, occupy
 * kept_idx[kept_offsets[b] .. kept_offsets[b] + kept_count[b]).  With an
 * index_map the value written is index_map[co_b + v] instead of v.
 */
int oracle_select(int B, int R, const int64_t *k_off, const double *scores,
                  const double *tau, const int32_t *index_map,
                  int32_t *kept_idx, int32_t *kept_count, int32_t *kept_offsets)
{
    if (B < 0 || R < 1)
        return -1;
    int32_t pos = 0;
    kept_offsets[0] = 0;
    for (int b = 0; b < B; ++b) {
        const int64_t N = k_off[b + 1] - k_off[b] - R;
        const int64_t co = k_off[b] - (int64_t)R * b;
        int32_t cnt = 0;
        for (int64_t v = 0; v < N; ++v) {
            if (scores[k_off[b] + R + v] >= tau[b]) {
                kept_idx[pos + cnt] = index_map ? index_map[co + v] : (int32_t)v;
                ++cnt;
            }
        }
        kept_count[b] = cnt;
        pos += cnt;
        kept_offsets[b + 1] = pos;
    }
    return 0;
}

/*
 * Fixed-budget variant of step 5: keep the K visual tokens of each sample with
 * the largest scores (all of them when N_b <= K).  Among equal scores the lower
 * index ranks first, so the kept set is unique.  The rank of v is the number of
 * visual tokens that come before it in that order; v is kept iff its rank is
 * below K.  Output as in oracle_select.
 */
int oracle_select_topk(int B, int R, const int64_t *k_off, const double *scores, int64_t K,
                       const int32_t *index_map, int32_t *kept_idx, int32_t *kept_count,
                       int32_t *kept_offsets)
{
    if (B < 0 || R < 1 || K < 0)
        return -1;
    int32_t pos = 0;
    kept_offsets[0] = 0;
    for (int b = 0; b < B; ++b) {
        const double *sv = scores + k_off[b] + R;
        const int64_t N = k_off[b + 1] - k_off[b] - R;
        const int64_t co = k_off[b] - (int64_t)R * b;
        int32_t cnt = 0;
        for (int64_t v = 0; v < N; ++v) {
            int64_t rank = 0;
            for (int64_t u = 0; u < N; ++u)
                if (sv[u] > sv[v] || (sv[u] == sv[v] && u < v))
                    ++rank;
            if (rank < K) {
                kept_idx[pos + cnt] = index_map ? index_map[co + v] : (int32_t)v;
                ++cnt;
            }
        }
        kept_count[b] = cnt;
        pos += cnt;
        kept_offsets[b + 1] = pos;
    }
    return 0;
}

/*
 * Step 6: dst row kept_offsets[b] + i  <-  src row of (b, kept_idx[...]).
 * Each sample owns N_b + src_pad_rows consecutive source rows whose visual
 * rows start at src_row0, so the source row of visual token v of sample b is
 * co_b + b * src_pad_rows + src_row0 + v.  Rows are copied byte for byte.
 */
int oracle_gather(int B, int R, const int64_t *k_off,
                  const unsigned char *src, int64_t src_pad_rows,
                  int64_t src_row0, int64_t src_row_stride_bytes,
                  unsigned char *dst, int64_t dst_row_stride_bytes, int64_t row_bytes,
                  const int32_t *kept_idx, const int32_t *kept_offsets)
{
    if (B < 0 || R < 1 || row_bytes < 0)
        return -1;
    for (int b = 0; b < B; ++b) {
        const int64_t co = k_off[b] - (int64_t)R * b;
        const int64_t base = co + (int64_t)b * src_pad_rows + src_row0;
        for (int32_t i = kept_offsets[b]; i < kept_offsets[b + 1]; ++i) {
            const int64_t row = base + kept_idx[i];
            memcpy(dst + (int64_t)i * dst_row_stride_bytes,
                   src + row * src_row_stride_bytes, (size_t)row_bytes);
        }
    }
    return 0;
}

/* Effective number of attended tokens, exp(-sum a ln a) (Sec. 3.2, Obs. 1). */
double oracle_neff(const double *alpha, int64_t n)
{
    double h = 0.0;
    for (int64_t i = 0; i < n; ++i)
        if (alpha[i] > 0.0)
            h -= alpha[i] * log(alpha[i]);
    return exp(h);
}

/*
 * Test-time register construction (Algorithm 1, "redirect sinks to r"; Appendix
 * Eq. register_redirect_appendix), in place on an activation tensor laid out like
 * the keys: sample b owns rows k_off[b] .. k_off[b+1]-1, R register rows first,
 * each `width` elements, `stride` elements apart.  For every listed channel k:
 * h[register row reg_slot, k] = max over the visual rows of h[v, k] (a zero maximum
 * is stored as +0), then h[v, k] = 0 for every visual row.  Readings: an index
 * outside [0, width) is ignored, a repeated index acts once (its first
 * occurrence), a sample without visual rows is left unchanged.
 */
static void store_elem(void *base, int dtype, int64_t idx, double v)
{
    if (dtype == ORACLE_BF16) {
        /* v is a value read from this tensor, so its bf16 encoding is exact. */
        float f = (float)v;
        uint32_t u;
        memcpy(&u, &f, sizeof u);
        ((uint16_t *)base)[idx] = (uint16_t)(u >> 16);
    } else {
        ((float *)base)[idx] = (float)v;
    }
}

int oracle_register_redirect(int B, int R, const int64_t *k_off, int dtype, void *h,
                             int64_t width, int64_t stride, const int32_t *channels,
                             int n_channels, int reg_slot)
{
    if (B < 0 || R < 1 || width < 1 || stride < width || n_channels < 0 ||
        reg_slot < 0 || reg_slot >= R)
        return -1;
    for (int b = 0; b < B; ++b) {
        const int64_t first = k_off[b], N = k_off[b + 1] - k_off[b] - R;
        if (N < 0)
            return -1;
        if (N == 0)
            continue;
        for (int j = 0; j < n_channels; ++j) {
            const int32_t k = channels[j];
            if (k < 0 || k >= width)
                continue;
            int repeat = 0;
            for (int i = 0; i < j; ++i)
                if (channels[i] == k)
                    repeat = 1;
            if (repeat)
                continue;
            double m = load_elem(h, dtype, (first + R) * stride + k);
            for (int64_t v = 1; v < N; ++v) {
                const double x = load_elem(h, dtype, (first + R + v) * stride + k);
                if (x > m)
                    m = x;
            }
            if (m == 0.0)
                m = 0.0; /* +0 */
            store_elem(h, dtype, (first + reg_slot) * stride + k, m);
            for (int64_t v = 0; v < N; ++v)
                store_elem(h, dtype, (first + R + v) * stride + k, 0.0);
        }
    }
    return 0;
}
