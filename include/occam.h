/*
 * occam.h -- C ABI of the MI355X (gfx950) register-anchored relative evidence
 * test of OccamToken (arXiv 2605.29657): the data-parallel step that decides
 * which visual tokens reach an LLM's prefill.
 *
 * The paper's rule (Sec. 3.2, Eq. framework; Sec. 3.4 Eq. stage1; Sec. 3.5
 * Eq. stage2) keeps a visual token v of sample x when
 *
 *      s_x(v) >= lambda * s_x(r(x)),
 *
 * where s_x is the head-averaged softmax attention that the anchor rows pay to
 * each key and r(x) is the test-time register token.  One entry point exists
 * per step of that rule, plus a fused one:
 *
 *   occam_score      steps 1-2: anchor logits, row softmax, head mean, anchor
 *                    reduction (Eq. (1); Eq. EQ:CLS; Eq. text_scoring)
 *   occam_threshold  step 3: tau_b = lambda * s_b(r) (Eqs.
 *                    stage1_threshold_appendix, stage2_set_appendix)
 *   occam_select     step 4-5: s(v) >= tau test and ascending prefix-scan
 *                    compaction of the survivors (Eqs. stage1, stage2)
 *   occam_gather     step 5: dense copy of the survivors' rows (the pruned
 *                    sequence [S; T] of Algorithm 1)
 *   occam_prune      all of the above on one stream, no host synchronisation
 *
 * Conventions shared by every call
 * --------------------------------
 * Shapes.  B samples; H query heads, Hkv key heads (H % Hkv == 0; query head h
 * reads key head h / (H / Hkv)); head dim d; R register keys; T_b anchor rows
 * of sample b (T = 1: the vision encoder's CLS row, Stage I; T > 1: the LLM's
 * text rows, Stage II); N_b visual candidates of sample b.
 *
 * Layouts (row-major, token-major, packed over the batch):
 *   q        [(qo_b + t) * H * d + h * d + e]        anchor rows
 *   k        [(ko_b + s) * Hkv * d + g * d + e]      s in [0,R): registers,
 *                                                   s in [R, R+N_b): visual
 *   scores   [ko_b + s]                              float32
 *   row_lse  [(qo_b + t) * H + h]                    float32, natural log
 *   tau      [b]                                     float32
 * with qo_b = q_offsets[b] (or b * rows) and ko_b = key_offsets[b] (or
 * b * (R + cands)).  The candidate prefix co_b = ko_b - R * b counts the
 * visual tokens of the samples before b.
 *
 * Survivor lists are packed over the batch: sample b's survivors occupy
 * kept_idx[kept_offsets[b] .. kept_offsets[b] + kept_count[b]), ascending
 * candidate-local indices v in [0, N_b).  Registers are never candidates and
 * are never listed; the caller keeps them (the paper's "union {r}").
 *
 * Ownership.  Every pointer argument is DEVICE memory owned by the caller,
 * except `const occam_problem *` and `const occam_rows *`, which are host
 * structs read during the call only.  The library allocates no memory; calls on
 * different streams may overlap when their output and workspace buffers are
 * distinct.  Its only global state is the built-in workspace of
 * occam_prune_noalloc (one static device array per GPU) and the per-device
 * addresses of that array, looked up once.
 *
 * Errors.  Arguments are validated on the host before anything is enqueued:
 * OCCAM_ERR_INVALID_ARG, OCCAM_ERR_UNSUPPORTED and OCCAM_ERR_WORKSPACE mean
 * nothing was launched and the outputs are untouched.  OCCAM_ERR_HIP means the
 * HIP runtime rejected a launch; kernels of the same call enqueued before it
 * may already run, so the outputs are then undefined.  Calls are
 * asynchronous: kernel faults surface at the caller's next synchronisation of
 * `stream`.  Inputs must be finite.  Device-side offsets must be
 * non-decreasing with 1 <= T_b <= max_rows and 0 <= N_b <= max_cands.
 * Batches are limited to B <= 65535 (OCCAM_ERR_UNSUPPORTED beyond).
 *
 * Precision.  Logits and probabilities are computed in float32 from float32
 * or bfloat16 inputs; bfloat16 products are exact in float32.
 *
 * Kernel coverage (anything else returns OCCAM_ERR_UNSUPPORTED):
 *   one anchor row (rows == 1, or max_rows == 1): f32 or bf16, H <= 64, any d
 *     that keeps a key head a whole number of 16-byte chunks, H*d small enough
 *     for the query to sit in 64 KB of LDS with its partial sums;
 *   several anchor rows: bf16 only (the MFMA path), d <= 128.
 */
#ifndef OCCAM_H
#define OCCAM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OCCAM_VERSION 2
#define OCCAM_MAX_ROW_TENSORS 8

typedef enum {
    OCCAM_OK = 0,
    OCCAM_ERR_INVALID_ARG = 1, /* a null/misaligned pointer or an impossible shape   */
    OCCAM_ERR_UNSUPPORTED = 2, /* a valid shape the library has no kernel for        */
    OCCAM_ERR_WORKSPACE = 3,   /* ws_bytes < occam_workspace_size(problem)          */
    OCCAM_ERR_HIP = 4          /* a kernel launch was rejected by the HIP runtime    */
} occam_status;

typedef enum { OCCAM_F32 = 0, OCCAM_BF16 = 1 } occam_dtype;

/* How the R register scores are combined into s(r).  The paper builds one
 * register (Appendix, "Parameter settings"); with several, MEAN is the default
 * reading and equals the paper's rule at R = 1.  CAND_MEAN replaces s(r) by the
 * mean score of the sample's visual tokens (0 when it has none): the mean-based
 * threshold of the component ablation (Appendix, Table
 * tab:qwen_compact_component_ablation). */
typedef enum {
    OCCAM_REG_MEAN = 0,
    OCCAM_REG_MAX = 1,
    OCCAM_REG_SUM = 2,
    OCCAM_REF_CAND_MEAN = 3
} occam_reg_reduce;

/* How a visual key's score is reduced over the anchor rows (registers always take
 * the mean).  MAX: the text rows of Stage II (Sec. 3.5, Eq. text_scoring).  MEAN:
 * the mutual-scoring Stage I for encoders without a CLS token (Sec. 3.4,
 * Eq. mutual_scoring; Appendix Eq. stage1_mutual_appendix), where the anchor rows
 * are the register and visual tokens themselves and every key is scored by the
 * attention it receives on average.  With one anchor row both are the same. */
typedef enum { OCCAM_ROWS_MAX = 0, OCCAM_ROWS_MEAN = 1 } occam_row_reduce;

typedef struct {
    int32_t batch;          /* B >= 1                                                */
    int32_t num_heads;      /* H >= 1                                                */
    int32_t num_kv_heads;   /* Hkv >= 1, H % Hkv == 0                                */
    int32_t head_dim;       /* d: multiple of 8 (bf16) or 4 (f32), <= 256            */
    int32_t num_registers;  /* R in [1, 32]                                          */
    int32_t rows;           /* T when q_offsets == NULL (>= 1)                       */
    int32_t cands;          /* N when key_offsets == NULL (>= 0)                     */
    const int32_t *q_offsets;   /* device [B+1] prefix of T_b, or NULL (uniform)     */
    const int32_t *key_offsets; /* device [B+1] prefix of R + N_b, or NULL (uniform) */
    int32_t max_rows;       /* upper bound of T_b when q_offsets != NULL             */
    int32_t max_cands;      /* upper bound of N_b when key_offsets != NULL           */
    int32_t dtype;          /* occam_dtype of q and k                                */
    float softmax_scale;    /* 0 => 1/sqrt(d), the scale of Eq. (1)                  */
    int32_t visual_row_reduce; /* occam_row_reduce; 0 (MAX) when zero-initialised    */
} occam_problem;
/* The two offset arrays are independent: ragged key counts with the same row count in
 * every sample (q_offsets NULL, key_offsets set) is a valid problem, and with T a
 * multiple of 128 it lets the text-row scoring use its full-row-block form. */

/* One row tensor gathered with the survivors (occam_gather / occam_prune).
 * The source row of visual token v of sample b is
 *     co_b + b * src_pad_rows + src_row0 + v
 * i.e. each sample owns N_b + src_pad_rows consecutive rows, of which the
 * visual ones start at src_row0 (a hidden-state tensor of visual tokens only:
 * pad 0, row0 0; the key/value rows of [registers ; visual]: pad R, row0 R).
 * The destination row of survivor i of sample b is kept_offsets[b] + i.
 * src/dst and both strides must be multiples of 4 bytes, row_bytes of 4;
 * 16-byte multiples take the vector path. */
typedef struct {
    const void *src;
    void *dst;
    int64_t src_pad_rows;
    int64_t src_row0;
    int64_t src_row_stride_bytes;
    int64_t dst_row_stride_bytes;
    int64_t row_bytes;
} occam_rows;

/* Human-readable name of a status code (static storage). */
const char *occam_status_string(occam_status status);

/* OCCAM_VERSION of the built library. */
int32_t occam_version(void);

/* Bytes of device workspace that every call below may use for this problem
 * (0 for an invalid problem).  The workspace needs no initialisation and
 * holds nothing between calls. */
size_t occam_workspace_size(const occam_problem *problem);

/* Steps 1-2 (Eq. (1); Eq. EQ:CLS; Eq. text_scoring; Eq. mutual_scoring).  For
 * every sample, every anchor row t and head h, the softmax over the R + N_b keys
 * of scale * <q[t,h], k[s, h/(H/Hkv)]> is averaged over heads; the score of a
 * visual key is the max (visual_row_reduce MAX) or the mean (MEAN) of that
 * average over the T_b rows, the score of a register the mean over the rows
 * (T_b = 1: the CLS row itself).
 * row_lse (nullable): the natural-log softmax normaliser of each (row, head)
 * over a larger key set (e.g. the LLM's full causal prefix); when given,
 * probabilities are exp(logit - row_lse) instead of the softmax over the keys
 * given.  Writes scores[sum_b (R + N_b)]. */
occam_status occam_score(const occam_problem *problem, const void *q, const void *k,
                         const float *row_lse, float *scores,
                         void *workspace, size_t ws_bytes, hipStream_t stream);

/* Step 3 (Eqs. stage1_threshold_appendix, stage2_set_appendix):
 * tau[b] = lambda * reduce(scores[ko_b + 0 .. ko_b + R)), lambda finite >= 0. */
occam_status occam_threshold(const occam_problem *problem, const float *scores,
                             float lambda, int32_t reduce, float *tau, hipStream_t stream);

/* Steps 4-5 (Eq. stage1 / Eq. stage2): keep visual token v of sample b iff
 * scores[ko_b + R + v] >= tau[b]; write the survivors ascending and packed,
 * kept_count[B] and kept_offsets[B+1] (exclusive prefix of the counts).
 * index_map (nullable, [sum N_b]): write index_map[co_b + v] instead of v,
 * which chains Stage II onto Stage I's original token indices.
 * kept_idx must hold sum_b N_b entries (the worst case). */
occam_status occam_select(const occam_problem *problem, const float *scores, const float *tau,
                          const int32_t *index_map, int32_t *kept_idx, int32_t *kept_count,
                          int32_t *kept_offsets, void *workspace, size_t ws_bytes,
                          hipStream_t stream);

/* Fixed-budget variant of steps 4-5 (the component ablation, Appendix Table
 * tab:qwen_compact_component_ablation): keep the min(k_keep, N_b) visual tokens
 * of each sample with the largest scores; among equal scores the lower index
 * ranks first, so the kept set is unique.  Output exactly as occam_select
 * (ascending, packed, counts, offsets, index_map).  k_keep >= 0. */
occam_status occam_select_topk(const occam_problem *problem, const float *scores,
                               int32_t k_keep, const int32_t *index_map, int32_t *kept_idx,
                               int32_t *kept_count, int32_t *kept_offsets, void *workspace,
                               size_t ws_bytes, hipStream_t stream);

/* Step 5, materialisation (Algorithm 1, the pruned sequence): for each of
 * the n row tensors, copy the row of every listed survivor, byte for byte, to
 * the packed destination.  kept_idx values are read as candidate-local v. */
occam_status occam_gather(const occam_problem *problem, int32_t n, const occam_rows *tensors,
                          const int32_t *kept_idx, const int32_t *kept_offsets,
                          hipStream_t stream);

/* Steps 1-5 fused on `stream` without host synchronisation: scores, tau,
 * survivors and the gather of n row tensors (n may be 0).  scores may be NULL
 * (kept in the workspace).  With index_map the emitted kept_idx values are
 * remapped as in occam_select while the gather still reads local rows v. */
occam_status occam_prune(const occam_problem *problem, const void *q, const void *k,
                         const float *row_lse, float lambda, int32_t reduce,
                         const int32_t *index_map, int32_t n, const occam_rows *tensors,
                         float *scores, float *tau, int32_t *kept_idx, int32_t *kept_count,
                         int32_t *kept_offsets, void *workspace, size_t ws_bytes,
                         hipStream_t stream);

/* occam_prune without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc).  It runs exactly the kernels of occam_prune, with the
 * workspace taken from a static device array built into the library: 32 MiB per
 * GPU, held from the library's first use on that GPU until the process ends.
 * A problem whose occam_workspace_size exceeds 32 MiB returns
 * OCCAM_ERR_WORKSPACE (use occam_prune with a workspace of its own).  The
 * array's device address is looked up once per device, on the first call whose
 * stream belongs to that device (OCCAM_ERR_HIP if the lookup fails).  The call
 * allocates nothing.  Every call on one GPU shares that GPU's array, so calls
 * that overlap on one GPU (different streams, or different host threads)
 * race; calls ordered on one stream do not.  The array needs no clearing: every
 * call writes what it reads. */
occam_status occam_prune_noalloc(const occam_problem *problem, const void *q, const void *k,
                                 const float *row_lse, float lambda, int32_t reduce,
                                 const int32_t *index_map, int32_t n,
                                 const occam_rows *tensors, float *scores, float *tau,
                                 int32_t *kept_idx, int32_t *kept_count, int32_t *kept_offsets,
                                 hipStream_t stream);

/* Budget matching (Appendix Eq. lambda2_budget_matching_appendix) over the batch
 * as the calibration set: the mean kept count (1/B) sum_b |{v : s_b(v) >= lambda *
 * s_b(r)}| is a step function of lambda that changes at the ratios s_b(v) / s_b(r)
 * (s_b(r) reduced from the register scores as in occam_threshold).  Among its
 * levels the one closest to k_target wins (ties: the smaller count, i.e. the
 * larger lambda) and lambda[0] receives the geometric midpoint of that level's
 * interval (the level's ratio and the next smaller distinct ratio; half the ratio
 * if there is no positive one), so that rounding lambda cannot move the count.
 * scores: device f32 in the layout occam_score writes.  lambda, mean_kept
 * (nullable): one device f32 each; mean_kept[0] receives the matched mean count.
 * A batch without candidates gives lambda 1.  Ratios are formed in float32; every
 * s_b(r) must be positive.  k_target finite >= 0.  The count is of visual
 * survivors only: the R registers, which every sample keeps whatever lambda is
 * (the union with {r} in Eqs. stage1 and stage2), are not counted, so a target
 * that includes them is k_target + R.  The selection state lives in the
 * workspace of the problem and is cleared by each call, so calls that share a
 * workspace must be ordered on one stream. */
occam_status occam_match_lambda(const occam_problem *problem, const float *scores,
                                int32_t reduce, float k_target, float *lambda,
                                float *mean_kept, void *workspace, size_t ws_bytes,
                                hipStream_t stream);

/* Test-time register construction (Algorithm 1, "redirect sinks to r"; Appendix
 * Eq. register_redirect_appendix), applied to an MLP activation tensor of the
 * vision encoder before Stage I.  For every sample b and every listed channel k:
 *     h[register row, k] = max over the sample's visual rows of h[v, k]
 *     h[v, k]            = 0 for every visual row v,
 * in place.  Rows follow the key layout of the problem: sample b owns rows
 * ko_b .. ko_b + R + N_b - 1 (R register rows first), each `width` elements of
 * `problem->dtype` (F32 or BF16) with `row_stride_bytes` between rows; only the
 * register row reg_slot (in [0, R)) receives the maxima.  A sample without visual
 * rows (N_b = 0) is left unchanged.  channels: device int32 [n_channels]
 * (n_channels in [0, 1024]); an index outside [0, width) is ignored and a repeated
 * index acts once.  The anchor-row fields of the problem are not used. */
occam_status occam_register_redirect(const occam_problem *problem, void *h, int32_t width,
                                     int64_t row_stride_bytes, const int32_t *channels,
                                     int32_t n_channels, int32_t reg_slot,
                                     hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* OCCAM_H */
