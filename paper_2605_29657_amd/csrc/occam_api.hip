// Host entry points of liboccam: argument validation, workspace layout and
// kernel launches for the C ABI declared in include/occam.h.  Validation runs
// before any HIP call, so an invalid call enqueues nothing.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>

#include "occam.h"
#include "occam_internal.hpp"

using namespace occam;

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

struct Plan {
    Prob p;
    int bf16;
    int text;          // 1: several anchor rows (MFMA path); 0: one anchor row (VALU path)
    int kpw;           // keys per workgroup of the one-row path
    int nchunks;       // key chunks per sample of the one-row path
    size_t off_logits, off_stats, off_lse2, off_part, off_done, off_clist, off_ccnt, off_scores,
        off_tau, off_slot, off_match, total;
};

bool aligned(const void* ptr, size_t a) { return (reinterpret_cast<uintptr_t>(ptr) % a) == 0; }

occam_status make_plan(const occam_problem* pr, Plan* pl) {
    if (!pr) return OCCAM_ERR_INVALID_ARG;
    const occam_problem& x = *pr;
    if (x.batch < 1 || x.num_heads < 1 || x.num_kv_heads < 1 ||
        x.num_heads % x.num_kv_heads != 0 || x.head_dim < 1 || x.head_dim > 256 ||
        x.num_registers < 1 || x.num_registers > 32)
        return OCCAM_ERR_INVALID_ARG;
    if (x.dtype != OCCAM_F32 && x.dtype != OCCAM_BF16) return OCCAM_ERR_INVALID_ARG;
    if (!(x.softmax_scale >= 0.f) || isinf(x.softmax_scale)) return OCCAM_ERR_INVALID_ARG;
    if (x.visual_row_reduce != OCCAM_ROWS_MAX && x.visual_row_reduce != OCCAM_ROWS_MEAN)
        return OCCAM_ERR_INVALID_ARG;
    const int max_rows = x.q_offsets ? x.max_rows : x.rows;
    const int max_cands = x.key_offsets ? x.max_cands : x.cands;
    if (max_rows < 1 || max_cands < 0) return OCCAM_ERR_INVALID_ARG;
    if (x.q_offsets && !aligned(x.q_offsets, 4)) return OCCAM_ERR_INVALID_ARG;
    if (x.key_offsets && !aligned(x.key_offsets, 4)) return OCCAM_ERR_INVALID_ARG;
    const int bf16 = x.dtype == OCCAM_BF16;
    const int H = x.num_heads, d = x.head_dim, R = x.num_registers, B = x.batch;
    // Index arithmetic is 32-bit for counts and rows: keep every extent below 2^31.
    const long long keys_cap = (long long)B * (R + (long long)max_cands);
    const long long rows_cap = (long long)B * max_rows;
    if (keys_cap * H >= (1LL << 31) || rows_cap * H >= (1LL << 31)) return OCCAM_ERR_UNSUPPORTED;
    // Several kernels put the sample index in grid.y, whose extent is at most 65535.
    if (B > kMaxGridY) return OCCAM_ERR_UNSUPPORTED;
    if (d % (bf16 ? 8 : 4) != 0) return OCCAM_ERR_UNSUPPORTED;

    Plan P;
    memset(&P, 0, sizeof P);
    P.p.B = B; P.p.H = H; P.p.Hkv = x.num_kv_heads; P.p.d = d; P.p.R = R;
    P.p.rows = x.rows; P.p.cands = x.cands;
    P.p.q_off = x.q_offsets; P.p.k_off = x.key_offsets;
    P.p.max_rows = max_rows; P.p.max_cands = max_cands;
    P.p.scale = x.softmax_scale > 0.f ? x.softmax_scale : 1.0f / sqrtf((float)d);
    P.p.mean_rows = x.visual_row_reduce == OCCAM_ROWS_MEAN;
    P.bf16 = bf16;
    P.text = max_rows > 1;
    size_t off = 0;
    if (P.text) {
        if (!bf16 || d > 128) return OCCAM_ERR_UNSUPPORTED;
        // The scoring kernel addresses a sample's rows and keys with 32-bit byte offsets.
        if ((long long)max_rows * H * d * 2 >= (1LL << 32) ||
            (R + (long long)max_cands) * x.num_kv_heads * d * 2 >= (1LL << 32))
            return OCCAM_ERR_UNSUPPORTED;
        if (text_score_smem(H, ((d + 15) / 16) * 16) > kScoreSmemMax) return OCCAM_ERR_UNSUPPORTED;
        const size_t nrb = (max_rows + kTxtRows - 1) / kTxtRows;
        // The statistics pass of a small batch splits every task's keys into ranges, each
        // with its own normaliser table (the scoring pass merges them); not for mutual scoring.
        const int rbw = stats_row_blocks((int)nrb);
        P.p.lse_splits = P.p.mean_rows ? 1 : stats_splits((long long)B * H * ((nrb + rbw - 1) / rbw),
                                                           R + (long long)max_cands);
        P.p.lse_stride = rows_cap * H;
        P.off_lse2 = off;
        off = align_up(off + (size_t)P.p.lse_splits * rows_cap * H * sizeof(float));
        P.off_part = off;
        if (P.p.mean_rows) {
            // Column sums of mutual scoring, per (sample, 128-row block, head, key).
            off = align_up(off + (size_t)B * nrb * H * (R + (size_t)max_cands) * sizeof(float));
        } else if (nrb > 1) {
            // Row maxima / sums of the max form, per (sample, 128-row block, key).
            off = align_up(off + (size_t)B * nrb * (R + (size_t)max_cands) * sizeof(float));
        }
    } else {
        P.kpw = cls_keys_per_wg(H, x.num_kv_heads, d, bf16 ? 2 : 4, B, R + (long long)max_cands);
        const int NC = d / (bf16 ? 8 : 4);
        const size_t smem = sizeof(float) * ((size_t)H * d + (size_t)NC * x.num_kv_heads +
                                             (size_t)P.kpw * H * NC + (size_t)P.kpw * H +
                                             2 * (size_t)kClsThreads);
        if (H > 64) return OCCAM_ERR_UNSUPPORTED;
        if (!cls_stream_nc(H, x.num_kv_heads, d, bf16 ? 2 : 4) && smem > 65536)
            return OCCAM_ERR_UNSUPPORTED;
        const long long nchunks = (R + (long long)max_cands + P.kpw - 1) / P.kpw;
        P.nchunks = nchunks > (1LL << 30) ? (1 << 30) : (int)nchunks;
        P.off_logits = off; off = align_up(off + (size_t)keys_cap * H * sizeof(float));
        P.off_stats = off; off = align_up(off + (size_t)B * nchunks * H * sizeof(float2));
        if (nchunks <= kMaxChunkLists) {
            // Per-chunk survivor lists and counts of the in-kernel threshold + compaction.
            P.off_clist = off; off = align_up(off + (size_t)B * nchunks * P.kpw * sizeof(int));
            P.off_ccnt = off; off = align_up(off + (size_t)B * nchunks * sizeof(int));
        }
    }
    // Finished workgroups per sample (the in-kernel threshold / compaction epilogue).
    P.off_done = off; off = align_up(off + (size_t)B * sizeof(unsigned));
    P.off_scores = off; off = align_up(off + (size_t)keys_cap * sizeof(float));
    P.off_tau = off; off = align_up(off + (size_t)B * sizeof(float));
    P.off_slot = off; off = align_up(off + (size_t)B * max_cands * sizeof(int));
    P.off_match = off; off = align_up(off + kMatchStateBytes);
    P.total = off;
    *pl = P;
    return OCCAM_OK;
}

template <typename T>
T* ws_at(void* ws, size_t off) { return reinterpret_cast<T*>(static_cast<char*>(ws) + off); }

occam_status check_ws(const Plan& P, void* ws, size_t ws_bytes) {
    if (ws_bytes < P.total) return OCCAM_ERR_WORKSPACE;
    if (!ws || !aligned(ws, kAlign)) return OCCAM_ERR_INVALID_ARG;
    return OCCAM_OK;
}

bool lambda_ok(float lambda) { return lambda >= 0.f && !isinf(lambda); }
bool reduce_ok(int32_t r) {
    return r == OCCAM_REG_MEAN || r == OCCAM_REG_MAX || r == OCCAM_REG_SUM ||
           r == OCCAM_REF_CAND_MEAN;
}

occam_status rows_from(int32_t n, const occam_rows* t, RowTensors* out) {
    memset(out, 0, sizeof *out);
    if (n < 0 || n > OCCAM_MAX_ROW_TENSORS) return OCCAM_ERR_INVALID_ARG;
    if (n > 0 && !t) return OCCAM_ERR_INVALID_ARG;
    int vec = 1;
    for (int i = 0; i < n; ++i) {
        const occam_rows& r = t[i];
        if (!r.src || !r.dst || r.row_bytes < 0 || r.src_pad_rows < 0 || r.src_row0 < 0 ||
            r.src_row_stride_bytes < r.row_bytes || r.dst_row_stride_bytes < r.row_bytes)
            return OCCAM_ERR_INVALID_ARG;
        if (r.row_bytes % 4 || r.src_row_stride_bytes % 4 || r.dst_row_stride_bytes % 4 ||
            !aligned(r.src, 4) || !aligned(r.dst, 4))
            return OCCAM_ERR_INVALID_ARG;
        if (r.row_bytes % 16 || r.src_row_stride_bytes % 16 || r.dst_row_stride_bytes % 16 ||
            !aligned(r.src, 16) || !aligned(r.dst, 16))
            vec = 0;
        RowTensor& o = out->t[i];
        o.src = static_cast<const char*>(r.src);
        o.dst = static_cast<char*>(r.dst);
        o.src_pad_rows = r.src_pad_rows;
        o.src_row0 = r.src_row0;
        o.src_stride = r.src_row_stride_bytes;
        o.dst_stride = r.dst_row_stride_bytes;
        o.row_bytes = r.row_bytes;
    }
    out->n = n;
    out->vec16 = vec;
    return OCCAM_OK;
}

inline occam_status hip_ok(hipError_t e) { return e == hipSuccess ? OCCAM_OK : OCCAM_ERR_HIP; }

// Steps 1-2 into `scores` (device), both paths.  With `sel` (occam_prune) the threshold and
// the compaction are applied as well, inside the scoring kernel, wherever the call has a
// kernel before it that clears the per-sample counters (the one-row logits; the text-row
// statistics, i.e. no caller normaliser): then *selected is set.  The multi-row max form
// then also combines its row blocks in the scoring kernel.
occam_status run_score(const Plan& P, const void* q, const void* k, const float* row_lse,
                       float* scores, void* ws, hipStream_t s, const Finish* sel = nullptr,
                       int* selected = nullptr, ChunkLists* lists = nullptr) {
    Finish fin{};
    if (selected) *selected = 0;
    if (P.text) {
        // Text rows: the sample's last scoring workgroup combines the row blocks and, when
        // the copy of the sample's scores fits in the kernel's LDS, selects.  The counters
        // are cleared by the statistics kernel, so not with a caller normaliser.
        const bool counters = !row_lse && !P.p.mean_rows;
        const bool combine = P.p.max_rows > kTxtRows;
        const size_t need = 128 + select_lds_bytes(P.p.R, P.p.max_cands);
        const bool do_select = sel && need <= text_score_smem(P.p.H, ((P.p.d + 15) / 16) * 16);
        if (counters && (do_select || combine)) {
            if (sel) fin = *sel;
            fin.done = ws_at<unsigned>(ws, P.off_done);
            fin.select = do_select ? 1 : 0;
            if (selected) *selected = fin.select;
        }
    } else if (sel && sel->reduce != kRefCandMean && P.nchunks <= kMaxChunkLists &&
               P.kpw <= kClsThreads) {
        // One row: every scoring workgroup thresholds and compacts its own chunk (the
        // candidate mean needs every score first, so it keeps the separate select).
        fin = *sel;
        fin.select = 1;
        fin.chunk_slot = ws_at<int>(ws, P.off_clist);
        fin.chunk_cnt = ws_at<int>(ws, P.off_ccnt);
        if (selected) *selected = 1;
        if (lists) *lists = ChunkLists{fin.chunk_slot, fin.chunk_cnt, P.nchunks, P.kpw};
    }
    if (P.text) {
        const float* lse = row_lse;
        if (!row_lse) {
            float* lse2 = ws_at<float>(ws, P.off_lse2);
            occam_status st = hip_ok(launch_text_stats(P.p, q, k, lse2, fin, s));
            if (st != OCCAM_OK) return st;
            lse = lse2;
        }
        const int natural = row_lse ? 1 : 0;
        float* part = ws_at<float>(ws, P.off_part);
        if (P.p.mean_rows) return hip_ok(launch_text_colsum(P.p, q, k, lse, natural, part, scores, s));
        return hip_ok(launch_text_score(P.p, q, k, lse, natural, scores, part, fin, s));
    }
    float* logits = ws_at<float>(ws, P.off_logits);
    float2* stats = ws_at<float2>(ws, P.off_stats);
    occam_status st = hip_ok(launch_cls_logits(P.p, P.bf16, q, k, logits, stats, P.kpw, fin, s));
    if (st != OCCAM_OK) return st;
    return hip_ok(launch_cls_scores(P.p, P.bf16, logits, stats, row_lse, scores, P.kpw, fin, s));
}

// The key layout of a problem alone (register construction reads no anchor rows).
occam_status key_layout(const occam_problem* pr, Prob* out, int* bf16) {
    if (!pr) return OCCAM_ERR_INVALID_ARG;
    const occam_problem& x = *pr;
    if (x.batch < 1 || x.num_registers < 1 || x.num_registers > 32) return OCCAM_ERR_INVALID_ARG;
    if (x.dtype != OCCAM_F32 && x.dtype != OCCAM_BF16) return OCCAM_ERR_INVALID_ARG;
    const int max_cands = x.key_offsets ? x.max_cands : x.cands;
    if (max_cands < 0) return OCCAM_ERR_INVALID_ARG;
    if (x.key_offsets && !aligned(x.key_offsets, 4)) return OCCAM_ERR_INVALID_ARG;
    if ((long long)x.batch * (x.num_registers + (long long)max_cands) >= (1LL << 31) ||
        x.batch > kMaxGridY)
        return OCCAM_ERR_UNSUPPORTED;
    Prob p;
    memset(&p, 0, sizeof p);
    p.B = x.batch; p.R = x.num_registers; p.cands = x.cands; p.k_off = x.key_offsets;
    p.max_cands = max_cands; p.rows = 1; p.max_rows = 1;
    *out = p;
    *bf16 = x.dtype == OCCAM_BF16;
    return OCCAM_OK;
}

// Argument checks of occam_prune (and its allocation-free variant) before any HIP call.
occam_status prune_args(const occam_problem* problem, const void* q, const void* k,
                        const float* row_lse, float lambda, int32_t reduce,
                        const int32_t* index_map, int32_t n, const occam_rows* tensors,
                        const float* scores, const float* tau, const int32_t* kept_idx,
                        const int32_t* kept_count, const int32_t* kept_offsets, Plan* P,
                        RowTensors* rows) {
    occam_status st = make_plan(problem, P);
    if (st != OCCAM_OK) return st;
    if (!q || !k || !kept_idx || !kept_count || !kept_offsets || !aligned(q, 16) ||
        !aligned(k, 16) || !aligned(kept_idx, 4) || !aligned(kept_count, 4) ||
        !aligned(kept_offsets, 4) || (scores && !aligned(scores, 4)) || (tau && !aligned(tau, 4)) ||
        (row_lse && !aligned(row_lse, 4)) || (index_map && !aligned(index_map, 4)) ||
        !lambda_ok(lambda) || !reduce_ok(reduce))
        return OCCAM_ERR_INVALID_ARG;
    return rows_from(n, tensors, rows);
}

// Steps 1-5 on a validated plan and a workspace of at least P.total bytes.
occam_status run_prune(const Plan& P, const void* q, const void* k, const float* row_lse,
                       float lambda, int32_t reduce, const int32_t* index_map,
                       const RowTensors& rows, float* scores, float* tau, int32_t* kept_idx,
                       int32_t* kept_count, int32_t* kept_offsets, void* workspace,
                       hipStream_t stream) {
    occam_status st;
    float* sc = scores ? scores : ws_at<float>(workspace, P.off_scores);
    float* tu = tau ? tau : ws_at<float>(workspace, P.off_tau);
    int* slot = ws_at<int>(workspace, P.off_slot);
    Finish sel{};
    sel.lambda = lambda;
    sel.reduce = reduce;
    sel.tau = tu;
    sel.slot = slot;
    sel.count = kept_count;
    int selected = 0;
    ChunkLists lists{};
    if ((st = run_score(P, q, k, row_lse, sc, workspace, stream, &sel, &selected, &lists)) !=
        OCCAM_OK)
        return st;
    if (!selected) {
        st = hip_ok(launch_select(P.p, sc, nullptr, 1, lambda, reduce, tu, slot, kept_count, stream));
        if (st != OCCAM_OK) return st;
    }
    return hip_ok(launch_pack_gather(P.p, slot, kept_count, index_map, kept_idx, kept_offsets,
                                     nullptr, nullptr, rows, stream, lists));
}

// ---------------------------------------------------------------------------
// Built-in workspace of occam_prune_noalloc, for callers that cannot allocate device
// memory.  The loader gives every GPU that runs this library its own copy of the array
// (held until the process ends).  In host code `scratch` names a host-side stand-in, not
// device memory: only the address that hipGetSymbolAddress returns for the device,
// looked up once per device and kept in scratch_ptr, is ever handed to a kernel.
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
std::atomic<void*> scratch_ptr[kMaxDevices];

// The device address of `scratch` on the device that `stream` belongs to, or null.
void* scratch_for(hipStream_t stream) {
    int dev = -1;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return nullptr;
    void* ptr = scratch_ptr[dev].load(std::memory_order_acquire);
    if (ptr) return ptr;
    std::lock_guard<std::mutex> lock(scratch_mu);
    ptr = scratch_ptr[dev].load(std::memory_order_acquire);
    if (ptr) return ptr;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return nullptr;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !ptr || !aligned(ptr, kAlign)) return nullptr;
    scratch_ptr[dev].store(ptr, std::memory_order_release);
    return ptr;
}

}  // namespace

extern "C" {

const char* occam_status_string(occam_status status) {
    switch (status) {
        case OCCAM_OK: return "OCCAM_OK";
        case OCCAM_ERR_INVALID_ARG: return "OCCAM_ERR_INVALID_ARG: invalid argument";
        case OCCAM_ERR_UNSUPPORTED: return "OCCAM_ERR_UNSUPPORTED: shape or type not supported";
        case OCCAM_ERR_WORKSPACE: return "OCCAM_ERR_WORKSPACE: workspace too small";
        case OCCAM_ERR_HIP: return "OCCAM_ERR_HIP: HIP runtime error";
    }
    return "unknown occam_status";
}

int32_t occam_version(void) { return OCCAM_VERSION; }

size_t occam_workspace_size(const occam_problem* problem) {
    Plan P;
    if (make_plan(problem, &P) != OCCAM_OK) return 0;
    return P.total;
}

occam_status occam_score(const occam_problem* problem, const void* q, const void* k,
                         const float* row_lse, float* scores, void* workspace, size_t ws_bytes,
                         hipStream_t stream) {
    Plan P;
    occam_status st = make_plan(problem, &P);
    if (st != OCCAM_OK) return st;
    if (!q || !k || !scores || !aligned(q, 16) || !aligned(k, 16) || !aligned(scores, 4) ||
        (row_lse && !aligned(row_lse, 4)))
        return OCCAM_ERR_INVALID_ARG;
    if ((st = check_ws(P, workspace, ws_bytes)) != OCCAM_OK) return st;
    return run_score(P, q, k, row_lse, scores, workspace, stream);
}

occam_status occam_threshold(const occam_problem* problem, const float* scores, float lambda,
                             int32_t reduce, float* tau, hipStream_t stream) {
    Plan P;
    occam_status st = make_plan(problem, &P);
    if (st != OCCAM_OK) return st;
    if (!scores || !tau || !aligned(scores, 4) || !aligned(tau, 4) || !lambda_ok(lambda) ||
        !reduce_ok(reduce))
        return OCCAM_ERR_INVALID_ARG;
    return hip_ok(launch_threshold(P.p, scores, lambda, reduce, tau, stream));
}

occam_status occam_select(const occam_problem* problem, const float* scores, const float* tau,
                          const int32_t* index_map, int32_t* kept_idx, int32_t* kept_count,
                          int32_t* kept_offsets, void* workspace, size_t ws_bytes,
                          hipStream_t stream) {
    Plan P;
    occam_status st = make_plan(problem, &P);
    if (st != OCCAM_OK) return st;
    if (!scores || !tau || !kept_idx || !kept_count || !kept_offsets || !aligned(scores, 4) ||
        !aligned(tau, 4) || !aligned(kept_idx, 4) || !aligned(kept_count, 4) ||
        !aligned(kept_offsets, 4) || (index_map && !aligned(index_map, 4)))
        return OCCAM_ERR_INVALID_ARG;
    if ((st = check_ws(P, workspace, ws_bytes)) != OCCAM_OK) return st;
    int* slot = ws_at<int>(workspace, P.off_slot);
    st = hip_ok(launch_select(P.p, scores, tau, 0, 0.f, 0, nullptr, slot, kept_count, stream));
    if (st != OCCAM_OK) return st;
    RowTensors none;
    memset(&none, 0, sizeof none);
    return hip_ok(launch_pack_gather(P.p, slot, kept_count, index_map, kept_idx, kept_offsets,
                                     nullptr, nullptr, none, stream));
}

occam_status occam_select_topk(const occam_problem* problem, const float* scores, int32_t k_keep,
                               const int32_t* index_map, int32_t* kept_idx, int32_t* kept_count,
                               int32_t* kept_offsets, void* workspace, size_t ws_bytes,
                               hipStream_t stream) {
    Plan P;
    occam_status st = make_plan(problem, &P);
    if (st != OCCAM_OK) return st;
    if (!scores || !kept_idx || !kept_count || !kept_offsets || !aligned(scores, 4) ||
        !aligned(kept_idx, 4) || !aligned(kept_count, 4) || !aligned(kept_offsets, 4) ||
        (index_map && !aligned(index_map, 4)) || k_keep < 0)
        return OCCAM_ERR_INVALID_ARG;
    if ((st = check_ws(P, workspace, ws_bytes)) != OCCAM_OK) return st;
    int* slot = ws_at<int>(workspace, P.off_slot);
    st = hip_ok(launch_select_topk(P.p, scores, k_keep, slot, kept_count, stream));
    if (st != OCCAM_OK) return st;
    RowTensors none;
    memset(&none, 0, sizeof none);
    return hip_ok(launch_pack_gather(P.p, slot, kept_count, index_map, kept_idx, kept_offsets,
                                     nullptr, nullptr, none, stream));
}

occam_status occam_gather(const occam_problem* problem, int32_t n, const occam_rows* tensors,
                          const int32_t* kept_idx, const int32_t* kept_offsets,
                          hipStream_t stream) {
    Plan P;
    occam_status st = make_plan(problem, &P);
    if (st != OCCAM_OK) return st;
    RowTensors rows;
    if ((st = rows_from(n, tensors, &rows)) != OCCAM_OK) return st;
    if (!kept_idx || !kept_offsets || !aligned(kept_idx, 4) || !aligned(kept_offsets, 4))
        return OCCAM_ERR_INVALID_ARG;
    if (n == 0) return OCCAM_OK;
    return hip_ok(launch_pack_gather(P.p, nullptr, nullptr, nullptr, nullptr, nullptr, kept_idx,
                                     kept_offsets, rows, stream));
}

occam_status occam_prune(const occam_problem* problem, const void* q, const void* k,
                         const float* row_lse, float lambda, int32_t reduce,
                         const int32_t* index_map, int32_t n, const occam_rows* tensors,
                         float* scores, float* tau, int32_t* kept_idx, int32_t* kept_count,
                         int32_t* kept_offsets, void* workspace, size_t ws_bytes,
                         hipStream_t stream) {
    Plan P;
    RowTensors rows;
    occam_status st = prune_args(problem, q, k, row_lse, lambda, reduce, index_map, n, tensors,
                                 scores, tau, kept_idx, kept_count, kept_offsets, &P, &rows);
    if (st != OCCAM_OK) return st;
    if ((st = check_ws(P, workspace, ws_bytes)) != OCCAM_OK) return st;
    return run_prune(P, q, k, row_lse, lambda, reduce, index_map, rows, scores, tau, kept_idx,
                     kept_count, kept_offsets, workspace, stream);
}

occam_status occam_prune_noalloc(const occam_problem* problem, const void* q, const void* k,
                                 const float* row_lse, float lambda, int32_t reduce,
                                 const int32_t* index_map, int32_t n,
                                 const occam_rows* tensors, float* scores, float* tau,
                                 int32_t* kept_idx, int32_t* kept_count, int32_t* kept_offsets,
                                 hipStream_t stream) {
    Plan P;
    RowTensors rows;
    occam_status st = prune_args(problem, q, k, row_lse, lambda, reduce, index_map, n, tensors,
                                 scores, tau, kept_idx, kept_count, kept_offsets, &P, &rows);
    if (st != OCCAM_OK) return st;
    if (P.total > kScratchBytes) return OCCAM_ERR_WORKSPACE;
    void* ws = scratch_for(stream);
    if (!ws) return OCCAM_ERR_HIP;
    return run_prune(P, q, k, row_lse, lambda, reduce, index_map, rows, scores, tau, kept_idx,
                     kept_count, kept_offsets, ws, stream);
}

occam_status occam_match_lambda(const occam_problem* problem, const float* scores, int32_t reduce,
                                float k_target, float* lambda, float* mean_kept, void* workspace,
                                size_t ws_bytes, hipStream_t stream) {
    Plan P;
    occam_status st = make_plan(problem, &P);
    if (st != OCCAM_OK) return st;
    if (!scores || !aligned(scores, 4) || !lambda || !aligned(lambda, 4) ||
        (mean_kept && !aligned(mean_kept, 4)) || !reduce_ok(reduce) || !(k_target >= 0.f) ||
        isinf(k_target))
        return OCCAM_ERR_INVALID_ARG;
    if ((st = check_ws(P, workspace, ws_bytes)) != OCCAM_OK) return st;
    return hip_ok(launch_match_lambda(P.p, scores, reduce, k_target,
                                      ws_at<char>(workspace, P.off_match), lambda, mean_kept,
                                      stream));
}

occam_status occam_register_redirect(const occam_problem* problem, void* h, int32_t width,
                                     int64_t row_stride_bytes, const int32_t* channels,
                                     int32_t n_channels, int32_t reg_slot, hipStream_t stream) {
    Prob p;
    int bf16 = 0;
    occam_status st = key_layout(problem, &p, &bf16);
    if (st != OCCAM_OK) return st;
    const int64_t e = bf16 ? 2 : 4;
    if (!h || !aligned(h, (size_t)e) || width < 1 || row_stride_bytes < width * e ||
        row_stride_bytes % e != 0 || n_channels < 0 || n_channels > 1024 ||
        (n_channels > 0 && (!channels || !aligned(channels, 4))) || reg_slot < 0 ||
        reg_slot >= p.R)
        return OCCAM_ERR_INVALID_ARG;
    return hip_ok(launch_register_redirect(p, bf16, h, width, row_stride_bytes, channels,
                                           n_channels, reg_slot, stream));
}

}  // extern "C"
