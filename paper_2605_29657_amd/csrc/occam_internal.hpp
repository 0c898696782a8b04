// Internal definitions shared by the HIP kernels and the host entry points of
// liboccam (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <tuple>
#include <utility>

namespace occam {

// Launch `kernel` and return the status of this launch alone (hipLaunchKernel reports
// its own result; hipGetLastError would also report an unrelated earlier failure).
// The arguments are converted to the kernel's parameter types before their addresses
// are taken.
template <typename... KArgs, typename... Args>
inline hipError_t launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t smem,
                         hipStream_t s, Args&&... args) {
    static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
    std::tuple<KArgs...> vals(std::forward<Args>(args)...);
    return std::apply(
        [&](auto&... v) {
            void* ptrs[] = {static_cast<void*>(&v)...};
            return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs,
                                   smem, s);
        },
        vals);
}

// Raise the dynamic LDS limit of `kernel` to `bytes` on the current device, once per
// device: `done` holds one bit per device ordinal (0..63) whose call succeeded.  A
// failure is returned and the call is tried again next time.
inline hipError_t allow_lds(const void* kernel, int bytes, std::atomic<uint64_t>& done) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = (dev >= 0 && dev < 64) ? (uint64_t(1) << dev) : 0;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_acq_rel);
    return e;
}

constexpr int kWave = 64;
constexpr int kMaxGridY = 65535;   // launch limit of grid.y (the sample index of several kernels)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr float kLog2e = 1.4426950408889634f;

// Loads and stores of values that other workgroups of the same launch write or read
// (possibly on other XCDs, each with its own L2): device-coherent when CC, i.e. they
// bypass the non-coherent caches instead of needing a cache-wide write-back or
// invalidation.
template <bool CC, typename T>
__device__ __forceinline__ T ld(const T* p) {
    if constexpr (CC) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else return *p;
}
template <typename T>
__device__ __forceinline__ void st_cc(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Problem view passed by value to every kernel.  Offsets are device pointers
// or null (uniform batch).
struct Prob {
    int B, H, Hkv, d, R;
    int rows, cands;          // uniform T and N (used when the offsets are null)
    const int* q_off;         // [B+1] prefix of T_b, or null
    const int* k_off;         // [B+1] prefix of R + N_b, or null
    int max_rows, max_cands;  // bounds of T_b and N_b
    float scale;              // softmax temperature of Eq. (1)
    int mean_rows;            // visual keys: mean over anchor rows (1) or max (0)
    int lse_splits;           // key ranges of the statistics pass (0 or 1: one)
    long long lse_stride;     // floats between the ranges' normaliser tables
};

__device__ __forceinline__ int q_begin(const Prob& p, int b) {
    return p.q_off ? p.q_off[b] : b * p.rows;
}
__device__ __forceinline__ int rows_of(const Prob& p, int b) {
    if (!p.q_off) return p.rows;
    int t = p.q_off[b + 1] - p.q_off[b];
    return t < p.max_rows ? t : p.max_rows;
}
__device__ __forceinline__ int k_begin(const Prob& p, int b) {
    return p.k_off ? p.k_off[b] : b * (p.R + p.cands);
}
// Keys of sample b (registers + visual), clamped to the launch bounds.
__device__ __forceinline__ int keys_of(const Prob& p, int b) {
    if (!p.k_off) return p.R + p.cands;
    int s = p.k_off[b + 1] - p.k_off[b];
    int hi = p.R + p.max_cands;
    s = s < hi ? s : hi;
    return s > p.R ? s : p.R;
}
// Visual tokens of the samples before b (indexes index_map and gather sources).
__device__ __forceinline__ int cand_begin(const Prob& p, int b) {
    return k_begin(p, b) - p.R * b;
}

// s_b(r): the register scores of one sample reduced by mean, max or sum.
template <bool CC = false>
__device__ __forceinline__ float reg_reduce(const float* s, int R, int reduce) {
    if (reduce == 1) {                     // OCCAM_REG_MAX
        float m = ld<CC>(s);
        for (int r = 1; r < R; ++r) m = fmaxf(m, ld<CC>(s + r));
        return m;
    }
    float acc = 0.f;
    for (int r = 0; r < R; ++r) acc += ld<CC>(s + r);
    return reduce == 0 ? acc / (float)R : acc;   // MEAN : SUM
}

constexpr int kRefCandMean = 3;            // OCCAM_REF_CAND_MEAN

// Reference score of one sample from its R + N scores s[0 .. R + N) (registers first),
// returned to every thread of a workgroup of at least NT threads (all of them must call
// it).  Register reductions read the R register scores; the candidate mean sums the visual
// scores in a fixed order (strided over the first NT threads, a fixed shuffle tree per
// wave, the waves in order; threads past NT take no part), so every kernel that calls it
// with the same NT gets the same bits, whatever its workgroup size and wherever the scores
// are held.  `red` is NT / 64 floats of LDS.
template <int NT, bool CC = false>
__device__ __forceinline__ float reference_of(const float* s, int R, int N, int reduce,
                                              float* red) {
    if (reduce != kRefCandMean) return reg_reduce<CC>(s, R, reduce);
    const float* sv = s + R;
    const bool part = threadIdx.x < NT;
    float acc = 0.f;
    if (part) {
        // Eight loads in flight per thread; the sum still runs over v in order.
        constexpr int U = 8;
        for (int v0 = threadIdx.x; v0 < N; v0 += U * NT) {
            float x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = v0 + u * NT < N ? ld<CC>(sv + v0 + u * NT) : 0.f;
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (v0 + u * NT < N) acc += x[u];
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    __syncthreads();                          // `red` may still be read by a previous call
    if (part && (threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) sum += red[w];
    return N > 0 ? sum / (float)N : 0.f;
}

// The reference of sample b read from the packed score array.
template <int NT, bool CC = false>
__device__ __forceinline__ float sample_reference(const Prob& p, const float* scores, int b,
                                                  int reduce, float* red) {
    return reference_of<NT, CC>(scores + k_begin(p, b), p.R, keys_of(p, b) - p.R, reduce, red);
}

// Ascending compaction of a sample's survivors (sv[v] >= tau over its N visual scores)
// into out[i] and *count, by a workgroup of NT threads (all must call it).  Wave w owns the
// contiguous range [w*Q, w*Q + Q) of the candidates (Q a multiple of 64) and walks it 64
// candidates at a time: a ballot of the keep flags, its population count for the wave's
// total, and in the second pass mbcnt (the set bits below the lane) for each survivor's
// position; an LDS scan of the NT/64 wave totals places the waves' ranges.  The result
// does not depend on NT.  `wsum` is NT / 64 ints of LDS.
template <int NT>
__device__ __forceinline__ void compact_of(const float* sv, int N, float tau, int* out,
                                           int* count, int* wsum) {
    constexpr int NW = NT / kWave;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int Q = (((N + NW - 1) / NW) + kWave - 1) & ~(kWave - 1);
    const int v0 = min(N, wave * Q), v1 = min(N, v0 + Q);
    // Both walks load U groups of 64 candidates before testing them, so that U loads are in
    // flight per lane (the scores may sit in global memory); the groups are taken in order.
    constexpr int U = 8;
    int cnt = 0;
    for (int vb = v0; vb < v1; vb += U * kWave) {
        float x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = vb + u * kWave + lane;
            x[u] = v < v1 ? sv[v] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            cnt += __popcll(__ballot(vb + u * kWave + lane < v1 && x[u] >= tau));
    }
    __syncthreads();                          // `wsum` may still be read by a previous call
    if (lane == 0) wsum[wave] = cnt;
    __syncthreads();
    int base = 0, total = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        base += w < wave ? wsum[w] : 0;
        total += wsum[w];
    }
    for (int vb = v0; vb < v1; vb += U * kWave) {
        float x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = vb + u * kWave + lane;
            x[u] = v < v1 ? sv[v] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = vb + u * kWave + lane;
            const bool keep = v < v1 && x[u] >= tau;
            const unsigned long long m = __ballot(keep);
            const int below = (int)__builtin_amdgcn_mbcnt_hi(
                (unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
            if (keep) out[base + below] = v;
            base += __popcll(m);
        }
    }
    if (threadIdx.x == 0) *count = total;
}

// The compaction of sample b from the packed score array into slot[co_b + i], count[b].
template <int NT>
__device__ __forceinline__ void compact_sample(const Prob& p, const float* scores, int b,
                                               float tau, int* slot, int* count, int* wsum) {
    compact_of<NT>(scores + k_begin(p, b) + p.R, keys_of(p, b) - p.R, tau,
                   slot + cand_begin(p, b), count + b, wsum);
}

// Floats as unsigned keys with the same order: -0 folds into +0, non-negative values
// set the top bit, negative values are bit-inverted.
__device__ __forceinline__ uint32_t order_key(float x) {
    const uint32_t u = x == 0.f ? 0u : __float_as_uint(x);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// bf16 <-> f32 on raw 16-bit patterns.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Row tensors gathered with the survivors (host struct occam_rows, by value).
constexpr int kMaxRowTensors = 8;
struct RowTensor {
    const char* src;
    char* dst;
    long long src_pad_rows, src_row0, src_stride, dst_stride, row_bytes;
};
struct RowTensors {
    RowTensor t[kMaxRowTensors];
    int n;
    int vec16;  // every pointer, stride and row length is a multiple of 16 bytes
};

// ---------------------------------------------------------------------------
// Tiling constants.
// Anchor (T = 1) path: VALU dot products, KPW keys per workgroup.
constexpr int kClsThreads = 256;
constexpr int kClsPartials = 8192;   // LDS floats of per-chunk partial dot products
// Text (T > 1) path: MFMA 32x32x16 bf16; 4 waves; a t-block of 128 anchor rows
// (4 sub-blocks of 32) and 32 keys per wave.
constexpr int kTxtThreads = 256;
constexpr int kStatsThreads = 256;
constexpr int kScoreThreads = 256;
constexpr int kTxtRows = 128;
constexpr int kTxtKeysPerWave = 32;
constexpr int kTxtKeysPerWg = 128;   // score kernel: 4 key blocks of 32
constexpr int kSelThreads = 256;    // threshold, top-K, budget matching; reference-sum order
constexpr int kSelectThreads = 512; // the select kernel (its reference sum uses kSelThreads)
constexpr int kGatherThreads = 256;

// The chip dispatches consecutive workgroups of a launch round-robin over its 8
// XCDs, each with its own L2.  xcd_remap turns a linear workgroup id into a task
// index such that each XCD receives one contiguous range of tasks (XCD x gets
// ranges of q+1 tasks for x < r, q otherwise, with total = 8 q + r), so tasks that
// share data (the key chunks of one sample share its query tiles) meet in one L2.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_remap(int id, int total) {
    const int q = total / kXcds, r = total % kXcds;
    const int x = id % kXcds, j = id / kXcds;
    return x < r ? x * (q + 1) + j : r * (q + 1) + (x - r) * q + j;
}

// Dynamic LDS of the text-row scoring kernel: two query tiles (128 rows x d bf16)
// and the [H][128] float normaliser tile; at most kScoreSmemMax.
constexpr size_t kScoreSmemMax = 160 * 1024;
inline size_t text_score_smem(int H, int d16) {
    return 2 * (size_t)kTxtRows * d16 * 2 + (size_t)H * kTxtRows * 4;
}

// Dynamic LDS of the text-row statistics kernel: a ring of kStatsRing key blocks
// (32 keys x d bf16) per key stream, plus the (max, sum) merge arrays.  Two stages (one
// block in flight per stream while the other is used) and four workgroups per CU read
// the head slices faster than deeper rings at fewer workgroups per CU: the scattered
// 256-byte slices stream better with fewer requests outstanding per CU.
constexpr int kStatsRing = 2;
// Row blocks per statistics workgroup for nrb 128-row blocks per sample (at most).
inline int stats_row_blocks(int nrb) { return nrb == 2 ? 2 : (nrb == 3 || nrb == 4) ? 4 : 1; }
// Key ranges of the statistics pass: a batch with fewer than kStatsMinWorkgroups
// (sample, head, row-block group) tasks splits each task's keys into up to kStatsMaxSplits
// ranges of at least kStatsMinSplitBlocks 32-key blocks; each range writes its own base-2
// log-sum-exp table, and the scoring pass merges them.
constexpr int kStatsMinWorkgroups = 1024;
constexpr int kStatsMaxSplits = 8;
constexpr int kStatsMinSplitBlocks = 16;
inline int stats_splits(long long tasks, long long keys) {
    if (tasks <= 0 || tasks >= kStatsMinWorkgroups) return 1;
    long long ks = (kStatsMinWorkgroups + tasks - 1) / tasks;
    const long long by_keys = ((keys + 31) / 32) / kStatsMinSplitBlocks;
    if (ks > by_keys) ks = by_keys;
    if (ks > kStatsMaxSplits) ks = kStatsMaxSplits;
    return ks < 1 ? 1 : (int)ks;
}
// rg: waves per key stream of one row block (2 or 4); rbw: row blocks per workgroup.
inline size_t text_stats_smem(int d16, int rg, int rbw = 1) {
    return (size_t)(kStatsThreads / kWave / rg) * kStatsRing * 32 * d16 * 2 +
           2 * (size_t)(kStatsThreads / kWave / rg) * rbw * kTxtRows * 4;
}

// Anchor-path keys per workgroup for a given row geometry.
// Streaming form of the one-row logits (cls_stream_kernel): every query head has its
// own key head, a head is NC 16-byte chunks with NC a power of two up to 16, and a key
// row is 1 to 4 whole 64-lane loads.  Returns NC when the form applies, else 0.
// Lanes per head of the streaming one-row form: the head's 16-byte chunk count rounded
// up to a power of two (at most 16; lanes past the real chunks contribute zero), or 0
// when the form does not apply.
inline int cls_stream_nc(int H, int Hkv, int d, int elem_bytes) {
    if (H != Hkv || (d * elem_bytes) % 16 != 0) return 0;
    const int nc = d * elem_bytes / 16;
    if (nc < 1 || nc > 16) return 0;
    int ncp = 1;
    while (ncp < nc) ncp *= 2;
    const int cpk = ncp * Hkv;
    if (cpk % 64 != 0 || cpk / 64 > 4) return 0;
    return ncp;
}
constexpr int kClsStreamKeys = 128;    // keys per workgroup of the streaming form
// Small batches: the streaming form halves its keys per workgroup (down to 16) until the
// launch has this many workgroups (two per CU), so that a single image is read by many
// CUs at once instead of a handful.
constexpr int kClsMinWorkgroups = 512;

inline int cls_keys_per_wg(int H, int Hkv, int d, int elem_bytes, int B = 0, long long keys = 0) {
    if (cls_stream_nc(H, Hkv, d, elem_bytes)) {
        int kpw = kClsStreamKeys;
        while (kpw > 16 && (long long)B * ((keys + kpw - 1) / kpw) < kClsMinWorkgroups) kpw /= 2;
        return kpw;
    }
    int chunks_per_head = d * elem_bytes / 16;
    int kpw = kClsPartials / (H * chunks_per_head);
    if (kpw > 64) kpw = 64;
    if (kpw < 1) kpw = 1;
    return kpw;
}

// Per-sample epilogue of occam_prune, run inside the scoring kernels by the last
// workgroup to finish each sample (so that no separate threshold / select or row-block
// combine launch is needed).  done[B] counts the finished workgroups of every sample; the
// kernel that runs just before the scoring kernel in the same call clears it.  done ==
// null: no epilogue.
struct Finish {
    unsigned* done;
    int select;            // threshold + compaction (else only the row-block combine)
    float lambda;
    int reduce;
    float* tau;            // [B], tau_b
    int* slot;             // survivors, slot[co_b + i]
    int* count;            // [B]
    // One-row path instead (chunk_cnt != null): every scoring workgroup thresholds and
    // compacts its own chunk of kpw keys into chunk_slot[(b * nchunks + c) * kpw + i],
    // writes chunk_cnt[b * nchunks + c] and adds it to count[b] (cleared by the logits
    // kernel); pack_gather places the chunk lists.
    int* chunk_slot;
    int* chunk_cnt;
};

// Zero the counters the scoring kernel accumulates into (one workgroup of the kernel that
// precedes it in the call): done[0 .. B), or count[0 .. B) for the per-chunk compaction.
__device__ __forceinline__ void clear_done(const Finish& f, int B) {
    if (f.done)
        for (int i = threadIdx.x; i < B; i += blockDim.x) f.done[i] = 0u;
    if (f.chunk_cnt)
        for (int i = threadIdx.x; i < B; i += blockDim.x) f.count[i] = 0;
}

// Most chunks per sample of the per-chunk compaction (pack_gather scans their counts in LDS).
constexpr int kMaxChunkLists = 1024;

// Every thread of the workgroup calls this after writing its share of sample b's scores
// (or row-block partials) with device-coherent stores (st_cc).  Each wave waits until its
// stores have completed, the workgroup counts itself, and the one that completes the
// sample's ntask workgroups gets true; it then reads the other workgroups' values with
// device-coherent loads (ld<true>).  No cache-wide write-back or invalidation is needed
// (measured: an agent-scope release/acquire fence pair in every workgroup of the Stage II
// scoring kernel cost ~90 us per launch).  flag: one int of LDS.
__device__ __forceinline__ bool last_of_sample(unsigned* done, int b, unsigned ntask, int* flag) {
    __builtin_amdgcn_s_waitcnt(0x0F70);          // vmcnt(0): this wave's stores are done
    __syncthreads();
    if (threadIdx.x == 0)
        *flag = __hip_atomic_fetch_add(done + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u ==
                ntask;
    __syncthreads();
    return *flag != 0;
}

// LDS the per-sample epilogue needs: its scratch words and a copy of the sample's scores.
constexpr size_t kSelectScratch = 64;
inline size_t select_lds_bytes(int R, int max_cands) {
    return kSelectScratch + 4 * ((size_t)R + (size_t)max_cands);
}

// Where select_sample keeps its copy of the sample's scores (lds as passed to it).
__device__ __forceinline__ float* select_scores_lds(char* lds) {
    return reinterpret_cast<float*>(lds + kSelectScratch);
}

// Threshold (tau_b = lambda * reference, the fused threshold of select_kernel) and
// compaction of sample b by one workgroup of kSelThreads threads.  The sample's scores,
// written by other workgroups of the launch, are first copied into LDS with
// device-coherent loads (eight in flight per thread), unless the caller has already put
// them there (in_lds, followed by a barrier); the reference and the compaction then read
// the copy, with select_kernel's arithmetic.  lds: select_lds_bytes(R, N_b).
__device__ __forceinline__ void select_sample(const Prob& p, const float* scores, int b,
                                              const Finish& f, char* lds, bool in_lds) {
    float* red = reinterpret_cast<float*>(lds);              // kSelThreads / 64 floats
    int* wsum = reinterpret_cast<int*>(lds + 16);            // kSelThreads / 64 ints
    float* tau_s = reinterpret_cast<float*>(lds + 32);
    float* sl = select_scores_lds(lds);
    const int S = keys_of(p, b);
    const float* src = scores + k_begin(p, b);
    constexpr int U = 8;
    for (int i0 = threadIdx.x; i0 < S && !in_lds; i0 += U * kSelThreads) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * kSelThreads;
            v[u] = i < S ? ld<true>(src + i) : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * kSelThreads;
            if (i < S) sl[i] = v[u];
        }
    }
    __syncthreads();
    const float t = f.lambda * reference_of<kSelThreads>(sl, p.R, S - p.R, f.reduce, red);
    if (threadIdx.x == 0) {
        if (f.tau) f.tau[b] = t;
        *tau_s = t;
    }
    __syncthreads();
    compact_of<kSelThreads>(sl + p.R, S - p.R, *tau_s, f.slot + cand_begin(p, b), f.count + b,
                            wsum);
}

// ---------------------------------------------------------------------------
// Launchers (defined in the .hip files).  Each returns the status of its own launches.
hipError_t launch_select_topk(const Prob& p, const float* scores, int k_keep, int* slot,
                              int* count, hipStream_t s);
// Selection state of budget matching, in the workspace.
constexpr size_t kMatchStateBytes = 8192;
hipError_t launch_match_lambda(const Prob& p, const float* scores, int reduce, float k_target,
                               void* state, float* lambda, float* mean_kept, hipStream_t s);
hipError_t launch_register_redirect(const Prob& p, int bf16, void* h, int width, long long stride,
                                    const int* channels, int n_channels, int reg_slot,
                                    hipStream_t s);
// fin.done (nullable) is cleared by launch_cls_logits / launch_text_stats and used by the
// scoring launch that follows them in the same call.
hipError_t launch_cls_logits(const Prob& p, int bf16, const void* q, const void* k,
                             float* logits, float2* stats, int kpw, const Finish& fin,
                             hipStream_t s);
hipError_t launch_cls_scores(const Prob& p, int bf16, const float* logits, const float2* stats,
                             const float* row_lse, float* scores, int kpw, const Finish& fin,
                             hipStream_t s);
hipError_t launch_text_stats(const Prob& p, const void* q, const void* k, float* lse2,
                             const Finish& fin, hipStream_t s);
// Mutual scoring (every key: mean over rows): column sums per (row block, head) into
// part [B][ceil(max_rows/128)][H][R + max_cands], then their fixed-order mean.
hipError_t launch_text_colsum(const Prob& p, const void* q, const void* k, const float* lse,
                              int lse_natural, float* part, float* scores, hipStream_t s);
// Max-over-rows scoring; with several 128-row blocks, per-block partials go to part
// [B][ceil(max_rows/128)][R + max_cands] and a combine kernel forms the scores.
// With fin.done the row-block combine (and with fin.select the threshold and the
// compaction) run in each sample's last workgroup; without it text_rows_combine follows.
hipError_t launch_text_score(const Prob& p, const void* q, const void* k, const float* lse,
                             int lse_natural, float* scores, float* part, const Finish& fin,
                             hipStream_t s);
hipError_t launch_threshold(const Prob& p, const float* scores, float lambda, int reduce,
                            float* tau, hipStream_t s);
hipError_t launch_select(const Prob& p, const float* scores, const float* tau, int fuse_tau,
                         float lambda, int reduce, float* tau_out, int* slot, int* count,
                         hipStream_t s);
// Survivors from the per-chunk lists of the one-row scoring kernel (chunk_cnt != null)
// or from slot[co_b + i] (select); counts per sample in count[B] either way.
struct ChunkLists {
    const int* slot;       // [B][nchunks][kpw]
    const int* cnt;        // [B][nchunks]
    int nchunks, kpw;
};
hipError_t launch_pack_gather(const Prob& p, const int* slot, const int* count,
                              const int* index_map, int* kept_idx, int* kept_offsets,
                              const int* packed_idx, const int* packed_offsets,
                              const RowTensors& rows, hipStream_t s,
                              const ChunkLists& lists = ChunkLists{});

}  // namespace occam
