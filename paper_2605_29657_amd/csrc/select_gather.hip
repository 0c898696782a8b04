// Steps 3-5 of the relative evidence test: the register-anchored threshold
// (Eqs. stage1_threshold_appendix, stage2_set_appendix), the >= test of
// Eqs. stage1 / stage2, the ascending compaction of the survivors, and the
// dense copy of their rows that forms the pruned sequence of Algorithm 1.
//
// threshold    one thread per sample: tau = lambda * reduce(register scores); for
//              the ablation's mean-based threshold one workgroup per sample
//              averages the visual scores instead (sample_reference).
// select       one workgroup per sample: every wave owns a contiguous range of
//              candidates and walks it 64 at a time, a ballot of the keep flags
//              counting its survivors; an LDS scan of the wave totals places the
//              ranges, and a second walk writes each survivor's candidate-local
//              index, ascending, at its position (mbcnt below the lane) in the
//              sample's slot of the workspace (slot[co_b + i]).  Optionally computes
//              tau first (fused threshold of occam_prune).  The same compaction runs
//              in the last workgroup of each sample of the Stage II scoring kernel.
// pack_gather  grid (G, sample): every wave forms its sample's packed offset
//              (exclusive sum of the counts before it, with shuffles: no
//              barrier); with Stage I's per-chunk lists, an LDS scan of the chunk
//              counts concatenates them.  The workgroups write the packed survivor
//              list (through index_map when given) and kept_offsets, and their
//              waves copy survivor rows of every row tensor with 16-byte
//              non-temporal loads and stores, one row per wave at a time.
#include "occam_internal.hpp"

namespace occam {

__global__ void threshold_kernel(Prob p, const float* __restrict__ scores, float lambda,
                                 int reduce, float* __restrict__ tau)
{
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= p.B) return;
    tau[b] = lambda * reg_reduce(scores + k_begin(p, b), p.R, reduce);
}

// Mean-based threshold: one workgroup per sample reduces its visual scores.
__global__ __launch_bounds__(kSelThreads) void threshold_mean_kernel(
    Prob p, const float* __restrict__ scores, float lambda, float* __restrict__ tau)
{
    __shared__ float red[kSelThreads / kWave];
    const float ref = sample_reference<kSelThreads>(p, scores, blockIdx.x, kRefCandMean, red);
    if (threadIdx.x == 0) tau[blockIdx.x] = lambda * ref;
}

__global__ __launch_bounds__(kSelectThreads) void select_kernel(
    Prob p, const float* __restrict__ scores, const float* __restrict__ tau_in, int fuse_tau,
    float lambda, int reduce, float* __restrict__ tau_out, int* __restrict__ slot,
    int* __restrict__ count)
{
    // The fused threshold's reference sum runs in the order of kSelThreads threads, the
    // same bits as occam_threshold and budget matching.
    __shared__ int wsum[kSelectThreads / kWave];
    __shared__ float red[kSelThreads / kWave];
    __shared__ float tau_s;
    const int b = blockIdx.x;
    if (fuse_tau) {
        const float t = lambda * sample_reference<kSelThreads>(p, scores, b, reduce, red);
        if (threadIdx.x == 0) {
            if (tau_out) tau_out[b] = t;
            tau_s = t;
        }
    } else if (threadIdx.x == 0) {
        tau_s = tau_in[b];
    }
    __syncthreads();
    compact_sample<kSelectThreads>(p, scores, b, tau_s, slot, count, wsum);
}

__global__ __launch_bounds__(kGatherThreads) void pack_gather_kernel(
    Prob p, const int* __restrict__ slot, const int* __restrict__ count,
    const int* __restrict__ index_map, int* __restrict__ kept_idx, int* __restrict__ kept_offsets,
    const int* __restrict__ packed_idx, const int* __restrict__ packed_offsets, RowTensors rows,
    ChunkLists lists)
{
    __shared__ int pc[kMaxChunkLists + 1];       // per-chunk lists: exclusive prefix of counts
    __shared__ int wsum[kGatherThreads / kWave];
    const int b = blockIdx.y, x = blockIdx.x, G = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int co = cand_begin(p, b);
    int off, cnt;
    const int* idx;
    const int nlist = lists.cnt ? lists.nchunks : 0;
    // The chunk counts are loaded before the counts of the earlier samples are summed, so
    // that both loads are in flight together.
    constexpr int PER = kMaxChunkLists / kGatherThreads;
    int v[PER], sum = 0;
    if (nlist) {
        const int* cc = lists.cnt + (size_t)b * nlist;
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int c = tid * PER + j;
            v[j] = c < nlist ? cc[c] : 0;
        }
    }
    int before = 0;
    if (!packed_idx) {
        // The sample's packed offset, the sum of the counts before it: every wave forms it
        // on its own (strided partial sums, then a shuffle tree), so no barrier is needed.
        for (int j = lane; j < b; j += kWave) before += count[j];
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) before += __shfl_xor(before, o);
    }
    if (nlist) {
        // The sample's survivors are the concatenation of its chunk lists: a block scan of
        // the chunk counts (four per thread) gives each list its start.
#pragma unroll
        for (int j = 0; j < PER; ++j) sum += v[j];
        int inc = sum;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int t = __shfl_up(inc, o);
            if (lane >= o) inc += t;
        }
        if (lane == kWave - 1) wsum[wave] = inc;
        __syncthreads();
        int run = inc - sum;
        for (int w = 0; w < wave; ++w) run += wsum[w];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int c = tid * PER + j;
            if (c < nlist) pc[c] = run;
            run += v[j];
        }
        if (tid == kGatherThreads - 1) pc[nlist] = run;
        __syncthreads();
    }
    // Candidate index of the sample's i-th survivor (any i, per thread).
    auto survivor = [&](int i) -> int {
        if (!nlist) return idx[i];
        int lo = 0, hi = nlist - 1;                // the chunk c with pc[c] <= i < pc[c + 1]
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (pc[mid] <= i) lo = mid; else hi = mid - 1;
        }
        return lists.slot[((size_t)b * nlist + lo) * lists.kpw + (i - pc[lo])];
    };
    // The same for an i that is uniform over the wave: the chunk is the number of list
    // starts at or below i, less one, counted 64 lists at a time with a ballot.
    auto survivor_w = [&](int i) -> int {
        if (!nlist) return idx[i];
        int n = 0;
        for (int c0 = 0; c0 < nlist; c0 += kWave) {
            const int c = c0 + lane;
            n += __popcll(__ballot(c < nlist && pc[c] <= i));
        }
        const int c = n - 1;
        return lists.slot[((size_t)b * nlist + c) * lists.kpw + (i - pc[c])];
    };
    if (packed_idx) {
        off = packed_offsets[b];
        cnt = packed_offsets[b + 1] - off;
        idx = packed_idx + off;
    } else {
        off = before;
        cnt = count[b];
        idx = slot + co;
        if (x == 0 && tid == 0) {
            kept_offsets[b] = off;
            if (b == p.B - 1) kept_offsets[p.B] = off + cnt;
        }
        for (int i = x * kGatherThreads + tid; i < cnt; i += G * kGatherThreads) {
            const int v = survivor(i);
            kept_idx[off + i] = index_map ? index_map[co + v] : v;
        }
    }
    const int nt = rows.n;
    if (nt == 0) return;
    const int jobs = cnt * nt;
    const int nw = kGatherThreads / kWave;
    for (int j = x * nw + wave; j < jobs; j += G * nw) {
        const int i = j / nt, t = j - i * nt;
        const int v = survivor_w(i);
        const RowTensor& rt = rows.t[t];
        const char* src = rt.src + ((long long)co + (long long)b * rt.src_pad_rows + rt.src_row0 + v) *
                                       rt.src_stride;
        char* dst = rt.dst + (long long)(off + i) * rt.dst_stride;
        const long long nb = rt.row_bytes;
        if (rows.vec16) {
            // Four 16-byte loads in flight per lane before the stores.  The copies are
            // non-temporal: the rows are touched once, and without the hint they would
            // take room in the 256 MB memory-side cache and leave dirty lines there
            // (measured with the steps cycling through three input copies: the
            // LLaVA-NeXT step 0.437 -> 0.428 ms).
            // A 2 KB row (Stage I hidden states) is two loads per lane, both issued
            // before either store.
            constexpr long long step = 16 * kWave;
            for (long long o = (long long)lane * 16; o < nb; o += 4 * step) {
                u32x4 a[4];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (o + u * step < nb)
                        a[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + o + u * step));
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (o + u * step < nb)
                        __builtin_nontemporal_store(a[u], reinterpret_cast<u32x4*>(dst + o + u * step));
            }
        } else {
            for (long long o = (long long)lane * 4; o < nb; o += 4 * kWave)
                *reinterpret_cast<uint32_t*>(dst + o) = *reinterpret_cast<const uint32_t*>(src + o);
        }
    }
}

hipError_t launch_threshold(const Prob& p, const float* scores, float lambda, int reduce,
                            float* tau, hipStream_t s)
{
    if (reduce == kRefCandMean)
        return launch(threshold_mean_kernel, dim3(p.B), dim3(kSelThreads), 0, s, p, scores, lambda,
                      tau);
    return launch(threshold_kernel, dim3((p.B + 255) / 256), dim3(256), 0, s, p, scores, lambda,
                  reduce, tau);
}

hipError_t launch_select(const Prob& p, const float* scores, const float* tau, int fuse_tau,
                         float lambda, int reduce, float* tau_out, int* slot, int* count,
                         hipStream_t s)
{
    return launch(select_kernel, dim3(p.B), dim3(kSelectThreads), 0, s, p, scores, tau, fuse_tau,
                  lambda, reduce, tau_out, slot, count);
}

hipError_t launch_pack_gather(const Prob& p, const int* slot, const int* count,
                              const int* index_map, int* kept_idx, int* kept_offsets,
                              const int* packed_idx, const int* packed_offsets,
                              const RowTensors& rows, hipStream_t s, const ChunkLists& lists)
{
    // Enough workgroups per sample to cover the worst-case survivor count with
    // one row per wave, but no more than ~4096 in total (16 per CU; fewer rows per
    // wave shorten the copy: 2048 measured ~2.5 us slower on the LLaVA-NeXT Stage I).
    const int nw = kGatherThreads / kWave;
    long long per = rows.n > 0 ? ((long long)p.max_cands * rows.n + nw - 1) / nw
                               : ((long long)p.max_cands + kGatherThreads - 1) / kGatherThreads;
    long long cap = (4096 + p.B - 1) / p.B;
    long long G = per < cap ? per : cap;
    if (G < 1) G = 1;
    if (lists.cnt && (lists.nchunks < 1 || lists.nchunks > kMaxChunkLists))
        return hipErrorInvalidValue;
    return launch(pack_gather_kernel, dim3((unsigned)G, p.B), dim3(kGatherThreads), 0, s, p, slot,
                  count, index_map, kept_idx, kept_offsets, packed_idx, packed_offsets, rows,
                  lists);
}

}  // namespace occam
