// Fixed-budget selection, the component ablation's alternative to the relative test
// (Appendix, Table tab:qwen_compact_component_ablation): per sample, the K visual tokens
// with the largest scores, the lower index first among equal scores.
//
// select_topk   one workgroup per sample.  A radix select over the float-ordered score
//               keys (8 bits per pass from the top, LDS histogram, a suffix scan picks
//               the digit) finds the K-th largest key t and how many keys equal to t
//               are kept (q).  Each thread then owns a contiguous strip of candidates:
//               two block scans give every strip its share of the equal keys (the
//               first q in index order) and its output position, and the strip writes
//               its survivors in ascending order into the same per-sample slot list
//               that the threshold selection fills, so the packing and the gathers are
//               shared with it.
#include "occam_internal.hpp"

namespace occam {

static_assert(kSelThreads == 256, "one histogram bin per thread");

// Exclusive scan of one int per thread over the workgroup; `total` gets the sum.
__device__ __forceinline__ int block_exclusive_scan(int x, int* wsum, int& total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int inc = x;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int o = __shfl_up(inc, off);
        if (lane >= off) inc += o;
    }
    if (lane == kWave - 1) wsum[wave] = inc;
    __syncthreads();
    int base = 0;
    total = 0;
#pragma unroll
    for (int w = 0; w < kSelThreads / kWave; ++w) {
        base += w < wave ? wsum[w] : 0;
        total += wsum[w];
    }
    __syncthreads();                              // wsum is free for the next scan
    return base + inc - x;
}

__global__ __launch_bounds__(kSelThreads) void select_topk_kernel(
    Prob p, const float* __restrict__ scores, int k_keep, int* __restrict__ slot,
    int* __restrict__ count)
{
    __shared__ uint32_t hist[256];
    __shared__ uint32_t suffix[257];
    __shared__ uint32_t sh_prefix, sh_rank;
    __shared__ int wsum[kSelThreads / kWave];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int N = keys_of(p, b) - p.R;
    const int co = cand_begin(p, b);
    const float* sv = scores + k_begin(p, b) + p.R;
    const int K = min(k_keep, N);
    if (tid == 0) count[b] = K;
    if (K == 0) return;

    // The K-th largest key t and the rank q of the target among the keys equal to t.
    uint32_t prefix = 0, mask = 0, rank = (uint32_t)K;
    for (int shift = 24; shift >= 0; shift -= 8) {
        hist[tid] = 0;
        __syncthreads();
        for (int v = tid; v < N; v += kSelThreads) {
            const uint32_t key = order_key(sv[v]);
            if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        suffix[tid] = hist[tid];
        if (tid == 0) suffix[256] = 0;
        __syncthreads();
        for (int off = 1; off < 256; off <<= 1) {
            const uint32_t add = tid + off < 256 ? suffix[tid + off] : 0u;
            __syncthreads();
            suffix[tid] += add;
            __syncthreads();
        }
        if (suffix[tid + 1] < rank && rank <= suffix[tid]) {
            sh_prefix = prefix | ((uint32_t)tid << shift);
            sh_rank = rank - suffix[tid + 1];
        }
        __syncthreads();
        prefix = sh_prefix;
        rank = sh_rank;
        mask |= 255u << shift;
    }
    const uint32_t t = prefix;
    const int q = (int)rank;                      // keys equal to t that are kept

    // Strips: counts above t and equal to t, then positions.
    const int P = (N + kSelThreads - 1) / kSelThreads;
    const int v0 = min(N, tid * P), v1 = min(N, v0 + P);
    int gt = 0, eq = 0;
    for (int v = v0; v < v1; ++v) {
        const uint32_t key = order_key(sv[v]);
        gt += key > t;
        eq += key == t;
    }
    int total;
    const int eq_before = block_exclusive_scan(eq, wsum, total);
    const int eq_take = min(max(q - eq_before, 0), eq);
    int pos = block_exclusive_scan(gt + eq_take, wsum, total);
    int eq_left = eq_take;
    for (int v = v0; v < v1; ++v) {
        const uint32_t key = order_key(sv[v]);
        if (key > t || (key == t && eq_left > 0)) {
            eq_left -= key == t;
            slot[co + pos++] = v;
        }
    }
}

hipError_t launch_select_topk(const Prob& p, const float* scores, int k_keep, int* slot,
                              int* count, hipStream_t s)
{
    return launch(select_topk_kernel, dim3(p.B), dim3(kSelThreads), 0, s, p, scores, k_keep, slot,
                  count);
}

}  // namespace occam
