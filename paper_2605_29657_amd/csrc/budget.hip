// Budget matching (Appendix Eq. lambda2_budget_matching_appendix) on the device: the
// lambda whose mean kept count over the batch is closest to a target.
//
// The count #{v : s_b(v) >= lambda s_b(r)} summed over samples is a step function of
// lambda that drops at each ratio s_b(v) / s_b(r).  With T = k_target * B and
// c = T rounded half down (clamped to [1, M], M candidates), the best level is either
// the level of the c-th largest ratio v1 (count #{r >= v1}) or the level just above it
// (count #{r > v1}, value = the smallest ratio above v1): every other level's count is
// farther from T.  Ties take the smaller count.  lambda is the geometric midpoint of
// the chosen level's value and the next smaller distinct ratio (half the value if
// there is no positive one; 0 if the level itself is not positive).
//
// Ratios are mapped to unsigned keys that order like the floats, and the c-th largest
// key is found by a radix select, 8 bits per pass from the top:
//   match_init   one workgroup: clears the selection state, counts M, sets c.
//   match_hist   grid (B, candidate chunks of 1024): LDS histogram of the pass's digit
//                over the keys that match the prefix chosen so far, added into one
//                global histogram; the last workgroup to finish picks the digit and
//                the rank left inside it.
//   match_count  same grid: #{key >= v1}, #{key > v1}, the nearest keys above and
//                below v1; the last workgroup chooses the level and writes lambda.
// Every workgroup recomputes its sample's reference (s_b(r), or the mean visual score
// of the ablation) with the same reduction as the threshold kernels.
#include "occam_internal.hpp"

namespace occam {

constexpr int kMatchThreads = kSelThreads;      // same reference bits as occam_threshold
constexpr int kMatchPer = 4;                              // keys per thread per chunk
constexpr int kMatchChunk = kMatchThreads * kMatchPer;

struct MatchState {
    uint32_t hist[4][256];
    uint32_t prefix[4];       // key bits chosen up to and including pass i
    uint32_t rank[5];         // rank of the target inside the prefix group (rank[0] = c)
    uint32_t done[5];         // finished workgroups per pass (4 histograms + count)
    uint32_t M;
    uint32_t c_hi, c_lo, v_above, v_below;
};
static_assert(sizeof(MatchState) <= kMatchStateBytes, "match state exceeds its workspace");

__device__ __forceinline__ uint32_t load_cc(const uint32_t* a) {  // coherent across workgroups
    return __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The chunk's keys: out-of-range slots get `valid` cleared.
struct ChunkKeys {
    uint32_t key[kMatchPer];
    bool valid[kMatchPer];
};
__device__ __forceinline__ ChunkKeys chunk_keys(const Prob& p, const float* scores, int reduce) {
    __shared__ float red[kMatchThreads / kWave];
    const int b = blockIdx.x;
    const int kb = k_begin(p, b);
    const int N = keys_of(p, b) - p.R;
    const float sr = sample_reference<kMatchThreads>(p, scores, b, reduce, red);
    ChunkKeys ck;
#pragma unroll
    for (int j = 0; j < kMatchPer; ++j) {
        const int v = blockIdx.y * kMatchChunk + j * kMatchThreads + threadIdx.x;
        ck.valid[j] = v < N;
        ck.key[j] = ck.valid[j] ? order_key(scores[kb + p.R + v] / sr) : 0u;
    }
    return ck;
}

// True in every thread of the workgroup that finished last among the grid.
__device__ __forceinline__ bool last_workgroup(uint32_t* done) {
    __shared__ bool last;
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0)
        last = atomicAdd(done, 1u) == gridDim.x * gridDim.y - 1;
    __syncthreads();
    if (last) __threadfence();
    return last;
}

__global__ __launch_bounds__(kMatchThreads) void match_init_kernel(Prob p, float k_target,
                                                                   MatchState* st)
{
    __shared__ uint32_t m_sh;
    const int tid = threadIdx.x;
    uint32_t* w = reinterpret_cast<uint32_t*>(st);
    for (int i = tid; i < (int)(sizeof(MatchState) / 4); i += kMatchThreads) w[i] = 0u;
    if (tid == 0) m_sh = 0;
    __syncthreads();
    uint32_t m = 0;
    for (int b = tid; b < p.B; b += kMatchThreads) m += (uint32_t)(keys_of(p, b) - p.R);
    atomicAdd(&m_sh, m);
    __syncthreads();
    if (tid == 0) {
        const uint32_t M = m_sh;
        double c = ceil((double)k_target * (double)p.B - 0.5);   // T rounded half down
        c = c < 1.0 ? 1.0 : (c > (double)M ? (double)M : c);
        st->M = M;
        st->rank[0] = (uint32_t)c;
        st->v_above = 0xFFFFFFFFu;
    }
}

template <int PASS>
__global__ __launch_bounds__(kMatchThreads) void match_hist_kernel(
    Prob p, const float* __restrict__ scores, int reduce, MatchState* st)
{
    __shared__ uint32_t hist[256];
    __shared__ uint32_t suffix[257];
    constexpr int shift = 24 - 8 * PASS;
    const int tid = threadIdx.x;
    hist[tid] = 0;
    const uint32_t mask = PASS == 0 ? 0u : ~0u << (32 - 8 * PASS);
    const uint32_t prefix = PASS == 0 ? 0u : st->prefix[PASS - 1];
    __syncthreads();
    const ChunkKeys ck = chunk_keys(p, scores, reduce);
#pragma unroll
    for (int j = 0; j < kMatchPer; ++j)
        if (ck.valid[j] && (ck.key[j] & mask) == prefix)
            atomicAdd(&hist[(ck.key[j] >> shift) & 255u], 1u);
    __syncthreads();
    if (hist[tid]) atomicAdd(&st->hist[PASS][tid], hist[tid]);
    if (!last_workgroup(&st->done[PASS])) return;

    // Pick the digit: suffix[d] = keys in the group with digit >= d; the target of rank
    // k (1 = largest) has the digit d with suffix[d + 1] < k <= suffix[d].
    const uint32_t k = load_cc(&st->rank[PASS]);
    suffix[tid] = load_cc(&st->hist[PASS][tid]);
    if (tid == 0) suffix[256] = 0;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const uint32_t add = tid + off < 256 ? suffix[tid + off] : 0u;
        __syncthreads();
        suffix[tid] += add;
        __syncthreads();
    }
    if (suffix[tid + 1] < k && k <= suffix[tid]) {
        st->prefix[PASS] = prefix | ((uint32_t)tid << shift);
        st->rank[PASS + 1] = k - suffix[tid + 1];
    }
}

__global__ __launch_bounds__(kMatchThreads) void match_count_kernel(
    Prob p, const float* __restrict__ scores, int reduce, float k_target, MatchState* st,
    float* __restrict__ lambda, float* __restrict__ mean_kept)
{
    __shared__ uint32_t s_hi, s_lo, s_above, s_below;
    const int tid = threadIdx.x;
    if (tid == 0) { s_hi = 0; s_lo = 0; s_above = 0xFFFFFFFFu; s_below = 0u; }
    const uint32_t v1 = st->prefix[3];
    __syncthreads();
    const ChunkKeys ck = chunk_keys(p, scores, reduce);
    uint32_t hi = 0, lo = 0, above = 0xFFFFFFFFu, below = 0u;    // below holds key + 1
#pragma unroll
    for (int j = 0; j < kMatchPer; ++j) {
        if (!ck.valid[j]) continue;
        const uint32_t key = ck.key[j];
        hi += key >= v1;
        lo += key > v1;
        if (key > v1) above = min(above, key);
        if (key < v1) below = max(below, key + 1u);
    }
    if (hi) atomicAdd(&s_hi, hi);
    if (lo) atomicAdd(&s_lo, lo);
    if (above != 0xFFFFFFFFu) atomicMin(&s_above, above);
    if (below) atomicMax(&s_below, below);
    __syncthreads();
    if (tid == 0) {
        if (s_hi) atomicAdd(&st->c_hi, s_hi);
        if (s_lo) atomicAdd(&st->c_lo, s_lo);
        if (s_above != 0xFFFFFFFFu) atomicMin(&st->v_above, s_above);
        if (s_below) atomicMax(&st->v_below, s_below);
    }
    if (!last_workgroup(&st->done[4]) || tid != 0) return;

    const uint32_t M = load_cc(&st->M);
    if (M == 0) {                                  // no candidates: nothing to match
        lambda[0] = 1.f;
        if (mean_kept) mean_kept[0] = 0.f;
        return;
    }
    const uint32_t c_hi = load_cc(&st->c_hi), c_lo = load_cc(&st->c_lo);
    const uint32_t v_above = load_cc(&st->v_above), v_below = load_cc(&st->v_below);
    const double T = (double)k_target * (double)p.B;
    uint32_t level, count;
    bool has_next;
    uint32_t next;
    if (c_lo >= 1 && fabs((double)c_lo - T) <= fabs((double)c_hi - T)) {
        level = v_above; count = c_lo; has_next = true; next = v1;
    } else {
        level = v1; count = c_hi; has_next = v_below != 0u; next = v_below - 1u;
    }
    const double lv = (double)key_value(level);
    const double nv = has_next ? (double)key_value(next) : 0.0;
    const double lam = (lv > 0.0 && nv > 0.0) ? sqrt(lv * nv) : (lv > 0.0 ? 0.5 * lv : 0.0);
    lambda[0] = (float)lam;
    if (mean_kept) mean_kept[0] = (float)((double)count / (double)p.B);
}

hipError_t launch_match_lambda(const Prob& p, const float* scores, int reduce, float k_target,
                               void* state, float* lambda, float* mean_kept, hipStream_t s)
{
    MatchState* st = static_cast<MatchState*>(state);
    const int chunks = (p.max_cands + kMatchChunk - 1) / kMatchChunk;
    const dim3 grid(p.B, chunks > 0 ? chunks : 1);
    const dim3 block(kMatchThreads);
    hipError_t e = launch(match_init_kernel, dim3(1), block, 0, s, p, k_target, st);
    if (e != hipSuccess) return e;
    if (chunks > 0) {
        if ((e = launch(match_hist_kernel<0>, grid, block, 0, s, p, scores, reduce, st)) != hipSuccess ||
            (e = launch(match_hist_kernel<1>, grid, block, 0, s, p, scores, reduce, st)) != hipSuccess ||
            (e = launch(match_hist_kernel<2>, grid, block, 0, s, p, scores, reduce, st)) != hipSuccess ||
            (e = launch(match_hist_kernel<3>, grid, block, 0, s, p, scores, reduce, st)) != hipSuccess)
            return e;
    }
    return launch(match_count_kernel, grid, block, 0, s, p, scores, reduce, k_target, st, lambda,
                  mean_kept);
}

}  // namespace occam
