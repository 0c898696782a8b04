// Anchor path for several anchor rows per sample (the text rows of Stage II,
// Eq. text_scoring), steps 1-2, on the gfx950 matrix cores.
//
// For T text rows, H heads and R+N keys the logits are a T x (R+N) x d
// contraction per head, done with v_mfma_f32_32x32x16_bf16.  The MFMA's A
// operand is a block of 32 keys and its B operand a block of 32 text rows, so
// each lane of the accumulator holds 16 keys of ONE text row: reductions over
// keys (the softmax statistics) stay inside a lane, and the head sum is an
// element-wise accumulation in registers.
//
// Every (row, head) softmax needs its normaliser before the head mean can be
// formed, so the path has two passes over the keys:
//
// text_stats  grid (row block of 128, head, sample).  Each wave owns every
//             4th block of 32 keys, keeps the 128 query rows of the head as
//             MFMA B fragments in registers, and maintains an online
//             (max, sum 2^x) pair per row; pairs are merged across the two
//             lane halves and the 4 waves in a fixed order.  Writes the base-2
//             log-sum-exp lse2[row, head] of x = logit * log2(e).
// text_score  grid (block of 128 keys, sample).  Each wave owns 32 keys.  For
//             every head the 128 x d query tile is staged in LDS (the next
//             head's tile is prefetched into registers during the current
//             head's MFMAs) and p = 2^(x - lse2) is accumulated over heads per
//             (key, row).  Afterwards the row reduction of Eq. text_scoring is
//             applied: max over rows for visual keys, mean for registers,
//             both over the head mean (1/H).  Rows beyond T_b carry
//             lse2 = +inf and so contribute exactly 0.
//
// When the caller supplies its own natural-log normaliser (row_lse), text_stats
// is skipped and text_score reads lse2 = row_lse * log2(e).
#include "occam_internal.hpp"

namespace occam {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
    return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row (key) index, inside a 32-key block, of accumulator element r of a lane
// whose upper-half flag is hi (lanes 32..63): 8*(r/4) + 4*hi + r%4.
__device__ __forceinline__ int acc_key(int r, int hi) { return 8 * (r >> 2) + 4 * hi + (r & 3); }

// Merge two online-softmax pairs (max, sum 2^(x - max)).
__device__ __forceinline__ void merge_pair(float& m, float& z, float mo, float zo) {
    const float mn = fmaxf(m, mo);
    if (mn == -INFINITY) return;
    z = z * __builtin_amdgcn_exp2f(m - mn) + zo * __builtin_amdgcn_exp2f(mo - mn);
    m = mn;
}

template <int DS>
__global__ __launch_bounds__(kTxtThreads) void text_stats_kernel(
    Prob p, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    float* __restrict__ lse2)
{
    __shared__ float red_m[kTxtThreads / kWave][kTxtRows];
    __shared__ float red_z[kTxtThreads / kWave][kTxtRows];
    const int tblk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int T = rows_of(p, b);
    const int t0 = tblk * kTxtRows;
    if (t0 >= T) return;
    const int S = keys_of(p, b);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int hi = lane >> 5, lo = lane & 31;
    const int H = p.H, Hkv = p.Hkv, d = p.d;
    const int g = h / (H / Hkv);
    const int nsb = min(4, (T - t0 + 31) >> 5);
    const int qb = q_begin(p, b), kb0 = k_begin(p, b);
    const float c2 = p.scale * kLog2e;

    bf16x8 qf[4][DS];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) {
        const int t = t0 + sb * 32 + lo;
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) {
            const int e = kk * 16 + hi * 8;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (t < T && e < d) v = load16(q + ((size_t)(qb + t) * H + h) * d + e);
            qf[sb][kk] = as_bf16x8(v);
        }
    }

    float m[4], z[4];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) { m[sb] = -INFINITY; z[sb] = 0.f; }

    const int nkb = (S + 31) >> 5;
    const uint16_t* kbase = k + ((size_t)kb0 * Hkv + g) * d;
    const size_t kstride = (size_t)Hkv * d;
    auto load_k = [&](int kbi, u32x4 (&kf)[DS]) {
        const int key = kbi * 32 + lo;
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) {
            const int e = kk * 16 + hi * 8;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (key < S && e < d) v = load16(kbase + (size_t)key * kstride + e);
            kf[kk] = v;
        }
    };

    u32x4 kcur[DS], knext[DS];
    int kbi = wave;
    if (kbi < nkb) load_k(kbi, kcur);
    for (; kbi < nkb; kbi += 4) {
        if (kbi + 4 < nkb) load_k(kbi + 4, knext);
        const int nvalid = S - kbi * 32;
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            if (sb >= nsb) break;
            f32x16 acc = {};
#pragma unroll
            for (int kk = 0; kk < DS; ++kk) acc = mfma32(as_bf16x8(kcur[kk]), qf[sb][kk], acc);
            float mx = -INFINITY;
            if (nvalid >= 32) {
#pragma unroll
                for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[r]);
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (acc_key(r, hi) < nvalid) mx = fmaxf(mx, acc[r]);
            }
            if (mx == -INFINITY) continue;
            const float mn = fmaxf(m[sb], mx * c2);
            float sum = 0.f;
            if (nvalid >= 32) {
#pragma unroll
                for (int r = 0; r < 16; ++r) sum += __builtin_amdgcn_exp2f(fmaf(acc[r], c2, -mn));
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (acc_key(r, hi) < nvalid) sum += __builtin_amdgcn_exp2f(fmaf(acc[r], c2, -mn));
            }
            z[sb] = z[sb] * __builtin_amdgcn_exp2f(m[sb] - mn) + sum;
            m[sb] = mn;
        }
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) kcur[kk] = knext[kk];
    }

    // Merge the two lane halves (same rows, different keys), then the waves.
#pragma unroll
    for (int sb = 0; sb < 4; ++sb) {
        const float mo = __shfl_xor(m[sb], 32);
        const float zo = __shfl_xor(z[sb], 32);
        merge_pair(m[sb], z[sb], mo, zo);
        if (hi == 0) {
            red_m[wave][sb * 32 + lo] = m[sb];
            red_z[wave][sb * 32 + lo] = z[sb];
        }
    }
    __syncthreads();
    if (threadIdx.x < kTxtRows) {
        const int i = threadIdx.x;
        float mm = red_m[0][i], zz = red_z[0][i];
        for (int w = 1; w < kTxtThreads / kWave; ++w) merge_pair(mm, zz, red_m[w][i], red_z[w][i]);
        const int t = t0 + i;
        if (t < T) lse2[(size_t)(qb + t) * H + h] = mm + __builtin_amdgcn_logf(zz);
    }
}

template <int DS>
__global__ __launch_bounds__(kTxtThreads) void text_score_kernel(
    Prob p, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const float* __restrict__ lse, int lse_natural, float* __restrict__ scores)
{
    constexpr int DP = DS * 16 + 8;             // padded LDS row (elements)
    constexpr int QCH = kTxtRows * DS * 2 / kTxtThreads;  // 16-byte Q chunks per thread
    extern __shared__ __attribute__((aligned(16))) char smem_raw[];
    uint16_t* qt = reinterpret_cast<uint16_t*>(smem_raw);                 // [128][DP]
    float* l2t = reinterpret_cast<float*>(smem_raw + kTxtRows * DP * 2);  // [H][128]

    const int c = blockIdx.x, b = blockIdx.y;
    const int S = keys_of(p, b);
    const int s_lo = c * kTxtKeysPerWg;
    if (s_lo >= S) return;
    const int T = rows_of(p, b);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hi = lane >> 5, lo = lane & 31;
    const int H = p.H, Hkv = p.Hkv, d = p.d, group = H / Hkv;
    const int qb = q_begin(p, b), kb0 = k_begin(p, b);
    const float c2 = p.scale * kLog2e;
    const int wkey0 = s_lo + wave * kTxtKeysPerWave;
    const bool wactive = wkey0 < S;
    const int R = p.R;

    auto load_q = [&](int hh, int t0, u32x4 (&qr)[QCH]) {
#pragma unroll
        for (int j = 0; j < QCH; ++j) {
            const int i = tid + j * kTxtThreads;
            const int row = i / (DS * 2), e = (i % (DS * 2)) * 8;
            const int t = t0 + row;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (t < T && e < d) v = load16(q + ((size_t)(qb + t) * H + hh) * d + e);
            qr[j] = v;
        }
    };
    auto store_q = [&](const u32x4 (&qr)[QCH]) {
#pragma unroll
        for (int j = 0; j < QCH; ++j) {
            const int i = tid + j * kTxtThreads;
            const int row = i / (DS * 2), e = (i % (DS * 2)) * 8;
            *reinterpret_cast<u32x4*>(qt + row * DP + e) = qr[j];
        }
    };
    auto load_k = [&](int gg, u32x4 (&kf)[DS]) {
        const int key = wkey0 + lo;
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) {
            const int e = kk * 16 + hi * 8;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (key < S && e < d) v = load16(k + ((size_t)(kb0 + key) * Hkv + gg) * d + e);
            kf[kk] = v;
        }
    };

    float vmax[16], rsum[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) { vmax[r] = 0.f; rsum[r] = 0.f; }

    for (int t0 = 0; t0 < T; t0 += kTxtRows) {
        const int nsb = min(4, (T - t0 + 31) >> 5);
        __syncthreads();  // previous row block is done with qt / l2t
        for (int i = tid; i < H * kTxtRows; i += kTxtThreads) {
            const int hh = i / kTxtRows, t = t0 + (i % kTxtRows);
            float v = INFINITY;
            if (t < T) {
                v = lse[(size_t)(qb + t) * H + hh];
                if (lse_natural) v *= kLog2e;
            }
            l2t[i] = v;
        }
        u32x4 qreg[QCH];
        u32x4 kcur[DS], knext[DS];
        load_q(0, t0, qreg);
        if (wactive) load_k(0, kcur);
        store_q(qreg);
        if (H > 1) load_q(1, t0, qreg);
        __syncthreads();

        float abar[4][16];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
            for (int r = 0; r < 16; ++r) abar[sb][r] = 0.f;

        for (int h = 0; h < H; ++h) {
            if (wactive) {
                if (h + 1 < H) load_k((h + 1) / group, knext);
#pragma unroll
                for (int sb = 0; sb < 4; ++sb) {
                    if (sb >= nsb) break;
                    f32x16 acc = {};
#pragma unroll
                    for (int kk = 0; kk < DS; ++kk) {
                        const u32x4 qv = *reinterpret_cast<const u32x4*>(
                            qt + (sb * 32 + lo) * DP + kk * 16 + hi * 8);
                        acc = mfma32(as_bf16x8(kcur[kk]), as_bf16x8(qv), acc);
                    }
                    const float l2 = l2t[h * kTxtRows + sb * 32 + lo];
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        abar[sb][r] += __builtin_amdgcn_exp2f(fmaf(acc[r], c2, -l2));
                }
#pragma unroll
                for (int kk = 0; kk < DS; ++kk) kcur[kk] = knext[kk];
            }
            __syncthreads();  // every wave is done reading head h's tile
            if (h + 1 < H) {
                store_q(qreg);
                if (h + 2 < H) load_q(h + 2, t0, qreg);
            }
            __syncthreads();
        }
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            if (sb >= nsb) break;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                vmax[r] = fmaxf(vmax[r], abar[sb][r]);
                rsum[r] += abar[sb][r];
            }
        }
    }

    // Row reduction across the 32 lanes that share a lane half (fixed order).
#pragma unroll
    for (int r = 0; r < 16; ++r) {
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) {
            vmax[r] = fmaxf(vmax[r], __shfl_xor(vmax[r], off));
            rsum[r] += __shfl_xor(rsum[r], off);
        }
    }
    if (wactive && lo == 0) {
        const float invH = 1.f / (float)H;
        const float invHT = 1.f / ((float)H * (float)T);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = wkey0 + acc_key(r, hi);
            if (key < S) scores[kb0 + key] = key < R ? rsum[r] * invHT : vmax[r] * invH;
        }
    }
}

template <int DS>
static hipError_t stats_ds(const Prob& p, const void* q, const void* k, float* lse2, hipStream_t s) {
    dim3 grid((p.max_rows + kTxtRows - 1) / kTxtRows, p.H, p.B);
    hipLaunchKernelGGL(text_stats_kernel<DS>, grid, dim3(kTxtThreads), 0, s, p,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), lse2);
    return hipGetLastError();
}

template <int DS>
static hipError_t score_ds(const Prob& p, const void* q, const void* k, const float* lse,
                           int lse_natural, float* scores, hipStream_t s) {
    dim3 grid((p.R + p.max_cands + kTxtKeysPerWg - 1) / kTxtKeysPerWg, p.B);
    const size_t smem = (size_t)kTxtRows * (DS * 16 + 8) * 2 + (size_t)p.H * kTxtRows * 4;
    hipLaunchKernelGGL(text_score_kernel<DS>, grid, dim3(kTxtThreads), smem, s, p,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), lse,
                       lse_natural, scores);
    return hipGetLastError();
}


hipError_t launch_text_stats(const Prob& p, const void* q, const void* k, float* lse2,
                             hipStream_t s) {
    const int ds = (p.d + 15) / 16;
#define OCCAM_STATS(DSV) stats_ds<DSV>(p, q, k, lse2, s)
    switch (ds) {
        case 1: return OCCAM_STATS(1); case 2: return OCCAM_STATS(2);
        case 3: return OCCAM_STATS(3); case 4: return OCCAM_STATS(4);
        case 5: return OCCAM_STATS(5); case 6: return OCCAM_STATS(6);
        case 7: return OCCAM_STATS(7); case 8: return OCCAM_STATS(8);
        default: return hipErrorInvalidValue;
    }
#undef OCCAM_STATS
}

hipError_t launch_text_score(const Prob& p, const void* q, const void* k, const float* lse,
                             int lse_natural, float* scores, hipStream_t s) {
    const int ds = (p.d + 15) / 16;
#define OCCAM_SCORE(DSV) score_ds<DSV>(p, q, k, lse, lse_natural, scores, s)
    switch (ds) {
        case 1: return OCCAM_SCORE(1); case 2: return OCCAM_SCORE(2);
        case 3: return OCCAM_SCORE(3); case 4: return OCCAM_SCORE(4);
        case 5: return OCCAM_SCORE(5); case 6: return OCCAM_SCORE(6);
        case 7: return OCCAM_SCORE(7); case 8: return OCCAM_SCORE(8);
        default: return hipErrorInvalidValue;
    }
#undef OCCAM_SCORE
}

}  // namespace occam
