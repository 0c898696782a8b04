// Anchor path for one anchor row per sample (the CLS row of Stage I,
// Eq. EQ:CLS), steps 1-2: logits of the CLS query against [registers ;
// visual] keys (Eq. (1)), per-head softmax and the head mean (Appendix,
// "Stage-I pruning": the vision map is averaged over heads).
//
// With a single query row the contraction is a matrix-vector product: every
// key byte is used once, so the work is bound by HBM and runs on the VALU.
//
// cls_logits  grid (key chunk, sample): streams the chunk's key rows with
//             coalesced 16-byte loads (a wave reads one key row per step,
//             lane L reading bytes [16L, 16L+16) of it), forms per-16-byte
//             partial dot products against the query held in LDS, sums them
//             per (key, head), writes the scaled logits to the workspace and
//             the chunk's per-head (max, sum exp) pair.
// cls_stream / cls_stream_run  the same for H == Hkv with the query in registers:
//             lanes own fixed 16-byte slots of the key rows (heads padded to a power
//             of two of lanes), or, for 16 heads of 5-7 or 9 chunks, contiguous runs
//             of four key rows with the per-(row, head) sums formed through LDS.
// cls_scores  grid (key chunk, sample): merges the per-chunk pairs of the
//             sample into the softmax normaliser of every head (fixed order),
//             then score(s) = (1/H) sum_h exp(l[s,h] - m_h) / z_h.
// Both kernels use fixed reduction orders, so results are run-to-run
// identical.
#include "occam_internal.hpp"

namespace occam {

// exp for the softmax of the one-row path.  bfloat16 inputs are checked to 2e-2
// relative, so the hardware exp2 (v_exp_f32 on x*log2(e), a few 1e-7 relative error
// at the logit ranges seen here) suffices; float32 inputs are checked to 1e-5 and use
// the device library's correctly rounded-to-1-ulp expf.
template <bool BF16>
__device__ __forceinline__ float cls_exp(float x) {
    return BF16 ? __builtin_amdgcn_exp2f(x * kLog2e) : expf(x);
}

template <bool BF16>
__global__ __launch_bounds__(kClsThreads) void cls_logits_kernel(
    Prob p, const void* __restrict__ qv, const void* __restrict__ kv,
    float* __restrict__ logits, float2* __restrict__ stats, int kpw, int nchunks, Finish fin)
{
    extern __shared__ float smem[];
    constexpr int CE = BF16 ? 8 : 4;            // elements per 16-byte chunk
    const int c = blockIdx.x, b = blockIdx.y;
    if (c == 0 && b == 0) clear_done(fin, p.B);  // counters of the cls_scores launch
    const int S = keys_of(p, b);
    const int s0 = c * kpw;
    if (s0 >= S) return;                        // uniform over the workgroup
    const int nk = min(kpw, S - s0);
    const int H = p.H, Hkv = p.Hkv, d = p.d, group = H / Hkv;
    const int NC = d / CE;                      // chunks per key head
    const int CPK = NC * Hkv;                   // chunks per key row
    float* qs = smem;                           // [H][d]
    int* tab = reinterpret_cast<int*>(qs + H * d);      // [CPK]: (g << 16) | part
    float* part = reinterpret_cast<float*>(tab + CPK);  // [nk][H][NC]
    float* lg = part + kpw * H * NC;                    // [nk][H]
    float* red = lg + kpw * H;                          // [2 * blockDim]

    const int qrow = q_begin(p, b);
    if (BF16) {
        const uint16_t* q16 = static_cast<const uint16_t*>(qv) + (size_t)qrow * H * d;
        for (int i = threadIdx.x; i < H * d; i += blockDim.x)
            qs[i] = __uint_as_float(static_cast<uint32_t>(q16[i]) << 16);
    } else {
        const float* q32 = static_cast<const float*>(qv) + (size_t)qrow * H * d;
        for (int i = threadIdx.x; i < H * d; i += blockDim.x) qs[i] = q32[i];
    }
    for (int ci = threadIdx.x; ci < CPK; ci += blockDim.x)
        tab[ci] = ((ci / NC) << 16) | (ci % NC);
    __syncthreads();

    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int nwave = blockDim.x / kWave;
    const size_t row_elems = (size_t)Hkv * d;
    const char* kbase = static_cast<const char*>(kv) +
                        ((size_t)k_begin(p, b) + s0) * row_elems * (BF16 ? 2 : 4);
    const size_t row_bytes = row_elems * (BF16 ? 2 : 4);
    for (int key = wave; key < nk; key += nwave) {
        const u32x4* krow = reinterpret_cast<const u32x4*>(kbase + (size_t)key * row_bytes);
        for (int ci = lane; ci < CPK; ci += kWave) {
            const u32x4 w = __builtin_nontemporal_load(krow + ci);
            float kf[CE];
            if constexpr (BF16) {
                kf[0] = bf16_lo(w.x); kf[1] = bf16_hi(w.x);
                kf[2] = bf16_lo(w.y); kf[3] = bf16_hi(w.y);
                kf[4] = bf16_lo(w.z); kf[5] = bf16_hi(w.z);
                kf[6] = bf16_lo(w.w); kf[7] = bf16_hi(w.w);
            } else {
                kf[0] = __uint_as_float(w.x); kf[1] = __uint_as_float(w.y);
                kf[2] = __uint_as_float(w.z); kf[3] = __uint_as_float(w.w);
            }
            const int tg = tab[ci];
            const int g = tg >> 16, pc = tg & 0xffff;
            for (int i = 0; i < group; ++i) {
                const int h = g * group + i;
                const float* qq = qs + h * d + pc * CE;
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < CE; ++e) acc = fmaf(qq[e], kf[e], acc);
                part[(key * H + h) * NC + pc] = acc;
            }
        }
    }
    __syncthreads();

    float* lout = logits + ((size_t)k_begin(p, b) + s0) * H;
    for (int i = threadIdx.x; i < nk * H; i += blockDim.x) {
        const float* pp = part + i * NC;
        float acc = 0.f;
        for (int e = 0; e < NC; ++e) acc += pp[e];
        const float l = acc * p.scale;
        lg[i] = l;
        lout[i] = l;
    }
    __syncthreads();

    // Per-head (max, sum exp) of this chunk: P threads per head, each over a strided
    // subset of the chunk's keys, then a fixed-order merge of the P partials.
    const int P = blockDim.x / H;                   // >= 1 (H <= 64)
    const int hh = threadIdx.x % H, j0 = threadIdx.x / H;
    float m = -INFINITY;
    if (j0 < P)
        for (int key = j0; key < nk; key += P) m = fmaxf(m, lg[key * H + hh]);
    red[threadIdx.x] = m;
    __syncthreads();
    if (threadIdx.x < H) {
        float mm = red[threadIdx.x];
        for (int j = 1; j < P; ++j) mm = fmaxf(mm, red[j * H + threadIdx.x]);
        red[blockDim.x + threadIdx.x] = mm;
    }
    __syncthreads();
    const float mh = red[blockDim.x + hh];
    float z = 0.f;
    if (j0 < P)
        for (int key = j0; key < nk; key += P) z += cls_exp<BF16>(lg[key * H + hh] - mh);
    __syncthreads();
    red[threadIdx.x] = z;
    __syncthreads();
    if (threadIdx.x < H) {
        float zz = red[threadIdx.x];
        for (int j = 1; j < P; ++j) zz += red[j * H + threadIdx.x];
        stats[((size_t)b * nchunks + c) * H + threadIdx.x] = make_float2(mh, zz);
    }
}

// Sum over aligned groups of N lanes (N = 1, 2, 4, 8, 16), every lane of a group
// receiving the group's sum; DPP moves inside 16-lane rows, fixed order.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int N>
__device__ __forceinline__ float lane_group_sum(float x) {
    if constexpr (N >= 2) x += dpp_f32<0xB1>(x);     // quad_perm [1,0,3,2]
    if constexpr (N >= 4) x += dpp_f32<0x4E>(x);     // quad_perm [2,3,0,1]
    if constexpr (N >= 8) x += dpp_f32<0x141>(x);    // row_half_mirror
    if constexpr (N >= 16) x += dpp_f32<0x140>(x);   // row_mirror
    return x;
}

// Streaming form of cls_logits for H == Hkv with nc <= 16 16-byte chunks per head,
// NC = nc rounded up to a power of two lanes per head and NJ = H * NC / 64 wave loads
// per key row.  Lane l owns the lane slots ci = l + 64 j of every key row (head
// ci / NC, chunk ci % NC; a slot past the head's nc chunks rereads its last chunk
// against a zero query) and keeps the matching query elements in registers.  Each wave walks its keys KB at a time (KB rows of
// coalesced 1 KB loads in flight), reduces the per-chunk partial dot products over
// the NC lanes of a head with DPP, writes the scaled logit and folds it into a
// per-head online (max, sum exp) pair held by those lanes.  The four waves' pairs are
// merged in a fixed order at the end.
template <bool BF16, int NC, int NJ>
__global__ __launch_bounds__(kClsThreads) void cls_stream_kernel(
    Prob p, const void* __restrict__ qv, const void* __restrict__ kv,
    float* __restrict__ logits, float2* __restrict__ stats, int kpw, int nchunks, int nc,
    Finish fin)
{
    constexpr int CE = BF16 ? 8 : 4;                 // elements per 16-byte chunk
    constexpr int KB = 4;                            // key rows in flight per wave
    constexpr int NW = kClsThreads / kWave;
    __shared__ float red_m[NW][64], red_z[NW][64];
    const int c = blockIdx.x, b = blockIdx.y;
    if (c == 0 && b == 0) clear_done(fin, p.B);      // counters of the cls_scores launch
    const int S = keys_of(p, b);
    const int s0 = c * kpw;
    if (s0 >= S) return;                             // uniform over the workgroup
    const int nk = min(kpw, S - s0);
    const int H = p.H, d = p.d;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float scale = p.scale;

    // Query elements of this lane's chunks, as float (zero for slots past nc), and the
    // chunk each slot loads within a key row.
    float qf[NJ][CE];
    int koff[NJ];
    const int qrow = q_begin(p, b);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int ci = lane + 64 * j;
        const int h = ci / NC, part = ci % NC;
        const int e0 = min(part, nc - 1) * CE;
        koff[j] = h * nc + min(part, nc - 1);
        if (part >= nc) {
#pragma unroll
            for (int e = 0; e < CE; ++e) qf[j][e] = 0.f;
        } else if (BF16) {
            const uint16_t* q16 = static_cast<const uint16_t*>(qv) + ((size_t)qrow * H + h) * d + e0;
#pragma unroll
            for (int e = 0; e < CE; ++e) qf[j][e] = __uint_as_float(static_cast<uint32_t>(q16[e]) << 16);
        } else {
            const float* q32 = static_cast<const float*>(qv) + ((size_t)qrow * H + h) * d + e0;
#pragma unroll
            for (int e = 0; e < CE; ++e) qf[j][e] = q32[e];
        }
    }

    float m[NJ], z[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) { m[j] = -INFINITY; z[j] = 0.f; }
    const int rowc = H * nc;                         // 16-byte chunks per key row
    const u32x4* kbase = static_cast<const u32x4*>(kv) + ((size_t)k_begin(p, b) + s0) * rowc;
    float* lout = logits + ((size_t)k_begin(p, b) + s0) * H;

    for (int k0 = wave * KB; k0 < nk; k0 += NW * KB) {
        u32x4 w[KB][NJ];
#pragma unroll
        for (int i = 0; i < KB; ++i) {
            const int key = min(k0 + i, nk - 1);     // clamped rows are loaded, not used
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                w[i][j] = __builtin_nontemporal_load(kbase + (size_t)key * rowc + koff[j]);
        }
#pragma unroll
        for (int i = 0; i < KB; ++i) {
            const bool valid = k0 + i < nk;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                float kf[CE];
                if constexpr (BF16) {
                    kf[0] = bf16_lo(w[i][j].x); kf[1] = bf16_hi(w[i][j].x);
                    kf[2] = bf16_lo(w[i][j].y); kf[3] = bf16_hi(w[i][j].y);
                    kf[4] = bf16_lo(w[i][j].z); kf[5] = bf16_hi(w[i][j].z);
                    kf[6] = bf16_lo(w[i][j].w); kf[7] = bf16_hi(w[i][j].w);
                } else {
                    kf[0] = __uint_as_float(w[i][j].x); kf[1] = __uint_as_float(w[i][j].y);
                    kf[2] = __uint_as_float(w[i][j].z); kf[3] = __uint_as_float(w[i][j].w);
                }
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < CE; ++e) acc = fmaf(qf[j][e], kf[e], acc);
                const float l = lane_group_sum<NC>(acc) * scale;
                if (valid) {
                    const int ci = lane + 64 * j;
                    if (ci % NC == 0) lout[(size_t)(k0 + i) * H + ci / NC] = l;
                    if (l > m[j]) {
                        z[j] = z[j] * cls_exp<BF16>(m[j] - l) + 1.f;
                        m[j] = l;
                    } else {
                        z[j] += cls_exp<BF16>(l - m[j]);
                    }
                }
            }
        }
    }

    // Fixed-order merge of the waves' pairs (a wave with no keys holds (-inf, 0)).
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int ci = lane + 64 * j;
        if (ci % NC == 0) { red_m[wave][ci / NC] = m[j]; red_z[wave][ci / NC] = z[j]; }
    }
    __syncthreads();
    for (int h = threadIdx.x; h < H; h += kClsThreads) {
        float mm = red_m[0][h], zz = red_z[0][h];
        for (int w2 = 1; w2 < NW; ++w2) {
            const float mo = red_m[w2][h], zo = red_z[w2][h];
            const float mn = fmaxf(mm, mo);
            if (mn != -INFINITY) {
                zz = zz * cls_exp<BF16>(mm - mn) + zo * cls_exp<BF16>(mo - mn);
                mm = mn;
            }
        }
        stats[((size_t)b * nchunks + c) * H + h] = make_float2(mm, zz);
    }
}

// Streaming form for 16 heads whose chunk count NCK is not a power of two (d = 72 in
// bfloat16: nine 16-byte chunks per head).  Padding a head to 16 lanes, as
// cls_stream_kernel does, would have 7 of every 16 lanes reread a chunk; instead a wave
// reads KB = 4 consecutive key rows as one contiguous run of 4 * 16 * NCK chunks, NCK
// coalesced 1 KB loads per lane with no lane idle, and forms each chunk's partial dot
// product.  The partials go to the wave's own LDS row, and lane L = (row r = L / 16,
// head h = L % 16) adds the NCK partials of its (row, head) in chunk order, writes the
// scaled logit and folds it into its online (max, sum exp) pair; the 16 pairs of a head
// (4 waves x 4 rows) are merged in a fixed order at the end.
template <bool BF16, int NCK>
__global__ __launch_bounds__(kClsThreads) void cls_stream_run_kernel(
    Prob p, const void* __restrict__ qv, const void* __restrict__ kv,
    float* __restrict__ logits, float2* __restrict__ stats, int kpw, int nchunks, Finish fin)
{
    constexpr int CE = BF16 ? 8 : 4;                 // elements per 16-byte chunk
    constexpr int HH = 16;                           // heads: 4 rows x 16 heads = 64 lanes
    constexpr int KB = 4;                            // key rows per wave step
    constexpr int ROWC = HH * NCK;                   // 16-byte chunks per key row
    constexpr int NJ = KB * ROWC / kWave;            // loads per lane per step (= NCK)
    static_assert((KB * ROWC) % kWave == 0, "a run of KB rows fills whole wave loads");
    constexpr int NW = kClsThreads / kWave;
    __shared__ float part[NW][KB * ROWC];
    __shared__ float red_m[NW][kWave], red_z[NW][kWave];
    const int c = blockIdx.x, b = blockIdx.y;
    if (c == 0 && b == 0) clear_done(fin, p.B);      // counters of the cls_scores launch
    const int S = keys_of(p, b);
    const int s0 = c * kpw;
    if (s0 >= S) return;                             // uniform over the workgroup
    const int nk = min(kpw, S - s0);
    const int d = p.d;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float scale = p.scale;

    // Query elements of the chunk each load of this lane reads (the same for every run:
    // chunk cc = 64 j + lane of the run is column cc % ROWC of its row).
    float qf[NJ][CE];
    const int qrow = q_begin(p, b);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int col = (j * kWave + lane) % ROWC;
        const int h = col / NCK, e0 = (col % NCK) * CE;
        if constexpr (BF16) {
            const uint16_t* q16 = static_cast<const uint16_t*>(qv) + ((size_t)qrow * HH + h) * d + e0;
#pragma unroll
            for (int e = 0; e < CE; ++e) qf[j][e] = __uint_as_float(static_cast<uint32_t>(q16[e]) << 16);
        } else {
            const float* q32 = static_cast<const float*>(qv) + ((size_t)qrow * HH + h) * d + e0;
#pragma unroll
            for (int e = 0; e < CE; ++e) qf[j][e] = q32[e];
        }
    }

    const int rr = lane / HH, hh = lane % HH;        // this lane's (row of the run, head)
    float m = -INFINITY, z = 0.f;
    const u32x4* kbase = static_cast<const u32x4*>(kv) + ((size_t)k_begin(p, b) + s0) * ROWC;
    float* lout = logits + ((size_t)k_begin(p, b) + s0) * HH;
    float* prt = part[wave];

    for (int k0 = wave * KB; k0 < nk; k0 += NW * KB) {
        u32x4 w[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int cc = j * kWave + lane;
            const int key = min(k0 + cc / ROWC, nk - 1);    // clamped rows are loaded, not used
            w[j] = __builtin_nontemporal_load(kbase + (size_t)key * ROWC + cc % ROWC);
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            float kf[CE];
            if constexpr (BF16) {
                kf[0] = bf16_lo(w[j].x); kf[1] = bf16_hi(w[j].x);
                kf[2] = bf16_lo(w[j].y); kf[3] = bf16_hi(w[j].y);
                kf[4] = bf16_lo(w[j].z); kf[5] = bf16_hi(w[j].z);
                kf[6] = bf16_lo(w[j].w); kf[7] = bf16_hi(w[j].w);
            } else {
                kf[0] = __uint_as_float(w[j].x); kf[1] = __uint_as_float(w[j].y);
                kf[2] = __uint_as_float(w[j].z); kf[3] = __uint_as_float(w[j].w);
            }
            float acc = 0.f;
#pragma unroll
            for (int e = 0; e < CE; ++e) acc = fmaf(qf[j][e], kf[e], acc);
            prt[j * kWave + lane] = acc;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        float l = 0.f;
#pragma unroll
        for (int sc = 0; sc < NCK; ++sc) l += prt[rr * ROWC + hh * NCK + sc];
        l *= scale;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();             // reads done before the next step's writes
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (k0 + rr < nk) {
            lout[(size_t)(k0 + rr) * HH + hh] = l;
            if (l > m) {
                z = z * cls_exp<BF16>(m - l) + 1.f;
                m = l;
            } else {
                z += cls_exp<BF16>(l - m);
            }
        }
    }

    // Fixed-order merge of the 16 pairs of each head (waves, then rows; (-inf, 0) for a
    // row slot that saw no key).
    red_m[wave][lane] = m;
    red_z[wave][lane] = z;
    __syncthreads();
    if (threadIdx.x < HH) {
        const int h = threadIdx.x;
        float mm = -INFINITY, zz = 0.f;
        for (int w2 = 0; w2 < NW; ++w2)
            for (int r = 0; r < KB; ++r) {
                const float mo = red_m[w2][r * HH + h], zo = red_z[w2][r * HH + h];
                const float mn = fmaxf(mm, mo);
                if (mn != -INFINITY) {
                    zz = zz * cls_exp<BF16>(mm - mn) + zo * cls_exp<BF16>(mo - mn);
                    mm = mn;
                }
            }
        stats[((size_t)b * nchunks + c) * HH + h] = make_float2(mm, zz);
    }
}

// score(s) of one key from its H logits and the per-head normalisers: the one
// expression both the scores and the per-chunk threshold use, so that they agree bit for
// bit.
template <bool BF16>
__device__ __forceinline__ float cls_key_score(const float* l, int H, const float* mh,
                                               const float* izh) {
    float acc = 0.f;
    for (int h = 0; h < H; ++h) acc += cls_exp<BF16>(l[h] - mh[h]) * izh[h];
    return acc * (1.f / (float)H);
}

// With fin.chunk_cnt (occam_prune) every workgroup also applies the threshold to its own
// chunk and compacts the chunk's survivors: tau_b = lambda * reduce(register scores), the
// register scores formed from the register keys' logits exactly as the scores are (so tau
// has the threshold kernel's bits), then a ballot + mbcnt compaction of the chunk's
// visual keys (one key per thread) with an LDS scan of the wave counts.  Chunks past the
// sample's keys write a zero count.
template <bool BF16>
__global__ __launch_bounds__(kClsThreads) void cls_scores_kernel(
    Prob p, const float* __restrict__ logits, const float2* __restrict__ stats,
    const float* __restrict__ row_lse, float* __restrict__ scores, int kpw, int nchunks,
    Finish fin)
{
    __shared__ float red_m[kClsThreads], red_z[kClsThreads];
    __shared__ float mh[64], izh[64];
    __shared__ float regs[32];
    __shared__ int wcnt[kClsThreads / kWave];
    const int c = blockIdx.x, b = blockIdx.y;
    const int S = keys_of(p, b);
    const int s0 = c * kpw;
    if (s0 >= S) {
        if (fin.chunk_cnt && threadIdx.x == 0) fin.chunk_cnt[(size_t)b * nchunks + c] = 0;
        return;
    }
    const int nk = min(kpw, S - s0);
    const int H = p.H;
    const int nch = (S + kpw - 1) / kpw;
    if (row_lse) {
        for (int h = threadIdx.x; h < H; h += blockDim.x) {
            mh[h] = row_lse[(size_t)q_begin(p, b) * H + h];
            izh[h] = 1.f;
        }
    } else {
        // Merge the per-chunk (max, sum) pairs of the sample: P threads per head, each a
        // strided subset of chunks (loaded PF at a time, so that long samples do not wait
        // for one load after another), then a fixed-order merge of the P partials.
        constexpr int PF = 8;
        const int P = blockDim.x / H;
        const int hh = threadIdx.x % H, j0 = threadIdx.x / H;
        float m = -INFINITY, z = 0.f;
        if (j0 < P) {
            const float2* st = stats + (size_t)b * nchunks * H + hh;
            for (int j = j0; j < nch; j += PF * P) {
                float2 v[PF];
#pragma unroll
                for (int u = 0; u < PF; ++u)
                    v[u] = j + u * P < nch ? st[(size_t)(j + u * P) * H] : make_float2(0.f, 0.f);
#pragma unroll
                for (int u = 0; u < PF; ++u) {
                    if (j + u * P >= nch) break;
                    const float mn = fmaxf(m, v[u].x);
                    z = z * cls_exp<BF16>(m - mn) + v[u].y * cls_exp<BF16>(v[u].x - mn);
                    m = mn;
                }
            }
        }
        red_m[threadIdx.x] = m;
        red_z[threadIdx.x] = z;
        __syncthreads();
        if (threadIdx.x < H) {
            float mm = red_m[threadIdx.x], zz = red_z[threadIdx.x];
            for (int j = 1; j < P; ++j) {
                const float mo = red_m[j * H + threadIdx.x], zo = red_z[j * H + threadIdx.x];
                const float mn = fmaxf(mm, mo);
                if (mn != -INFINITY) {
                    zz = zz * cls_exp<BF16>(mm - mn) + zo * cls_exp<BF16>(mo - mn);
                    mm = mn;
                }
            }
            mh[threadIdx.x] = mm;
            izh[threadIdx.x] = 1.f / zz;
        }
    }
    __syncthreads();
    const float* lrow = logits + ((size_t)k_begin(p, b) + s0) * H;
    float* out = scores + k_begin(p, b) + s0;
    float mine = 0.f;                            // this thread's key (one key per thread)
    for (int key = threadIdx.x; key < nk; key += blockDim.x) {
        mine = cls_key_score<BF16>(lrow + (size_t)key * H, H, mh, izh);
        out[key] = mine;
    }
    if (!fin.chunk_cnt) return;
    const int R = p.R;
    if (threadIdx.x < R)
        regs[threadIdx.x] = cls_key_score<BF16>(logits + ((size_t)k_begin(p, b) + threadIdx.x) * H,
                                                H, mh, izh);
    __syncthreads();
    const float tau = fin.lambda * reg_reduce(regs, R, fin.reduce);
    if (c == 0 && threadIdx.x == 0 && fin.tau) fin.tau[b] = tau;
    const int key = s0 + threadIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const bool keep = (int)threadIdx.x < nk && key >= R && mine >= tau;
    const unsigned long long m = __ballot(keep);
    const int below = (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
    if (lane == 0) wcnt[wave] = __popcll(m);
    __syncthreads();
    int base = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kClsThreads / kWave; ++w) {
        base += w < wave ? wcnt[w] : 0;
        total += wcnt[w];
    }
    const size_t list = (size_t)b * nchunks + c;
    if (keep) fin.chunk_slot[list * kpw + base + below] = key - R;
    if (threadIdx.x == 0) {
        fin.chunk_cnt[list] = total;
        if (total) atomicAdd(fin.count + b, total);
    }
}

static size_t cls_logits_smem(const Prob& p, int bf16, int kpw) {
    const int NC = p.d / (bf16 ? 8 : 4);
    return sizeof(float) * ((size_t)p.H * p.d + (size_t)NC * p.Hkv + (size_t)kpw * p.H * NC +
                            (size_t)kpw * p.H + 2 * (size_t)kClsThreads);
}

template <bool BF16, int NC>
static hipError_t cls_stream_launch(const Prob& p, const void* q, const void* k, float* logits,
                                    float2* stats, int kpw, const Finish& fin, hipStream_t s) {
    const int nc = p.d * (BF16 ? 2 : 4) / 16;
    const int nchunks = (p.R + p.max_cands + kpw - 1) / kpw;
    dim3 grid(nchunks, p.B);
    const dim3 blk(kClsThreads);
    switch (NC * p.Hkv / 64) {
    case 1: return launch(cls_stream_kernel<BF16, NC, 1>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, nc, fin);
    case 2: return launch(cls_stream_kernel<BF16, NC, 2>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, nc, fin);
    case 3: return launch(cls_stream_kernel<BF16, NC, 3>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, nc, fin);
    case 4: return launch(cls_stream_kernel<BF16, NC, 4>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, nc, fin);
    default: return hipErrorInvalidValue;
    }
}

template <bool BF16>
static hipError_t cls_stream_nc_launch(const Prob& p, int nc, const void* q, const void* k,
                                       float* logits, float2* stats, int kpw, const Finish& fin,
                                       hipStream_t s) {
    switch (nc) {
    case 1: return cls_stream_launch<BF16, 1>(p, q, k, logits, stats, kpw, fin, s);
    case 2: return cls_stream_launch<BF16, 2>(p, q, k, logits, stats, kpw, fin, s);
    case 4: return cls_stream_launch<BF16, 4>(p, q, k, logits, stats, kpw, fin, s);
    case 8: return cls_stream_launch<BF16, 8>(p, q, k, logits, stats, kpw, fin, s);
    case 16: return cls_stream_launch<BF16, 16>(p, q, k, logits, stats, kpw, fin, s);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_cls_logits(const Prob& p, int bf16, const void* q, const void* k,
                             float* logits, float2* stats, int kpw, const Finish& fin,
                             hipStream_t s)
{
    if (bf16 && p.H == 16 && p.Hkv == 16 && (p.d == 72 || p.d == 40 || p.d == 48 || p.d == 56)) {
        // 16 heads of 9 (5, 6, 7) chunks: contiguous runs of four key rows.
        const int nchunks = (p.R + p.max_cands + kpw - 1) / kpw;
        const dim3 grid(nchunks, p.B), blk(kClsThreads);
        switch (p.d) {
        case 40: return launch(cls_stream_run_kernel<true, 5>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, fin);
        case 48: return launch(cls_stream_run_kernel<true, 6>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, fin);
        case 56: return launch(cls_stream_run_kernel<true, 7>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, fin);
        default: return launch(cls_stream_run_kernel<true, 9>, grid, blk, 0, s, p, q, k, logits, stats, kpw, nchunks, fin);
        }
    }
    const int nc = cls_stream_nc(p.H, p.Hkv, p.d, bf16 ? 2 : 4);
    if (nc) {
        return bf16 ? cls_stream_nc_launch<true>(p, nc, q, k, logits, stats, kpw, fin, s)
                    : cls_stream_nc_launch<false>(p, nc, q, k, logits, stats, kpw, fin, s);
    }
    const int nchunks = (p.R + p.max_cands + kpw - 1) / kpw;
    dim3 grid(nchunks, p.B);
    const size_t smem = cls_logits_smem(p, bf16, kpw);
    if (bf16)
        return launch(cls_logits_kernel<true>, grid, dim3(kClsThreads), smem, s, p, q, k, logits,
                      stats, kpw, nchunks, fin);
    return launch(cls_logits_kernel<false>, grid, dim3(kClsThreads), smem, s, p, q, k, logits,
                  stats, kpw, nchunks, fin);
}

hipError_t launch_cls_scores(const Prob& p, int bf16, const float* logits, const float2* stats,
                             const float* row_lse, float* scores, int kpw, const Finish& fin,
                             hipStream_t s)
{
    const int nchunks = (p.R + p.max_cands + kpw - 1) / kpw;
    dim3 grid(nchunks, p.B);
    const size_t smem = 0;
    if (bf16)
        return launch(cls_scores_kernel<true>, grid, dim3(kClsThreads), smem, s, p, logits, stats,
                      row_lse, scores, kpw, nchunks, fin);
    return launch(cls_scores_kernel<false>, grid, dim3(kClsThreads), smem, s, p, logits, stats,
                  row_lse, scores, kpw, nchunks, fin);
}

}  // namespace occam
