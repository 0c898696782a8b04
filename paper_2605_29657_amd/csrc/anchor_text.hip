// Anchor path for several anchor rows per sample (the text rows of Stage II,
// Eq. text_scoring), steps 1-2, on the gfx950 matrix cores.
//
// For T text rows, H heads and R+N keys the logits are a T x (R+N) x d
// contraction per head, done with v_mfma_f32_32x32x16_bf16.  The MFMA's A
// operand is a block of 32 keys and its B operand a block of 32 text rows, so
// each lane of the accumulator holds 16 keys of ONE text row: reductions over
// keys (the softmax statistics) stay inside a lane, and the head sum is an
// element-wise accumulation in registers.  (The column-sum form below swaps the
// operands, so that a lane holds 16 rows of one key.)
//
// Every (row, head) softmax needs its normaliser before the head mean can be
// formed, so the path has two passes over the keys:
//
// text_stats  task (sample, head, group of 1, 2 or 4 row blocks of 128; groups only
//             when a sample has at most four row blocks[, key range]), XCD-aware; a
//             batch with few such tasks splits their keys into ranges whose tables
//             text_lse_merge combines.
//             One key stream consumed by four waves of 32 rows per row block (the
//             kernel also has a two-stream form of two 64-row waves each), so each
//             key block is copied once for every row block of the group; the
//             query rows of the head sit in
//             registers as MFMA B fragments, and a (reference, sum 2^(x - reference))
//             pair is kept per row: the reference is the first key block's maximum
//             and moves only when a block's sum would exceed 2^64, so a logit costs
//             a multiply-add, an exponential and an add (no running maximum); pairs
//             are merged across the two lane halves (and
//             streams) in a fixed order.  Key blocks reach LDS through direct global -> LDS
//             copies (a 2-stage ring per stream).  Writes the base-2
//             log-sum-exp lse2[row, head] of x = logit * log2(e).  Its COLSUM
//             form streams the keys the same way with the normalisers known and
//             writes per-(row block, head) column sums for mutual scoring (Eq.
//             mutual_scoring, every key takes the mean over rows);
//             text_colsum_reduce adds them in a fixed order.
// text_score  one workgroup per (sample, block of 128 keys, row block).  Each
//             wave owns 32 keys.  For every head the 128 x d query tile is copied
//             global -> LDS (double-buffered) and the wave's key fragments are
//             loaded into registers one head ahead, while p = 2^(x - lse2) of the
//             current head is accumulated over heads per (key, row); the workgroups
//             of one XCD walk the heads from the same start.  Afterwards the row
//             reduction of Eq. text_scoring is applied: max over rows for visual
//             keys, mean for registers, both over the head mean (1/H); with several
//             row blocks the per-block maxima and sums are combined by the sample's
//             last workgroup (or text_rows_combine), which with a threshold also
//             selects the survivors.  Rows beyond T_b carry lse2 = +inf and so
//             contribute exactly 0.
//
// The LDS copies are issued as inline global_load_lds so that the compiler does
// not fold them into its own memory-counter waits; each kernel waits for them
// explicitly (s_waitcnt vmcnt, then a barrier) before the stage is read.
//
// When the caller supplies its own natural-log normaliser (row_lse), text_stats
// is skipped and the second pass reads lse2 = row_lse * log2(e).
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

// Loads are unconditional so that the compiler can count outstanding loads and
// keep prefetches in flight: key and row indices are clamped into range (a
// clamped key's logits are never used, a clamped row's results are never
// written or carry zero weight), and when d % 16 == 8 (HALF) the upper lane
// half of the last 16-wide step reads a valid address and is zeroed by select.
template <int DS, bool HALF>
__device__ __forceinline__ u32x4 frag16(const uint16_t* row, int kk, int hi) {
    const bool pad = HALF && kk == DS - 1 && hi;
    u32x4 v = load16(row + kk * 16 + (pad ? 0 : hi * 8));
    const u32x4 zero = {0u, 0u, 0u, 0u};
    return pad ? zero : v;
}

// The same copy with a wave-uniform base address and a 32-bit per-lane byte offset,
// issued as inline assembly: the compiler does not see it, so it neither counts it
// among the wave's outstanding loads nor makes later LDS reads wait for it.  The
// caller orders it explicitly (wait_vmem + barrier before the copied data is read).
// lds is the wave-uniform LDS byte address of lane 0's 16 bytes.
__device__ __forceinline__ void dma16_async(const void* base, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :: "v"(voff), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}
// Make the compiler treat v as produced here: a load into v must be complete before
// this point (the compiler inserts the wait), and no later code waits for it again.
__device__ __forceinline__ void settle(u32x4& v) { asm volatile("" : "+v"(v)); }
// Wait until every global load of this wave (including LDS copies) has landed.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// vmcnt(n) wait with expcnt / lgkmcnt left unconstrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmem_le() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// COLSUM = false: the base-2 log-sum-exp of every (row, head) over the sample's keys
// (lse2).  COLSUM = true (mutual scoring, Eq. mutual_scoring): with the normalisers
// given (lse_in), the sum over this workgroup's 128 rows of p = 2^(x - lse2) for every
// key, written to part[b][row block][h][key]; the mean over rows and heads is then a
// fixed-order sum over the partials (text_colsum_reduce).  Both modes stream the keys
// the same way; the column sums use the MFMA the other way round (rows as the A
// operand), so that a lane holds 16 rows of one key and sums them in registers.
template <int DS, bool HALF, bool COLSUM, int RG, int RING, int RBW>
__device__ __forceinline__ void stats_task(
    const Prob& p, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    float* __restrict__ lse2, const float* __restrict__ lse_in, int lse_natural,
    float* __restrict__ part, int b, int h, int tblk, int split, int nsplit, char* smem_raw)
{
    // Keys: range split of nsplit (32-key blocks [kb_lo, kb_lo + nkb_s) of the sample);
    // the base-2 log-sum-exp over that range goes to table split of lse2.
    // RBW row blocks (tblk * RBW + rbl, rbl < RBW) of kStatsThreads / 64 waves each; the
    // waves of a row block form kStreams key streams of RG waves: wave w of row block rbl
    // owns the RPW = 128 / RG rows [rg*RPW, +RPW) of it (rg = w % RG) and the key stream
    // ks = w / RG (key blocks kbi = ks mod kStreams).  The RG * RBW waves of a stream (all
    // row blocks) consume the same key blocks, so each block is copied once per stream,
    // global -> LDS, into a ring of RING stages per stream: RING - 1 blocks are in
    // flight while one is used.  RG = 4 (32 rows per wave) needs half the registers of
    // RG = 2 and runs more waves per SIMD; the launcher uses it for every row count.
    // A row block past T_b computes nothing but still copies its share of the blocks and
    // meets every barrier.
    // A block is 32 keys x NCH 16-byte chunks; chunk c of key j sits in LDS unit
    // j*NCH + (c ^ (j & SW)), SW = NCH - 1 when NCH is a power of two (else 0), so a
    // copy writes whole 256-byte key slices and the MFMA fragment reads of 32
    // consecutive keys spread over the banks.
    static_assert(RG == 2 || RG == 4, "row groups per stream");
    static_assert(RBW == 1 || !COLSUM, "column sums take one row block per workgroup");
    constexpr int RPW = kTxtRows / RG;               // rows per wave
    constexpr int NSBW = RPW / 32;                   // 32-row sub-blocks per wave
    constexpr int kStreams = kStatsThreads / kWave / RG;
    constexpr int NW = RG * RBW;                     // waves of one key stream
    constexpr int NCH = 2 * DS;                      // 16-byte chunks per key row
    constexpr int UNITS = 32 * NCH;                  // 16-byte units per block
    constexpr int COPIES = UNITS / kWave;            // = DS copies of 64 lanes per block
    constexpr int MINE = (COPIES + NW - 1) / NW;     // most copies a stream member issues
    constexpr int MINE_MIN = COPIES / NW;            // fewest copies a stream member issues
    constexpr int SW = (NCH & (NCH - 1)) == 0 ? NCH - 1 : 0;
    u32x4* ring = reinterpret_cast<u32x4*>(smem_raw);              // [stream][stage][UNITS]
    float* red_m = reinterpret_cast<float*>(ring + kStreams * RING * UNITS);
    float* red_z = red_m + kStreams * RBW * kTxtRows;
    const int nrb = (p.max_rows + kTxtRows - 1) / kTxtRows;
    const int T = rows_of(p, b);
    if (tblk * RBW * kTxtRows >= T) return;
    const int S = keys_of(p, b);
    const int lane = threadIdx.x & 63;
    const int wave_all = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int rbl = wave_all / (kStatsThreads / kWave), wave = wave_all % (kStatsThreads / kWave);
    const int t0 = (tblk * RBW + rbl) * kTxtRows;
    const int hi = lane >> 5, lo = lane & 31;
    const int rg = wave % RG, ks = wave / RG;
    const int mi = rbl * RG + rg;                      // member index within the stream
    const int H = p.H, Hkv = p.Hkv, d = p.d;
    const int g = h / (H / Hkv);
    const int tw = t0 + rg * RPW;                      // first row of this wave
    const int nsb = max(0, min(NSBW, (T - tw + 31) >> 5));
    const int qb = q_begin(p, b), kb0 = k_begin(p, b);
    const float c2 = p.scale * kLog2e;

    bf16x8 qf[NSBW][DS];
#pragma unroll
    for (int sb = 0; sb < NSBW; ++sb) {
        const int t = min(tw + sb * 32 + lo, T - 1);
        const uint16_t* qrow = q + ((size_t)(qb + t) * H + h) * d;
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) qf[sb][kk] = as_bf16x8(frag16<DS, HALF>(qrow, kk, hi));
    }

    float m[NSBW], z[NSBW];
#pragma unroll
    for (int sb = 0; sb < NSBW; ++sb) { m[sb] = -INFINITY; z[sb] = 0.f; }
    // COLSUM: base-2 normaliser of the 16 rows this lane holds in each sub-block (row
    // 8*(r/4) + 4*hi + r%4 of the sub-block); rows past T_b get +inf and weigh 0.
    float lsev[COLSUM ? NSBW : 1][16];
    if (COLSUM) {
#pragma unroll
        for (int sb = 0; sb < NSBW; ++sb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int t = tw + sb * 32 + acc_key(r, hi);
                float v = INFINITY;
                if (t < T) {
                    v = lse_in[(size_t)(qb + t) * H + h];
                    if (lse_natural) v *= kLog2e;
                }
                lsev[sb][r] = v;
            }
    }

    const int nkb = (S + 31) >> 5;
    const int kb_lo = __builtin_amdgcn_readfirstlane(nkb * split / nsplit);   // wave-uniform
    const int nkb_s = __builtin_amdgcn_readfirstlane(nkb * (split + 1) / nsplit) - kb_lo;
    const int nmine = (nkb_s - ks + kStreams - 1) / kStreams;   // blocks of this stream
    const char* kbase = reinterpret_cast<const char*>(k + ((size_t)kb0 * Hkv + g) * d);
    const int kstride = Hkv * d;                      // elements per key row
    u32x4* sring = ring + ks * RING * UNITS;
    const uint32_t sring_lds = lds_addr(sring);

    // Copy block j of this stream (clamped to the stream's last block) into its stage.
    // Copy c of the block fills units 64c .. 64c+63; this wave issues c = mi, mi+NW, ...
    // Lane offsets inside a block are fixed (key kc = u / NCH of the block, chunk
    // (u % NCH) ^ (kc & SW)); only a block running past S_b clamps its keys.  The pad
    // chunk past d (HALF) reads chunk 0 of the key: its fragment is zeroed below.
    uint32_t coff[MINE];
#pragma unroll
    for (int i = 0; i < MINE; ++i) {
        const int u = min(mi + NW * i, COPIES - 1) * kWave + lane;
        const int kc = u / NCH, ch = (u % NCH) ^ (kc & SW);
        const int e = (HALF && ch == NCH - 1) ? 0 : ch * 8;
        coff[i] = (uint32_t)(kc * kstride + e) * 2u;
    }
    auto issue = [&](int j) {
        const int jj = min(j, max(nmine - 1, 0));
        // A stream with no block of its own (nmine == 0) copies the range's (or the
        // sample's) last block: every copy stays inside the sample's keys, and the stage is
        // never read.
        const int klast = nkb_s > 0 ? kb_lo + nkb_s - 1 : nkb - 1;
        const int kbi = min(kb_lo + ks + jj * kStreams, klast);
        const char* bbase = kbase + (size_t)kbi * 32 * kstride * 2;
        const uint32_t dst = sring_lds + (uint32_t)((jj % RING) * UNITS * 16);
        const bool full = kbi * 32 + 32 <= S;
#pragma unroll
        for (int i = 0; i < MINE; ++i) {
            const int c = mi + NW * i;
            if (c >= COPIES) break;
            uint32_t off = coff[i];
            if (!full) {
                const int u = c * kWave + lane;
                const int kc = u / NCH, ch = (u % NCH) ^ (kc & SW);
                const int e = (HALF && ch == NCH - 1) ? 0 : ch * 8;
                off = (uint32_t)(min(kc, S - 1 - kbi * 32) * kstride + e) * 2u;
            }
            dma16_async(bbase, off, dst + (uint32_t)(c * kWave * 16));
        }
    };
    // Byte offset in a block of fragment (key lo, chunk hi) for k-step 0; k-step kk
    // reads (kfrag ^ kk*32) with SW, (kfrag + kk*32) without.
    const uint32_t kfrag = (uint32_t)(lo * NCH + (hi ^ (lo & SW))) * 16u;

    // One key block: MFMA logits from the LDS stage, then the (reference, sum) update.
    // The reference m of a row is the largest logit of the wave's first block (all later
    // blocks see a full first block, so m is finite there).  Later blocks add
    // 2^(x - m) with m fixed; x may exceed m, and a block whose sum passes 2^64 (or
    // overflows) is redone with its own maximum, which also moves m.  Terms below
    // 2^-126 relative to m are below float32 resolution of z >= 1.
    auto block = [&](int kbi, const u32x4* blk, bool first) -> float {
        const int nvalid = S - kbi * 32;
        u32x4 kf[DS];
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) {
            const uint32_t fo = SW ? (kfrag ^ (uint32_t)(kk * 32)) : kfrag + kk * 32;
            const u32x4 v = *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(blk) + fo);
            const u32x4 zero = {0u, 0u, 0u, 0u};
            kf[kk] = (HALF && kk == DS - 1 && hi) ? zero : v;
        }
        f32x16 acc[NSBW];
#pragma unroll
        for (int sb = 0; sb < NSBW; ++sb) acc[sb] = f32x16{};
        if (COLSUM) {
            // Rows as the A operand: lane (key lo, half hi) holds rows acc_key(r, hi).
            // Both sub-blocks always: a branch between the MFMAs costs more than the
            // clamped rows of a partial second sub-block (whose terms are skipped below).
#pragma unroll
            for (int kk = 0; kk < DS; ++kk)
#pragma unroll
                for (int sb = 0; sb < NSBW; ++sb)
                    acc[sb] = mfma32(qf[sb][kk], as_bf16x8(kf[kk]), acc[sb]);
            // Four partial sums (r mod 4) keep the dependent add chains short.
            float c4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int sb = 0; sb < NSBW; ++sb) {
                if (sb >= nsb) break;
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    c4[r & 3] += __builtin_amdgcn_exp2f(fmaf(acc[sb][r], c2, -lsev[sb][r]));
            }
            const float cs = (c4[0] + c4[1]) + (c4[2] + c4[3]);
            return cs + __shfl_xor(cs, 32);
        }
#pragma unroll
        for (int kk = 0; kk < DS; ++kk)
#pragma unroll
            for (int sb = 0; sb < NSBW; ++sb)
                acc[sb] = mfma32(as_bf16x8(kf[kk]), qf[sb][kk], acc[sb]);
#pragma unroll
        for (int sb = 0; sb < NSBW; ++sb) {
            if (sb >= nsb) break;
            if (!first) {
                // Sum against the fixed reference in four partial chains (r mod 4).
                float a4[4] = {0.f, 0.f, 0.f, 0.f};
                if (nvalid >= 32) {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        a4[r & 3] += __builtin_amdgcn_exp2f(fmaf(acc[sb][r], c2, -m[sb]));
                } else {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (acc_key(r, hi) < nvalid)
                            a4[r & 3] += __builtin_amdgcn_exp2f(fmaf(acc[sb][r], c2, -m[sb]));
                }
                const float asum = (a4[0] + a4[1]) + (a4[2] + a4[3]);
                if (asum <= 0x1p64f) { z[sb] += asum; continue; }
            }
            // Maximum and sum over the lane's 16 keys in four partial chains (r mod 4).
            float m4[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
            if (nvalid >= 32) {
#pragma unroll
                for (int r = 0; r < 16; ++r) m4[r & 3] = fmaxf(m4[r & 3], acc[sb][r]);
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (acc_key(r, hi) < nvalid) m4[r & 3] = fmaxf(m4[r & 3], acc[sb][r]);
            }
            const float mx = fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]));
            if (mx == -INFINITY) continue;
            const float mn = fmaxf(m[sb], mx * c2);
            float s4[4] = {0.f, 0.f, 0.f, 0.f};
            if (nvalid >= 32) {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    s4[r & 3] += __builtin_amdgcn_exp2f(fmaf(acc[sb][r], c2, -mn));
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (acc_key(r, hi) < nvalid)
                        s4[r & 3] += __builtin_amdgcn_exp2f(fmaf(acc[sb][r], c2, -mn));
            }
            const float sum = (s4[0] + s4[1]) + (s4[2] + s4[3]);
            z[sb] = z[sb] * __builtin_amdgcn_exp2f(m[sb] - mn) + sum;
            m[sb] = mn;
        }
        return 0.f;
    };

    // Every wave runs the same number of iterations (the most any stream has), so the
    // barriers match; a stream past its last block only re-issues its last block.
    const int iters = (nkb_s + kStreams - 1) / kStreams;
    // COLSUM: the RG waves of a stream leave their column sums of block j in
    // sums[j & 1][ks][rg][key] (red_m and red_z together); after the next barrier the
    // rg = 0 wave adds them in order of rg and stores the workgroup's partial.
    float* sums = red_m;
    float* prow = part + (((size_t)b * nrb + tblk) * H + h) * (size_t)(p.R + p.max_cands);
    auto store_sums = [&](int j) {
        const float* sp = sums + ((j & 1) * kStreams + ks) * (RG * 32);
        const int key = (ks + j * kStreams) * 32 + lane;
        if (lane < 32 && key < S) {
            float v = sp[lane];
#pragma unroll
            for (int w = 1; w < RG; ++w) v += sp[w * 32 + lane];
            prow[key] = v;
        }
    };
#pragma unroll
    for (int j = 0; j < RING - 1; ++j) issue(j);
    for (int i = 0; i < iters; ++i) {
        // Own copies of block i have landed once at most RING-2 later blocks remain
        // (counted with the fewest copies a member issues: a stronger wait for the others).
        wait_vmem_le<(RING - 2) * MINE_MIN>();
        __syncthreads();                 // partner's copies landed; stage (i-1) is free
        issue(i + RING - 1);
        if (COLSUM && rg == 0 && i >= 1 && i - 1 < nmine) store_sums(i - 1);
        if (i < nmine) {
            float cs = 0.f;
            if (nsb > 0) cs = block(kb_lo + ks + i * kStreams, sring + (i % RING) * UNITS, i == 0);
            if (COLSUM && hi == 0) sums[((i & 1) * kStreams + ks) * (RG * 32) + rg * 32 + lo] = cs;
        }
    }
    wait_vmem_le<0>();
    if (COLSUM) {
        __syncthreads();
        if (rg == 0 && iters >= 1 && iters - 1 < nmine) store_sums(iters - 1);
        return;
    }

    // Merge the two lane halves (same rows, different keys), then the key streams.
#pragma unroll
    for (int sb = 0; sb < NSBW; ++sb) {
        const float mo = __shfl_xor(m[sb], 32);
        const float zo = __shfl_xor(z[sb], 32);
        merge_pair(m[sb], z[sb], mo, zo);
        if (hi == 0) {
            red_m[(rbl * kStreams + ks) * kTxtRows + rg * RPW + sb * 32 + lo] = m[sb];
            red_z[(rbl * kStreams + ks) * kTxtRows + rg * RPW + sb * 32 + lo] = z[sb];
        }
    }
    __syncthreads();
    if (threadIdx.x < RBW * kTxtRows) {
        const int rr = threadIdx.x / kTxtRows, i = threadIdx.x % kTxtRows;
        const float* rm = red_m + rr * kStreams * kTxtRows;
        const float* rz = red_z + rr * kStreams * kTxtRows;
        float mm = rm[i], zz = rz[i];
        for (int w = 1; w < kStreams; ++w) merge_pair(mm, zz, rm[w * kTxtRows + i], rz[w * kTxtRows + i]);
        const int t = (tblk * RBW + rr) * kTxtRows + i;
        if (t < T) lse2[(size_t)split * p.lse_stride + (size_t)(qb + t) * H + h] =
            mm + __builtin_amdgcn_logf(zz);
    }
}

// One statistics task per workgroup.  Task = (sample, head, group of RBW row blocks),
// groups fastest, XCD-aware: the groups of one (sample, head) read the same keys and
// meet in one L2; the RBW row blocks of a group share one copy of every key block.
// Workgroup 0 also clears the per-sample counters of the scoring kernel that follows.
template <int DS, bool HALF, bool COLSUM, int RG, int RBW>
__global__ __launch_bounds__(kStatsThreads * RBW, 1) void text_stats_kernel(
    Prob p, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    float* __restrict__ lse2, const float* __restrict__ lse_in, int lse_natural,
    float* __restrict__ part, Finish fin)
{
    extern __shared__ __attribute__((aligned(16))) char smem_raw[];
    if (blockIdx.x == 0) clear_done(fin, p.B);
    const int nrb = (p.max_rows + kTxtRows - 1) / kTxtRows;
    const int ngrp = (nrb + RBW - 1) / RBW;
    const int ns = COLSUM || p.lse_splits < 1 ? 1 : p.lse_splits;
    const int task = xcd_remap((int)blockIdx.x, ngrp * p.H * p.B * ns);
    const int split = task % ns, rest = task / ns;
    const int tblk = rest % ngrp, h = (rest / ngrp) % p.H, b = rest / (ngrp * p.H);
    stats_task<DS, HALF, COLSUM, RG, kStatsRing, RBW>(p, q, k, lse2, lse_in, lse_natural, part,
                                                      b, h, tblk, split, ns, smem_raw);
}

// Ragged launches: workgroup id -> the id-th non-empty (sample, key chunk, row block)
// task of the scoring pass, so that the active tasks take the lowest ids and spread over
// the CUs in dispatch order, instead of sitting among the empty chunks of short samples
// (where two of them can share a CU while other CUs idle).  Samples in reverse order,
// chunks then row blocks, as in the uniform mapping; xcd_remap over the A active tasks
// keeps a sample's tasks on one XCD.  Called by wave 0: each lane counts the tasks of a
// run of consecutive samples, a scan finds the lane and sample holding the task, which
// leaves (b, c, rb) in sh[0..2], or b = -1 past the last task.
__device__ void ragged_score_task(const Prob& p, int id, int* sh) {
    const int lane = threadIdx.x;
    const int per = (p.B + kWave - 1) / kWave;
    const int i0 = min(lane * per, p.B), i1 = min(i0 + per, p.B);
    auto ntask = [&](int b) {
        const int T = rows_of(p, b), S = keys_of(p, b);
        if (T <= 0 || S <= 0) return 0;
        return ((S + kTxtKeysPerWg - 1) / kTxtKeysPerWg) * ((T + kTxtRows - 1) / kTxtRows);
    };
    int cnt = 0;
    for (int i = i0; i < i1; ++i) cnt += ntask(p.B - 1 - i);
    int incl = cnt;
    for (int off = 1; off < kWave; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
    }
    const int A = __shfl(incl, kWave - 1);
    if (id >= A) {
        if (lane == 0) sh[0] = -1;
        return;
    }
    const int t = xcd_remap(id, A);
    int acc = incl - cnt;
    if (t < acc || t >= incl) return;
    for (int i = i0; i < i1; ++i) {
        const int b = p.B - 1 - i, n = ntask(b);
        if (t < acc + n) {
            const int nrb_b = (rows_of(p, b) + kTxtRows - 1) / kTxtRows;
            sh[0] = b;
            sh[1] = (t - acc) / nrb_b;
            sh[2] = (t - acc) % nrb_b;
            return;
        }
        acc += n;
    }
}

// One scoring task: keys [128 c, 128 c + 128) of sample b against its row block rb.
// CC: the normalisers were written earlier in the same launch (by other workgroups), so
// they are read with device-coherent loads.  cc_out: the scores / partials are read later
// in the same launch by another workgroup, so they are written with device-coherent
// stores.  rot_id picks the starting head (rot_id % 8 of 8 heads spread over H).
template <int DS, bool HALF, bool FULL, bool CC>
__device__ __forceinline__ void score_task(
    const Prob& p, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const float* __restrict__ lse, int lse_natural, float* __restrict__ scores,
    float* __restrict__ part, int b, int c, int rb, int rot_id, char* smem_raw, bool cc_out)
{
    // 4 waves: wave w owns the 32 keys [s_lo + 32 w, +32) and the 128 rows of the
    // workgroup's row block (4 sub-blocks of 32 rows, one MFMA accumulator chain each).  Two workgroups share a CU, so one workgroup's MFMAs
    // overlap the other's exponentials.
    //
    // The query tile of a head (128 rows x NCH 16-byte chunks) lives in LDS row-major
    // with an XOR swizzle: chunk c of row t sits in unit t*NCH + (c ^ (t & SW)), SW =
    // NCH - 1 when NCH is a power of two (else 0).  It is double-buffered: the next
    // head's tile is copied global -> LDS directly (buffer loads) while the current
    // head is computed, so the copy needs no registers and each head needs one
    // barrier.  A copy writes 64 consecutive units, i.e. reads whole 256-byte row
    // slices from memory; an MFMA fragment read (32 rows, one chunk each) touches 16
    // distinct 16-byte bank groups per 16 lanes.
    constexpr int NCH = 2 * DS;                                   // 16-byte chunks per row
    constexpr int QTILE = kTxtRows * NCH;                         // 16-byte units per tile
    constexpr int COPIES = QTILE / kWave / (kScoreThreads / kWave);  // per wave per tile
    constexpr int SW = (NCH & (NCH - 1)) == 0 ? NCH - 1 : 0;
    u32x4* qt = reinterpret_cast<u32x4*>(smem_raw);                         // [2][QTILE]
    float* l2t = reinterpret_cast<float*>(smem_raw + 2 * QTILE * 16);       // [H][128]
    // With several row blocks (part != null) each task writes its row maximum (visual
    // keys) or row sum (registers) to part[b][row block][key]; the scores are formed from
    // them afterwards (text_rows_combine, or the last task of the sample).
    const int nrb = (p.max_rows + kTxtRows - 1) / kTxtRows;
    const int S = keys_of(p, b);
    const int s_lo = c * kTxtKeysPerWg;
    const int t0 = rb * kTxtRows;
    if (s_lo >= S || t0 >= rows_of(p, b)) return;
    const int T = rows_of(p, b);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hi = lane >> 5, lo = lane & 31;
    const int H = p.H, Hkv = p.Hkv, d = p.d, group = H / Hkv;
    const int qb = q_begin(p, b), kb0 = k_begin(p, b);
    const float c2 = p.scale * kLog2e;
    const int wkey0 = s_lo + wave * kTxtKeysPerWave;
    const bool wactive = wkey0 < S;
    const int R = p.R;
    // Loop step hh works on head (hh + rot) mod H: a key row's head slices all sit at
    // the same offset within 8 KB rows, so workgroups moving through the heads in step
    // would load the same memory channels at the same time.  Eight starting heads,
    // spread over the H heads, balance the channels as well as H of them do; with one
    // start per XCD (rot_id % 8 is the XCD), the workgroups that share an L2 also share
    // the query tile and key slices they are reading.  Steps past the last head repeat
    // the last one (clamped prefetches).
    const int nrot = H < 8 ? H : 8;
    const int rot = (int)((unsigned)rot_id % (unsigned)nrot) * (H / nrot);
    auto head_of = [&](int hh) {
        const int hc = min(hh, H - 1) + rot;
        return hc >= H ? hc - H : hc;
    };

    // Copy head hh's query tile (rows t0..t0+127) into buffer buf.  Copy j of this
    // wave fills units U = (wave*COPIES + j)*64 + lane: row t = U / NCH, the chunk
    // stored there is (U % NCH) ^ (t & SW).  Rows past T_b are clamped (their lse2 is
    // +inf, so they weigh exactly 0); the pad chunk past d (HALF) reads chunk 0
    // instead, harmless because the matching key chunk is zero.  The per-lane byte
    // offsets are fixed for a row block (set_rows); a head only moves the base.
    uint32_t qoff[COPIES];
    const char* qrows = nullptr;
    auto set_rows = [&](int t0) {
#pragma unroll
        for (int j = 0; j < COPIES; ++j) {
            const int U = (wave * COPIES + j) * kWave + lane;
            const int t = min(U / NCH, T - t0 - 1), ch = (U % NCH) ^ ((U / NCH) & SW);
            const int e = (HALF && ch == NCH - 1) ? 0 : ch * 8;
            qoff[j] = (uint32_t)(t * H * d + e) * 2u;
        }
        qrows = reinterpret_cast<const char*>(q + ((size_t)qb + t0) * H * d);
    };
    const uint32_t qt_lds = lds_addr(qt);
    auto copy_q = [&](int hh, int buf) {
        const char* base = qrows + (size_t)head_of(hh) * d * 2;
#pragma unroll
        for (int j = 0; j < COPIES; ++j)
            dma16_async(base, qoff[j],
                        qt_lds + (uint32_t)((buf * QTILE + (wave * COPIES + j) * kWave) * 16));
    };
    // Byte offset in a tile of fragment (row lo of a 32-row block, chunk hi) for k-step
    // 0; k-step kk reads (qfrag ^ kk*32) with SW, (qfrag + kk*32) without.
    const uint32_t qfrag = (uint32_t)(lo * NCH + (hi ^ (lo & SW))) * 16u;
    // Key fragments: lane offset within the sample's key rows, fixed; the head picks the base.
    const int kclamp = min(wkey0 + lo, S - 1);        // keys past S_b are never written
    const uint32_t koff = (uint32_t)(kclamp * Hkv * d) * 2u;
    const char* ksample = reinterpret_cast<const char*>(k + (size_t)kb0 * Hkv * d);
    auto load_k = [&](int hh, u32x4 (&kf)[DS]) {
        const char* base = ksample + (size_t)(head_of(hh) / group) * d * 2;
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) {
            const bool pad = HALF && kk == DS - 1 && hi;
            const u32x4 v = *reinterpret_cast<const u32x4*>(
                base + koff + (uint32_t)((kk * 16 + (pad ? 0 : hi * 8)) * 2));
            const u32x4 zero = {0u, 0u, 0u, 0u};
            kf[kk] = pad ? zero : v;
        }
    };

    float abar[4][16];
    {
        const int nsb = min(4, (T - t0 + 31) >> 5);
        for (int i = tid; i < H * kTxtRows; i += kScoreThreads) {
            const int hh = i / kTxtRows, t = t0 + (i % kTxtRows);
            float v = INFINITY;
            if (t < T) {
                const float* src = lse + (size_t)(qb + t) * H + hh;
                v = CC ? __hip_atomic_load(src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : *src;
                if (lse_natural) v *= kLog2e;
            }
            l2t[i] = v;
        }
        u32x4 k0[DS], k1[DS];
        set_rows(t0);
        load_k(0, k0);
        copy_q(0, 0);
        wait_vmem();
#pragma unroll
        for (int kk = 0; kk < DS; ++kk) settle(k0[kk]);
        __syncthreads();

#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
            for (int r = 0; r < 16; ++r) abar[sb][r] = 0.f;

        // One head: start the copies of head h+1 (query tile to the other buffer, key
        // fragments to registers), MFMA logits of the wave's 32 keys x 128 rows (two
        // accumulator chains at a time), p = 2^(x - lse2), head sum; then wait for the
        // copies and synchronise.
        auto head = [&](int h, const u32x4 (&kf)[DS], u32x4 (&kn)[DS]) {
            const int buf = h & 1;
            // Nothing of this wave is in flight here except compiler reloads; waiting for
            // them now keeps the compiler from waiting inside the head, where that wait
            // would also cover the copies issued next.
            wait_vmem();
            copy_q(h + 1, buf ^ 1);
            load_k(h + 1, kn);
            if (wactive) {
                const char* qtile = reinterpret_cast<const char*>(qt) + buf * QTILE * 16;
                // MFMA logits of the wave's 32 keys x one 32-row sub-block (one accumulator
                // chain), and p = 2^(x - lse2) of a finished chain added to the head sum.
                auto chain = [&](int sp) {
                    f32x16 acc = {};
#pragma unroll
                    for (int kk = 0; kk < DS; ++kk) {
                        const uint32_t fo = SW ? (qfrag ^ (uint32_t)(kk * 32)) : qfrag + kk * 32;
                        const u32x4 qv = *reinterpret_cast<const u32x4*>(qtile + sp * 32 * NCH * 16 + fo);
                        acc = mfma32(as_bf16x8(kf[kk]), as_bf16x8(qv), acc);
                    }
                    return acc;
                };
                auto soft = [&](int sp, const f32x16& acc) {
                    const float l2 = l2t[head_of(h) * kTxtRows + sp * 32 + lo];
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        abar[sp][r] += __builtin_amdgcn_exp2f(fmaf(acc[r], c2, -l2));
                };
                // The chain of sub-block sp+1 is issued next to the exponentials of
                // sub-block sp (scheduling barriers keep each pair together), so the wave
                // keeps the matrix core and the vector unit busy at once; left to itself
                // the compiler issues all 32 MFMAs first.
                auto pipelined = [&]() {
                    f32x16 a0 = chain(0);
                    __builtin_amdgcn_sched_barrier(0);
                    f32x16 a1 = chain(1);
                    soft(0, a0);
                    __builtin_amdgcn_sched_barrier(0);
                    a0 = chain(2);
                    soft(1, a1);
                    __builtin_amdgcn_sched_barrier(0);
                    a1 = chain(3);
                    soft(2, a0);
                    __builtin_amdgcn_sched_barrier(0);
                    soft(3, a1);
                };
                if constexpr (FULL) {
                    // Every row block full (FULL: uniform T, a multiple of 128).  With one
                    // workgroup per CU (few keys per sample) the pipelined order is 13 %
                    // faster.  A separate instantiation: the two forms in one kernel need
                    // more registers, and the uniform batches run slower with them.
                    pipelined();
                } else if (nsb == 4) {
                    // A full row block of a ragged or partial batch takes the same order
                    // (Qwen3-VL batch: ~1 % faster step).
                    pipelined();
                } else {
#pragma unroll
                    for (int sp = 0; sp < 4; ++sp) {
                        if (sp >= nsb) break;
                        soft(sp, chain(sp));
                    }
                }
            }
            wait_vmem();
            __syncthreads();
        };
        for (int h = 0; h < H; h += 2) {
            head(h, k0, k1);
            if (h + 1 >= H) break;
            head(h + 1, k1, k0);
        }
    }

    // Row reduction of Eq. text_scoring (visual keys: max over rows, registers: mean):
    // over the lane's sub-blocks, then across the 32 lanes of a lane half (fixed
    // order).  Rows past T_b hold exact zeros.
    const bool regs = wactive && wkey0 < R;              // keys whose row sum is needed
    float mx[16], sm[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        mx[r] = fmaxf(fmaxf(abar[0][r], abar[1][r]), fmaxf(abar[2][r], abar[3][r]));
        sm[r] = (abar[0][r] + abar[1][r]) + (abar[2][r] + abar[3][r]);
#pragma unroll
        for (int off = 16; off >= 1; off >>= 1) {
            mx[r] = fmaxf(mx[r], __shfl_xor(mx[r], off));
            if (regs) sm[r] += __shfl_xor(sm[r], off);
        }
    }
    if (wactive && lo == 0) {
        const float invH = 1.f / (float)H;
        const float invHT = 1.f / ((float)H * (float)T);
        float* prow = part ? part + ((size_t)b * nrb + rb) * (size_t)(p.R + p.max_cands) : nullptr;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key = wkey0 + acc_key(r, hi);
            if (key >= S) continue;
            float* dst = prow ? prow + key : scores + kb0 + key;
            const float v = prow ? (key < R ? sm[r] : mx[r]) : (key < R ? sm[r] * invHT : mx[r] * invH);
            if (cc_out) st_cc(dst, v);
            else *dst = v;
        }
    }
}

// One scoring task per workgroup.  Task = (sample, key chunk, row block), row blocks
// fastest, XCD-aware: the chunks of one sample run on one XCD and share its L2 for the
// query tiles, and the row blocks of one chunk read the same keys there.  Samples in
// reverse order: the statistics pass streamed sample B-1 last, so its keys are the
// likeliest to still sit in the memory-side cache.
// With fin.done, the last workgroup of each sample forms its scores from the row blocks'
// partials (text_rows_combine's arithmetic) and, with fin.select, applies the threshold
// and the compaction (select_kernel's arithmetic).
template <int DS, bool HALF, bool FULL>
__global__ __launch_bounds__(kScoreThreads, 2) void text_score_kernel(
    Prob p, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const float* __restrict__ lse, int lse_natural, float* __restrict__ scores,
    float* __restrict__ part, Finish fin)
{
    extern __shared__ __attribute__((aligned(16))) char smem_raw[];
    const int nchunk = (p.R + p.max_cands + kTxtKeysPerWg - 1) / kTxtKeysPerWg;
    const int nrb = (p.max_rows + kTxtRows - 1) / kTxtRows;
    int b, c, rb;
    if (p.k_off || p.q_off) {
        // The decoded task passes through the start of query buffer 1 (after the first
        // 128 x d tile), which is first written (head 1's copy) after the barrier that
        // ends the task's prologue.
        int* sh = reinterpret_cast<int*>(smem_raw + (size_t)kTxtRows * 2 * DS * 16);
        if (threadIdx.x < kWave) ragged_score_task(p, (int)blockIdx.x, sh);
        __syncthreads();
        b = sh[0];
        if (b < 0) return;
        c = sh[1];
        rb = sh[2];
    } else {
        const int task = xcd_remap((int)blockIdx.x, nchunk * nrb * p.B);
        rb = task % nrb;
        c = (task / nrb) % nchunk;
        b = p.B - 1 - task / (nrb * nchunk);
    }
    // The starting head follows the XCD (workgroups are dealt to the 8 XCDs round-robin,
    // and each XCD runs one contiguous range of tasks): every workgroup of an XCD walks the
    // heads in the same order, so the chunks of a sample read its query tiles, and the row
    // blocks of a chunk its key slices, at about the same time, and share them in that
    // XCD's L2.  A start per key chunk instead fetched 1062 MB per launch at the
    // LLaVA-NeXT shape and 3586 MB on the ragged Qwen3-VL batch; per XCD, 807 and 2654 MB,
    // ~1 % faster.
    score_task<DS, HALF, FULL, false>(p, q, k, lse, lse_natural, scores, part, b, c, rb,
                                      (int)blockIdx.x, smem_raw, fin.done != nullptr);
    if (!fin.done) return;
    const int S = keys_of(p, b), T = rows_of(p, b);
    const int nrb_b = (T + kTxtRows - 1) / kTxtRows;
    const unsigned ntask = (unsigned)(((S + kTxtKeysPerWg - 1) / kTxtKeysPerWg) * nrb_b);
    if (!last_of_sample(fin.done, b, ntask, reinterpret_cast<int*>(smem_raw + 64))) return;
    if (part) {
        // Row maxima (visual keys) / row sums (registers) over the row blocks in order,
        // then the head (and row) mean: text_rows_combine's arithmetic.  Each thread takes
        // U keys at a time, so that U coherent loads per row block are in flight (one at a
        // time cost ~40 us on the video batch's 16384-key samples).  With the threshold to
        // follow, the scores also go straight into the LDS copy that it reads.
        constexpr int U = 16;
        const size_t smax = (size_t)(p.R + p.max_cands);
        const float* pb = part + (size_t)b * nrb * smax;
        float* out = scores + k_begin(p, b);
        float* sl = fin.select ? select_scores_lds(smem_raw + 128) : nullptr;
        const float inv_reg = 1.f / ((float)p.H * (float)T), inv_vis = 1.f / (float)p.H;
        for (int s0 = threadIdx.x; s0 < S; s0 += U * kScoreThreads) {
            float v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = 0.f;
            for (int r = 0; r < nrb_b; ++r) {
                float x[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int s = s0 + u * kScoreThreads;
                    x[u] = s < S ? ld<true>(pb + (size_t)r * smax + s) : 0.f;
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
                    v[u] = s0 + u * kScoreThreads < p.R ? v[u] + x[u] : fmaxf(v[u], x[u]);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int s = s0 + u * kScoreThreads;
                if (s < S) {
                    const float w = v[u] * (s < p.R ? inv_reg : inv_vis);
                    st_cc(out + s, w);
                    if (sl) sl[s] = w;
                }
            }
        }
        if (fin.select) {
            __syncthreads();
            select_sample(p, scores, b, fin, smem_raw + 128, true);
        }
        return;
    }
    if (fin.select) select_sample(p, scores, b, fin, smem_raw + 128, false);
}

// Scores from the row blocks' partials: the maximum over row blocks (visual keys) or
// the sum in row-block order (registers), then the head mean (and row mean).
__global__ __launch_bounds__(256) void text_rows_combine_kernel(Prob p, const float* __restrict__ part,
                                                                float* __restrict__ scores)
{
    const int b = blockIdx.y, s = blockIdx.x * 256 + threadIdx.x;
    const int S = keys_of(p, b), T = rows_of(p, b);
    if (s >= S) return;
    const int nrb_max = (p.max_rows + kTxtRows - 1) / kTxtRows, nrb = (T + kTxtRows - 1) / kTxtRows;
    const size_t smax = (size_t)(p.R + p.max_cands);
    const float* pb = part + (size_t)b * nrb_max * smax + s;
    float v = 0.f;
    if (s < p.R) {
        for (int rb = 0; rb < nrb; ++rb) v += pb[(size_t)rb * smax];
        v *= 1.f / ((float)p.H * (float)T);
    } else {
        for (int rb = 0; rb < nrb; ++rb) v = fmaxf(v, pb[(size_t)rb * smax]);
        v *= 1.f / (float)p.H;
    }
    scores[k_begin(p, b) + s] = v;
}

// Key ranges of the statistics pass: merge the ranges' base-2 log-sum-exps, in range
// order, into the first table (every (row, head) entry of the workspace's tables; entries
// of rows past a sample's T_b are never read).
__global__ __launch_bounds__(256) void text_lse_merge_kernel(Prob p, float* __restrict__ lse2,
                                                             long long n)
{
    const int ns = min(p.lse_splits, kStatsMaxSplits);
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long long)gridDim.x * 256) {
        float l[kStatsMaxSplits];
        float mx = -INFINITY;
        for (int r = 0; r < ns; ++r) {
            l[r] = lse2[(size_t)r * p.lse_stride + i];
            mx = fmaxf(mx, l[r]);
        }
        float z = 0.f;
        for (int r = 0; r < ns; ++r) z += __builtin_amdgcn_exp2f(l[r] - mx);
        lse2[i] = mx == -INFINITY ? mx : mx + __builtin_amdgcn_logf(z);
    }
}

template <int DS, bool HALF, bool COLSUM, int RG, int RBW>
static hipError_t stats_launch_rg(const Prob& p, const void* q, const void* k, float* lse2,
                                  const float* lse_in, int lse_natural, float* part,
                                  const Finish& fin, hipStream_t s) {
    const size_t smem = text_stats_smem(DS * 16, RG, RBW);
    static std::atomic<uint64_t> lds_set{0};
    const hipError_t attr = allow_lds(
        reinterpret_cast<const void*>(&text_stats_kernel<DS, HALF, COLSUM, RG, RBW>),
        (int)kScoreSmemMax, lds_set);
    if (attr != hipSuccess) return attr;
    const int nrb = (p.max_rows + kTxtRows - 1) / kTxtRows;
    const int ns = COLSUM || p.lse_splits < 1 ? 1 : p.lse_splits;
    dim3 grid((nrb + RBW - 1) / RBW * p.H * p.B * ns);
    const hipError_t e = launch(text_stats_kernel<DS, HALF, COLSUM, RG, RBW>, grid,
                                dim3(kStatsThreads * RBW), smem, s, p,
                                static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                                lse2, lse_in, lse_natural, part, fin);
    if (e != hipSuccess || ns == 1) return e;
    const long long n = p.lse_stride;
    const long long nblk = (n + 255) / 256;
    return launch(text_lse_merge_kernel, dim3((unsigned)(nblk < 2048 ? nblk : 2048)), dim3(256), 0,
                  s, p, lse2, n);
}

// Four waves of 32 rows on one key stream.  Two streams of two 64-row waves reuse each
// key fragment twice per wave but need twice the registers; at one 128-row block (T =
// 128, LLaVA-NeXT) the one-stream form measured 6 % faster (137-139 against 146-147 us).
template <int DS, bool HALF, bool COLSUM>
static hipError_t stats_launch(const Prob& p, const void* q, const void* k, float* lse2,
                               const float* lse_in, int lse_natural, float* part,
                               const Finish& fin, hipStream_t s) {
    // With two to four row blocks per sample, one workgroup takes two or four of them and
    // copies each key block once for all: on the ragged Qwen3-VL batch (up to 4 row
    // blocks) the pass fetches 1403 MB, its algorithmic bytes, instead of 1965 MB with
    // one row block per workgroup (1722 MB with two), ~1 % faster.  Taller batches keep
    // one row block per workgroup: the mutual-scoring Stage I of the same batch (up to 32
    // row blocks) took 4.42 ms with four per workgroup, 3.84 ms with two, 3.83 ms with one.
    if constexpr (!COLSUM) {
        const int rbw = stats_row_blocks((p.max_rows + kTxtRows - 1) / kTxtRows);
        if (rbw == 4)
            return stats_launch_rg<DS, HALF, COLSUM, 4, 4>(p, q, k, lse2, lse_in, lse_natural, part,
                                                           fin, s);
        if (rbw == 2)
            return stats_launch_rg<DS, HALF, COLSUM, 4, 2>(p, q, k, lse2, lse_in, lse_natural, part,
                                                           fin, s);
    }
    return stats_launch_rg<DS, HALF, COLSUM, 4, 1>(p, q, k, lse2, lse_in, lse_natural, part, fin, s);
}

template <int DS, bool HALF>
static hipError_t stats_ds(const Prob& p, const void* q, const void* k, float* lse2,
                           const Finish& fin, hipStream_t s) {
    return stats_launch<DS, HALF, false>(p, q, k, lse2, nullptr, 0, nullptr, fin, s);
}

template <int DS, bool HALF>
static hipError_t colsum_ds(const Prob& p, const void* q, const void* k, const float* lse,
                            int lse_natural, float* part, hipStream_t s) {
    return stats_launch<DS, HALF, true>(p, q, k, nullptr, lse, lse_natural, part, Finish{}, s);
}

// Mutual scores: the mean over rows and heads of p, from the per-(row block, head)
// column sums, added in a fixed order (row blocks outer, heads inner).
__global__ __launch_bounds__(256) void text_colsum_reduce_kernel(Prob p, const float* __restrict__ part,
                                                                 float* __restrict__ scores)
{
    const int b = blockIdx.y, s = blockIdx.x * 256 + threadIdx.x;
    const int S = keys_of(p, b), T = rows_of(p, b);
    if (s >= S) return;
    const int nrb_max = (p.max_rows + kTxtRows - 1) / kTxtRows, nrb = (T + kTxtRows - 1) / kTxtRows;
    const size_t smax = (size_t)(p.R + p.max_cands);
    const float* pb = part + (size_t)b * nrb_max * p.H * smax + s;
    // Up to 16 partials are loaded before they are added (in order): the loads do not
    // depend on the running sum, so they are in flight together.
    const int n = nrb * p.H;
    float acc = 0.f;
    int i = 0;
    for (; i + 16 <= n; i += 16) {
        float v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = pb[(size_t)(i + j) * smax];
#pragma unroll
        for (int j = 0; j < 16; ++j) acc += v[j];
    }
    for (; i < n; ++i) acc += pb[(size_t)i * smax];
    scores[k_begin(p, b) + s] = T > 0 ? acc * (1.f / ((float)p.H * (float)T)) : 0.f;
}

template <int DS, bool HALF, bool FULL>
static hipError_t score_launch(const Prob& p, const void* q, const void* k, const float* lse,
                               int lse_natural, float* scores, float* part, const Finish& fin,
                               hipStream_t s) {
    const size_t smem = text_score_smem(p.H, DS * 16);
    // The tile needs more than the default 64 KB of dynamic LDS: raise the limit (once per
    // device).
    static std::atomic<uint64_t> lds_set{0};
    const hipError_t attr = allow_lds(
        reinterpret_cast<const void*>(&text_score_kernel<DS, HALF, FULL>), (int)kScoreSmemMax,
        lds_set);
    if (attr != hipSuccess) return attr;
    const int nrb = (p.max_rows + kTxtRows - 1) / kTxtRows;
    dim3 grid((p.R + p.max_cands + kTxtKeysPerWg - 1) / kTxtKeysPerWg * nrb * p.B);
    return launch(text_score_kernel<DS, HALF, FULL>, grid, dim3(kScoreThreads), smem, s, p,
                  static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), lse,
                  lse_natural, scores, nrb > 1 ? part : nullptr, fin);
}

template <int DS, bool HALF>
static hipError_t score_ds(const Prob& p, const void* q, const void* k, const float* lse,
                           int lse_natural, float* scores, float* part, const Finish& fin,
                           hipStream_t s) {
    // Uniform rows that fill whole 128-row blocks take the pipelined form.
    const bool full = !p.q_off && p.rows == p.max_rows && p.rows % kTxtRows == 0;
    const hipError_t e =
        full ? score_launch<DS, HALF, true>(p, q, k, lse, lse_natural, scores, part, fin, s)
             : score_launch<DS, HALF, false>(p, q, k, lse, lse_natural, scores, part, fin, s);
    if (e != hipSuccess) return e;
    const int nrb = (p.max_rows + kTxtRows - 1) / kTxtRows;
    if (nrb == 1 || fin.done) return hipSuccess;
    dim3 cgrid((p.R + p.max_cands + 255) / 256, p.B);
    return launch(text_rows_combine_kernel, cgrid, dim3(256), 0, s, p, part, scores);
}

// d = 16*DS (HALF = false) or 16*DS - 8 (HALF = true), d <= 128.
#define OCCAM_D_SWITCH(FN, ...)                                                  \
    switch (p.d) {                                                               \
        case 8: return FN<1, true>(__VA_ARGS__);    case 16: return FN<1, false>(__VA_ARGS__);  \
        case 24: return FN<2, true>(__VA_ARGS__);   case 32: return FN<2, false>(__VA_ARGS__);  \
        case 40: return FN<3, true>(__VA_ARGS__);   case 48: return FN<3, false>(__VA_ARGS__);  \
        case 56: return FN<4, true>(__VA_ARGS__);   case 64: return FN<4, false>(__VA_ARGS__);  \
        case 72: return FN<5, true>(__VA_ARGS__);   case 80: return FN<5, false>(__VA_ARGS__);  \
        case 88: return FN<6, true>(__VA_ARGS__);   case 96: return FN<6, false>(__VA_ARGS__);  \
        case 104: return FN<7, true>(__VA_ARGS__);  case 112: return FN<7, false>(__VA_ARGS__); \
        case 120: return FN<8, true>(__VA_ARGS__);  case 128: return FN<8, false>(__VA_ARGS__); \
        default: return hipErrorInvalidValue;                                    \
    }

hipError_t launch_text_stats(const Prob& p, const void* q, const void* k, float* lse2,
                             const Finish& fin, hipStream_t s) {
    OCCAM_D_SWITCH(stats_ds, p, q, k, lse2, fin, s)
}

hipError_t launch_text_score(const Prob& p, const void* q, const void* k, const float* lse,
                             int lse_natural, float* scores, float* part, const Finish& fin,
                             hipStream_t s) {
    OCCAM_D_SWITCH(score_ds, p, q, k, lse, lse_natural, scores, part, fin, s)
}

static hipError_t colsum_any(const Prob& p, const void* q, const void* k, const float* lse,
                             int lse_natural, float* part, hipStream_t s) {
    OCCAM_D_SWITCH(colsum_ds, p, q, k, lse, lse_natural, part, s)
}

hipError_t launch_text_colsum(const Prob& p, const void* q, const void* k, const float* lse,
                              int lse_natural, float* part, float* scores, hipStream_t s) {
    const hipError_t e = colsum_any(p, q, k, lse, lse_natural, part, s);
    if (e != hipSuccess) return e;
    dim3 grid((p.R + p.max_cands + 255) / 256, p.B);
    return launch(text_colsum_reduce_kernel, grid, dim3(256), 0, s, p, part, scores);
}

}  // namespace occam
