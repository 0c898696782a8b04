// Test-time register construction (Algorithm 1, "redirect sinks to r"; Appendix
// Eq. register_redirect_appendix): for each listed MLP channel k of the vision
// encoder, the register row of a sample takes the max of channel k over the
// sample's visual rows, and the visual rows' values of channel k become 0.
//
// register_redirect  grid (sample, group of 4 listed channels), one wave per listed
//                    channel: the wave's lanes stride over the visual rows for the
//                    max (one 2- or 4-byte read per row), a wave reduction, then
//                    lane 0 writes the register and the lanes zero the rows.  A
//                    wave skips an index outside [0, width) and a repeat of an
//                    earlier list entry, so distinct waves never touch the same
//                    element.  A maximum of zero is written as +0.
#include "occam_internal.hpp"

namespace occam {

template <bool BF16>
__device__ __forceinline__ float load_act(const char* p) {
    if (BF16) return __uint_as_float(static_cast<uint32_t>(*reinterpret_cast<const uint16_t*>(p)) << 16);
    return *reinterpret_cast<const float*>(p);
}
template <bool BF16>
__device__ __forceinline__ void store_act(char* p, float v) {
    // A value read from the tensor converts back exactly (bf16 -> f32 -> bf16).
    if (BF16) *reinterpret_cast<uint16_t*>(p) = static_cast<uint16_t>(__float_as_uint(v) >> 16);
    else *reinterpret_cast<float*>(p) = v;
}

template <bool BF16>
__global__ __launch_bounds__(256) void register_redirect_kernel(
    Prob p, char* __restrict__ h, int width, long long stride, const int* __restrict__ channels,
    int n_channels, int reg_slot)
{
    const int b = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int j = blockIdx.y * 4 + (threadIdx.x >> 6);        // list entry of this wave
    if (j >= n_channels) return;
    const int k = channels[j];
    if (k < 0 || k >= width) return;
    for (int i = 0; i < j; ++i)
        if (channels[i] == k) return;                          // a repeat acts once
    const int N = keys_of(p, b) - p.R;
    if (N <= 0) return;
    constexpr int E = BF16 ? 2 : 4;
    char* base = h + (long long)k_begin(p, b) * stride + (long long)k * E;
    char* vis = base + (long long)p.R * stride;
    float m = -INFINITY;
    for (int v = lane; v < N; v += kWave) m = fmaxf(m, load_act<BF16>(vis + (long long)v * stride));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if (m == 0.f) m = 0.f;                                     // +0 for a zero maximum
    if (lane == 0) store_act<BF16>(base + (long long)reg_slot * stride, m);
    for (int v = lane; v < N; v += kWave) store_act<BF16>(vis + (long long)v * stride, 0.f);
}

hipError_t launch_register_redirect(const Prob& p, int bf16, void* h, int width, long long stride,
                                    const int* channels, int n_channels, int reg_slot,
                                    hipStream_t s)
{
    if (n_channels == 0) return hipSuccess;
    dim3 grid(p.B, (n_channels + 3) / 4);
    if (bf16)
        return launch(register_redirect_kernel<true>, grid, dim3(256), 0, s, p,
                      static_cast<char*>(h), width, stride, channels, n_channels, reg_slot);
    return launch(register_redirect_kernel<false>, grid, dim3(256), 0, s, p, static_cast<char*>(h),
                  width, stride, channels, n_channels, reg_slot);
}

}  // namespace occam
