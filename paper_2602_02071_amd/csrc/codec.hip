// Streaming HiF8 encode / decode kernels (HBM-bound, grid-stride).
//
// Every wave-wide memory instruction touches one contiguous range: a lane
// handles 4 consecutive elements per step (16 bytes of fp32, 4 bytes of
// codes), and each lane issues several independent steps back to back so
// that enough bytes are in flight.
#include "common.hpp"

namespace baps {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;                     // 4-element groups per lane per iteration

// Rounding to nearest with ties away from zero depends only on the sign, the
// exponent and the top four mantissa bits of the fp32 input (bits 31..19),
// so each workgroup tabulates the code of every such prefix once (8 KiB of
// LDS) and the streaming loop is a shift and a table read.  The one case the
// prefix cannot tell is a NaN whose payload sits below bit 19: its prefix
// reads as +-Inf, so NaN is tested on the full pattern.  With ties to even
// (EVEN) an input can sit exactly halfway only when bits 18..0 are zero: a
// second table holds the code of each prefix with those bits zero, and every
// other input is not a tie, where both rules agree.
template <bool EVEN>
__device__ __forceinline__ uint32_t encode1(const uint8_t* tab8, float x)
{
    const uint32_t u = hif8::f2u(x);
    uint32_t i = u >> kTabShift;
    if constexpr (EVEN) i |= (u & 0x7ffffu) ? 0u : (uint32_t)kTabEntries;
    const uint32_t c = tab8[i];
    return (u & 0x7fffffffu) > 0x7f800000u ? 0x80u : c;
}

template <bool EVEN>
__device__ __forceinline__ uint32_t encode4(const uint8_t* tab8, f32x4 v)
{
    return encode1<EVEN>(tab8, v[0]) | (encode1<EVEN>(tab8, v[1]) << 8) | (encode1<EVEN>(tab8, v[2]) << 16) |
           (encode1<EVEN>(tab8, v[3]) << 24);
}

template <bool EVEN>
__global__ __launch_bounds__(kThreads) void hif8_encode_kernel(const float* __restrict__ x,
                                                               uint8_t* __restrict__ codes,
                                                               long long n, int saturate)
{
    const bool sat = saturate != 0;
    __shared__ uint8_t tab8[(EVEN ? 2 : 1) * kTabEntries];
    for (int i = threadIdx.x; i < kTabEntries; i += kThreads) {
        const float xi = hif8::u2f((uint32_t)i << kTabShift);
        tab8[i] = hif8::encode(xi, sat);
        if constexpr (EVEN) tab8[kTabEntries + i] = hif8::encode(xi, sat, true);
    }
    __syncthreads();
    const long long ngroups = n / 4;                              // 4-element groups
    const long long per_iter = (long long)gridDim.x * kThreads * kUnroll;
    const f32x4* src = reinterpret_cast<const f32x4*>(x);
    uint32_t* dst = reinterpret_cast<uint32_t*>(codes);
    for (long long g0 = (long long)blockIdx.x * kThreads * kUnroll + threadIdx.x; g0 < ngroups; g0 += per_iter) {
        f32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long long gi = g0 + (long long)u * kThreads;
            if (gi < ngroups) v[u] = __builtin_nontemporal_load(src + gi);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long long gi = g0 + (long long)u * kThreads;
            if (gi < ngroups) __builtin_nontemporal_store(encode4<EVEN>(tab8, v[u]), dst + gi);
        }
    }
    // ragged tail (fewer than 4 elements)
    const long long i = ngroups * 4 + (long long)blockIdx.x * kThreads + threadIdx.x;
    if (blockIdx.x == 0 && i < n) codes[i] = (uint8_t)encode1<EVEN>(tab8, x[i]);
}

__global__ __launch_bounds__(kThreads) void hif8_encode_scalar_kernel(const float* __restrict__ x,
                                                                      uint8_t* __restrict__ codes,
                                                                      long long n, int saturate, int even)
{
    const long long stride = (long long)gridDim.x * kThreads;
    for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        codes[i] = hif8::encode(x[i], saturate != 0, even != 0);
}

__global__ __launch_bounds__(kThreads) void hif8_decode_kernel(const uint8_t* __restrict__ codes,
                                                               float* __restrict__ x, long long n)
{
    __shared__ float lut[256];
    lut[threadIdx.x] = hif8::decode((uint8_t)threadIdx.x);
    __syncthreads();
    const long long ngroups = n / 4;
    const long long per_iter = (long long)gridDim.x * kThreads * kUnroll;
    const uint32_t* src = reinterpret_cast<const uint32_t*>(codes);
    f32x4* dst = reinterpret_cast<f32x4*>(x);
    for (long long g0 = (long long)blockIdx.x * kThreads * kUnroll + threadIdx.x; g0 < ngroups; g0 += per_iter) {
        uint32_t c[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long long gi = g0 + (long long)u * kThreads;
            if (gi < ngroups) c[u] = __builtin_nontemporal_load(src + gi);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const long long gi = g0 + (long long)u * kThreads;
            if (gi < ngroups) {
                f32x4 v = {lut[c[u] & 0xff], lut[(c[u] >> 8) & 0xff], lut[(c[u] >> 16) & 0xff], lut[c[u] >> 24]};
                __builtin_nontemporal_store(v, dst + gi);
            }
        }
    }
    const long long i = ngroups * 4 + (long long)blockIdx.x * kThreads + threadIdx.x;
    if (blockIdx.x == 0 && i < n) x[i] = lut[codes[i]];
}

__global__ __launch_bounds__(kThreads) void hif8_decode_scalar_kernel(const uint8_t* __restrict__ codes,
                                                                      float* __restrict__ x, long long n)
{
    const long long stride = (long long)gridDim.x * kThreads;
    for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        x[i] = hif8::decode(codes[i]);
}

int grid_for(long long work_items)
{
    long long g = (work_items + kThreads - 1) / kThreads;
    const long long cap = 256 * 8;               // 8 workgroups per CU, grid-stride beyond
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    return (int)g;
}

}  // namespace

hipError_t launch_hif8_encode(const float* x, uint8_t* codes, long long n, bool saturate, bool even, hipStream_t st)
{
    const bool aligned = ((uintptr_t)x % 16 == 0) && ((uintptr_t)codes % 4 == 0);
    const dim3 grid(grid_for(n / (4 * kUnroll) + 1));
    if (aligned && even)
        hipLaunchKernelGGL(hif8_encode_kernel<true>, grid, dim3(kThreads), 0, st, x, codes, n, (int)saturate);
    else if (aligned)
        hipLaunchKernelGGL(hif8_encode_kernel<false>, grid, dim3(kThreads), 0, st, x, codes, n, (int)saturate);
    else
        hipLaunchKernelGGL(hif8_encode_scalar_kernel, dim3(grid_for(n)), dim3(kThreads), 0, st,
                           x, codes, n, (int)saturate, (int)even);
    return hipGetLastError();
}

hipError_t launch_hif8_decode(const uint8_t* codes, float* x, long long n, hipStream_t st)
{
    const bool aligned = ((uintptr_t)x % 16 == 0) && ((uintptr_t)codes % 4 == 0);
    if (aligned)
        hipLaunchKernelGGL(hif8_decode_kernel, dim3(grid_for(n / (4 * kUnroll) + 1)), dim3(kThreads), 0, st,
                           codes, x, n);
    else
        hipLaunchKernelGGL(hif8_decode_scalar_kernel, dim3(grid_for(n)), dim3(kThreads), 0, st, codes, x, n);
    return hipGetLastError();
}

}  // namespace baps
