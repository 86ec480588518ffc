// Streaming HiF8 encode / decode kernels (HBM-bound, grid-stride).
#include "common.hpp"

namespace baps {

namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = 16;     // elements per thread per step: 64 B of fp32, 16 B of codes

__global__ __launch_bounds__(kThreads) void hif8_encode_kernel(const float* __restrict__ x,
                                                               uint8_t* __restrict__ codes,
                                                               long long n, int saturate)
{
    const long long nvec = n / kPerThread;
    const long long stride = (long long)gridDim.x * kThreads;
    const bool sat = saturate != 0;
    for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < nvec; i += stride) {
        const f32x4* src = reinterpret_cast<const f32x4*>(x) + i * 4;
        f32x4 a = __builtin_nontemporal_load(src + 0);
        f32x4 b = __builtin_nontemporal_load(src + 1);
        f32x4 c = __builtin_nontemporal_load(src + 2);
        f32x4 d = __builtin_nontemporal_load(src + 3);
        float e[16] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3],
                       c[0], c[1], c[2], c[3], d[0], d[1], d[2], d[3]};
        u32x4 out;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            uint32_t word = 0;
#pragma unroll
            for (int t = 0; t < 4; ++t) word |= (uint32_t)hif8::encode(e[w * 4 + t], sat) << (8 * t);
            out[w] = word;
        }
        __builtin_nontemporal_store(out, reinterpret_cast<u32x4*>(codes) + i);
    }
    // ragged tail
    for (long long i = nvec * kPerThread + (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        codes[i] = hif8::encode(x[i], sat);
}

__global__ __launch_bounds__(kThreads) void hif8_encode_scalar_kernel(const float* __restrict__ x,
                                                                      uint8_t* __restrict__ codes,
                                                                      long long n, int saturate)
{
    const long long stride = (long long)gridDim.x * kThreads;
    for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        codes[i] = hif8::encode(x[i], saturate != 0);
}

__global__ __launch_bounds__(kThreads) void hif8_decode_kernel(const uint8_t* __restrict__ codes,
                                                               float* __restrict__ x, long long n)
{
    __shared__ float lut[256];
    lut[threadIdx.x] = hif8::decode((uint8_t)threadIdx.x);
    __syncthreads();
    const long long nvec = n / kPerThread;
    const long long stride = (long long)gridDim.x * kThreads;
    for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < nvec; i += stride) {
        u32x4 c = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(codes) + i);
        f32x4* dst = reinterpret_cast<f32x4*>(x) + i * 4;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            f32x4 v;
            v[0] = lut[c[w] & 0xff];
            v[1] = lut[(c[w] >> 8) & 0xff];
            v[2] = lut[(c[w] >> 16) & 0xff];
            v[3] = lut[c[w] >> 24];
            __builtin_nontemporal_store(v, dst + w);
        }
    }
    for (long long i = nvec * kPerThread + (long long)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        x[i] = lut[codes[i]];
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
    const long long cap = 256 * 16;               // 16 workgroups per CU, grid-stride beyond
    if (g > cap) g = cap;
    if (g < 1) g = 1;
    return (int)g;
}

}  // namespace

hipError_t launch_hif8_encode(const float* x, uint8_t* codes, long long n, bool saturate, hipStream_t st)
{
    const bool aligned = ((uintptr_t)x % 16 == 0) && ((uintptr_t)codes % 16 == 0);
    if (aligned)
        hipLaunchKernelGGL(hif8_encode_kernel, dim3(grid_for(n / kPerThread + 1)), dim3(kThreads), 0, st,
                           x, codes, n, (int)saturate);
    else
        hipLaunchKernelGGL(hif8_encode_scalar_kernel, dim3(grid_for(n)), dim3(kThreads), 0, st,
                           x, codes, n, (int)saturate);
    return hipGetLastError();
}

hipError_t launch_hif8_decode(const uint8_t* codes, float* x, long long n, hipStream_t st)
{
    const bool aligned = ((uintptr_t)x % 16 == 0) && ((uintptr_t)codes % 16 == 0);
    if (aligned)
        hipLaunchKernelGGL(hif8_decode_kernel, dim3(grid_for(n / kPerThread + 1)), dim3(kThreads), 0, st,
                           codes, x, n);
    else
        hipLaunchKernelGGL(hif8_decode_scalar_kernel, dim3(grid_for(n)), dim3(kThreads), 0, st, codes, x, n);
    return hipGetLastError();
}

}  // namespace baps
