// The vector-side steps of Alg. 1 (block-aware precision rescaling) on fp32
// score rows that are already in log2 units: per key block, the row maximum,
// the restart decision of the B1 loop, the integer running maximum (Sec. 3.3),
// T = HiF8(S - ref), P = HiF8(2^T), and the running denominator.
//
// One wave owns one row.  The row streams through registers 1024 columns at
// a time (16 per lane, lane-interleaved so every load and store of the wave
// is contiguous); blocks inside a chunk are processed in order, which is the
// only sequential dependency of the method (the reference of block j depends
// on the running maximum after block j-1).  HBM-bound: 4 B read and 1 B
// written per score.
#include "common.hpp"

namespace baps {

namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerBlock = kThreads / 64;
constexpr int kChunk = 1024;               // columns per wave per step
constexpr int kPerLane = kChunk / 64;

template <int BLOCK>
__global__ __launch_bounds__(kThreads) void softmax_block_kernel(SoftmaxBlockParams p)
{
    __shared__ uint32_t tab[kTabEntries];
    for (int i = threadIdx.x; i < kTabEntries; i += kThreads) tab[i] = p.tab[i];
    __syncthreads();

    constexpr int kBPL = BLOCK / 64;                      // elements of a block per lane
    constexpr int kBlocksPerChunk = kChunk / BLOCK;
    const int lane = threadIdx.x & 63;
    const long long row = (long long)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= p.rows) return;

    const long long cols = p.cols;
    const long long nblk = (cols + BLOCK - 1) / BLOCK;
    const float* S = p.s + row * p.ld;
    uint8_t* code = p.codes + row * cols;
    int32_t* refs_out = p.ref_shift + row * nblk;
    const float ninf = -__builtin_huge_valf();

    float m = ninf;            // running integer maximum m^(j)
    float dl = 0.0f;           // this lane's share of the denominator d^(j)
    float myref = ninf;        // reference of block (64*g + lane) of the current group
    long long j = 0;

    float cur[kPerLane], nxt[kPerLane];
    auto load = [&](float* v, long long c0) {
#pragma unroll
        for (int i = 0; i < kPerLane; ++i) {
            const long long c = c0 + lane + 64 * i;
            v[i] = c < cols ? __builtin_nontemporal_load(S + c) : ninf;
        }
    };
    load(cur, 0);
    for (long long c0 = 0; c0 < cols; c0 += kChunk) {
        if (c0 + kChunk < cols) load(nxt, c0 + kChunk);
#pragma unroll
        for (int b = 0; b < kBlocksPerChunk; ++b) {
            if (j >= nblk) break;
            float M = ninf;
#pragma unroll
            for (int t = 0; t < kBPL; ++t) M = fmaxf(M, cur[b * kBPL + t]);
            M = wave_max_uniform(M);

            // Alg. 1: B0 blocks always take the high-precision path; B1 blocks
            // test ceil(rowmax T) > lambda with T = S - m~ cast to 8 bits.
            // HiF8 rounding is monotone, so rowmax of the cast T is the cast
            // of (rowmax S) - m~.
            bool restart;
            float tq = ninf;
            if (j < p.n_b0) {
                restart = true;
            } else {
                if (M != ninf) tq = hif8::round(M - m);     // m = -inf gives +inf: restart
                restart = ceilf(tq) > (float)p.lambda;
            }
            float m_new, ref;
            if (restart) {
                m_new = fmaxf(m, ceilf(M));
                ref = m_new;
            } else {
                m_new = m + fmaxf(0.0f, ceilf(tq));
                ref = m;
            }
            const float alpha = (m == ninf) ? 0.0f : exp2_int(m - m_new);
            const float beta = (ref == ninf) ? 0.0f : exp2_int(ref - m_new);

            float rowsum = 0.0f;
#pragma unroll
            for (int t = 0; t < kBPL; ++t) {
                const float s = cur[b * kBPL + t];
                const float T = (s == ninf || ref == ninf) ? ninf : s - ref;
                const uint32_t e = tab[hif8::f2u(T) >> kTabShift];
                const long long c = c0 + (long long)b * BLOCK + lane + 64 * t;
                if (c < cols) code[c] = (uint8_t)(e & 0xffu);
                rowsum += hif8::u2f(e & 0xffffff00u);
            }
            dl = alpha * dl + beta * rowsum;
            m = m_new;
            if (p.restarted && lane == 0) p.restarted[row * nblk + j] = restart ? 1 : 0;
            if (lane == (int)(j & 63)) myref = ref;
            if ((j & 63) == 63 || j == nblk - 1) {
                if (nblk > 64) {            // park the group's references until m is final
                    const long long idx = (j & ~63LL) + lane;
                    if (idx < nblk) refs_out[idx] = (int32_t)hif8::f2u(myref);
                }
            }
            ++j;
        }
#pragma unroll
        for (int i = 0; i < kPerLane; ++i) cur[i] = nxt[i];
    }

    const float d = wave_sum(dl);
    if (lane == 0) {
        p.m_final[row] = m;
        p.d_final[row] = d;
    }
    auto shift = [&](float ref) -> int32_t {
        if (ref == ninf || m == ninf) return INT32_MIN;
        return (int32_t)fmaxf(ref - m, -2147483520.0f);
    };
    if (nblk <= 64) {
        if (lane < nblk) refs_out[lane] = shift(myref);
    } else {
        for (long long idx = lane; idx < nblk; idx += 64)
            refs_out[idx] = shift(hif8::u2f((uint32_t)refs_out[idx]));
    }
}

// Row-group variant for 16-byte aligned rows whose length is a multiple of 4
// and blocks of at most 256 columns: a wave owns 4 rows and each row is a
// DPP row of 16 lanes, so the per-block maximum is 4 in-row DPP steps and the
// per-block state update runs for 4 rows at once.  A lane holds 4 adjacent
// columns per 64-column group: fp32x4 loads and 4-code stores, contiguous
// per row.
__device__ __forceinline__ float row16_max(float v)
{
    int o = __builtin_bit_cast(int, v);
    v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0xB1, 0xF, 0xF, false)));
    o = __builtin_bit_cast(int, v);
    v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x4E, 0xF, 0xF, false)));
    o = __builtin_bit_cast(int, v);
    v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x141, 0xF, 0xF, false)));
    o = __builtin_bit_cast(int, v);
    return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x140, 0xF, 0xF, false)));
}

__device__ __forceinline__ float row16_sum(float v)
{
    int o = __builtin_bit_cast(int, v);
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0xB1, 0xF, 0xF, false));
    o = __builtin_bit_cast(int, v);
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x4E, 0xF, 0xF, false));
    o = __builtin_bit_cast(int, v);
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x141, 0xF, 0xF, false));
    o = __builtin_bit_cast(int, v);
    return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x140, 0xF, 0xF, false));
}

constexpr int kRowsPerWave4 = 4;

// NT threads per workgroup, 4 rows per wave.  With rows enough to give every
// CU a workgroup, 1024 threads (64 rows, one workgroup and one 32 KiB table
// copy per CU) run about 10 % faster than 256 threads (four workgroups and
// four table copies per CU).  KCH columns of a row stream per step, and the
// next step's loads are in flight while one is processed.  256 columns keep
// the kernel at 64 VGPRs (8 waves per SIMD), which suits grids of many
// workgroups per CU and short rows; wider steps put more bytes in flight per
// wave where fewer waves share a CU: 512 columns (96 VGPRs) for rows of at
// least 4096 columns at 1024 threads, 1024 columns (162 VGPRs) for grids of
// at most two 256-thread workgroups per CU.
template <int BLOCK, int NT, int KCH>
__global__ __launch_bounds__(NT) void softmax_block4_kernel(SoftmaxBlockParams p)
{
    constexpr int kRows4PerBlock = kRowsPerWave4 * (NT / 64);
    __shared__ uint32_t tab[kTabEntries];
    for (int i = threadIdx.x; i < kTabEntries; i += NT) tab[i] = p.tab[i];
    __syncthreads();

    constexpr int kCh = BLOCK < KCH ? KCH : BLOCK;        // columns per row per step
    constexpr int kG = kCh / 64;                          // fp32x4 groups per lane per step
    constexpr int kGPB = BLOCK / 64;                      // groups per block (>= 1)
    constexpr int kBPS = kCh / BLOCK;                     // blocks per step
    const int lane = threadIdx.x & 63;
    const int sub = lane & 15;
    const long long row = (long long)blockIdx.x * kRows4PerBlock + (threadIdx.x >> 6) * kRowsPerWave4 + (lane >> 4);
    const bool row_ok = row < p.rows;                     // whole DPP rows agree
    const long long rr = row_ok ? row : 0;

    const long long cols = p.cols;
    const long long nblk = (cols + BLOCK - 1) / BLOCK;
    const float* S = p.s + rr * p.ld;
    uint8_t* code = p.codes + rr * cols;
    int32_t* refs_out = p.ref_shift + rr * nblk;
    const float ninf = -__builtin_huge_valf();

    float m = ninf, dl = 0.0f, myref = ninf;
    long long j = 0;
    f32x4 cur[kG], nxt[kG];
    auto load = [&](f32x4* v, long long c0) {
#pragma unroll
        for (int i = 0; i < kG; ++i) {
            const long long c = c0 + 64 * i + 4 * sub;
            v[i] = (row_ok && c < cols) ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(S + c))
                                        : f32x4{ninf, ninf, ninf, ninf};
        }
    };
    load(cur, 0);
    for (long long c0 = 0; c0 < cols; c0 += kCh) {
        if (c0 + kCh < cols) load(nxt, c0 + kCh);
#pragma unroll
        for (int bb = 0; bb < kBPS; ++bb) {
            if (j >= nblk) break;
            float M = ninf;
#pragma unroll
            for (int gi = 0; gi < kGPB; ++gi)
#pragma unroll
                for (int e = 0; e < 4; ++e) M = fmaxf(M, cur[bb * kGPB + gi][e]);
            M = row16_max(M);
            bool restart;
            float tq = ninf;
            if (j < p.n_b0) {
                restart = true;
            } else {
                if (M != ninf) tq = hif8::round(M - m);
                restart = ceilf(tq) > (float)p.lambda;
            }
            const float m_new = restart ? fmaxf(m, ceilf(M)) : m + fmaxf(0.0f, ceilf(tq));
            const float ref = restart ? m_new : m;
            const float alpha = (m == ninf) ? 0.0f : exp2_int(m - m_new);
            const float beta = (ref == ninf) ? 0.0f : exp2_int(ref - m_new);
            float rowsum = 0.0f;
#pragma unroll
            for (int gi = 0; gi < kGPB; ++gi) {
                uint32_t word = 0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float sv = cur[bb * kGPB + gi][e];
                    const float T = (sv == ninf || ref == ninf) ? ninf : sv - ref;
                    const uint32_t ent = tab[hif8::f2u(T) >> kTabShift];
                    word |= (ent & 0xffu) << (8 * e);
                    rowsum += hif8::u2f(ent & 0xffffff00u);
                }
                const long long c = c0 + (long long)bb * BLOCK + 64 * gi + 4 * sub;
                if (row_ok && c < cols) *reinterpret_cast<uint32_t*>(code + c) = word;
            }
            dl = alpha * dl + beta * rowsum;
            m = m_new;
            if (row_ok && p.restarted && sub == 0) p.restarted[rr * nblk + j] = restart ? 1 : 0;
            if (sub == (int)(j & 15)) myref = ref;
            if ((j & 15) == 15 || j == nblk - 1) {
                if (nblk > 16 && row_ok) {      // park the group's references until m is final
                    const long long idx = (j & ~15LL) + sub;
                    if (idx < nblk) refs_out[idx] = (int32_t)hif8::f2u(myref);
                }
            }
            ++j;
        }
#pragma unroll
        for (int i = 0; i < kG; ++i) cur[i] = nxt[i];
    }
    const float d = row16_sum(dl);
    if (!row_ok) return;
    if (sub == 0) {
        p.m_final[rr] = m;
        p.d_final[rr] = d;
    }
    auto shift = [&](float ref) -> int32_t {
        if (ref == ninf || m == ninf) return INT32_MIN;
        return (int32_t)fmaxf(ref - m, -2147483520.0f);
    };
    if (nblk <= 16) {
        if (sub < nblk) refs_out[sub] = shift(myref);
    } else {
        for (long long idx = sub; idx < nblk; idx += 16)
            refs_out[idx] = shift(hif8::u2f((uint32_t)refs_out[idx]));
    }
}

template <int NT, int KCH>
hipError_t launch_block4(const SoftmaxBlockParams& p, hipStream_t st)
{
    constexpr int kRows4PerBlock = kRowsPerWave4 * (NT / 64);
    const dim3 grid4((unsigned)((p.rows + kRows4PerBlock - 1) / kRows4PerBlock));
    switch (p.block) {
    case 64: hipLaunchKernelGGL((softmax_block4_kernel<64, NT, KCH>), grid4, dim3(NT), 0, st, p); break;
    case 128: hipLaunchKernelGGL((softmax_block4_kernel<128, NT, KCH>), grid4, dim3(NT), 0, st, p); break;
    default: hipLaunchKernelGGL((softmax_block4_kernel<256, NT, KCH>), grid4, dim3(NT), 0, st, p); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_softmax_block(const SoftmaxBlockParams& p, hipStream_t st)
{
    const bool vec = ((uintptr_t)p.s % 16 == 0) && (p.ld % 4 == 0) && (p.cols % 4 == 0) &&
                     ((uintptr_t)p.codes % 4 == 0) && p.block <= 256;
    if (vec) {
        // one 1024-thread workgroup per CU when the rows fill every CU
        static std::atomic<int> ncu_of[64] = {};    // CU count per device, read once
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        int ncu = (dev >= 0 && dev < 64) ? ncu_of[dev].load(std::memory_order_relaxed) : 0;
        if (ncu == 0) {
            e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
            if (e != hipSuccess) return e;
            if (dev >= 0 && dev < 64) ncu_of[dev].store(ncu, std::memory_order_relaxed);
        }
        const long long wg1024 = (p.rows + 4 * 16 - 1) / (4 * 16);
        if (wg1024 >= ncu) return p.cols >= 4096 ? launch_block4<1024, 512>(p, st) : launch_block4<1024, 256>(p, st);
        // fewer rows than CUs x 64: at most two 256-thread workgroups per CU
        // take 1024 columns per step (162 VGPRs), more take 256
        const long long wg256 = (p.rows + 4 * 4 - 1) / (4 * 4);
        return wg256 <= 2 * ncu ? launch_block4<256, 1024>(p, st) : launch_block4<256, 256>(p, st);
    }
    const dim3 grid((unsigned)((p.rows + kRowsPerBlock - 1) / kRowsPerBlock));
    switch (p.block) {
    case 64: hipLaunchKernelGGL(softmax_block_kernel<64>, grid, dim3(kThreads), 0, st, p); break;
    case 128: hipLaunchKernelGGL(softmax_block_kernel<128>, grid, dim3(kThreads), 0, st, p); break;
    case 256: hipLaunchKernelGGL(softmax_block_kernel<256>, grid, dim3(kThreads), 0, st, p); break;
    case 512: hipLaunchKernelGGL(softmax_block_kernel<512>, grid, dim3(kThreads), 0, st, p); break;
    case 1024: hipLaunchKernelGGL(softmax_block_kernel<1024>, grid, dim3(kThreads), 0, st, p); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace baps
