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
            M = wave_max(M);

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

}  // namespace

hipError_t launch_softmax_block(const SoftmaxBlockParams& p, hipStream_t st)
{
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
