// Fused BAPS attention forward (Alg. 1, the "E2E HiF8" workflow) for gfx950.
//
// One workgroup = 4 waves = 128 query rows of one key/value head: the rows
// are the flattened (query position, query head of the group) pairs, so GQA
// heads that share K/V share the workgroup, and batched decode (one query
// position) packs its Hq/Hkv heads into one tile.  Each wave owns 32 rows.
//
// Per key block j (the paper's key tile, processed in ascending order):
//   - K_j and V_j are staged in LDS (V transposed, so that the key index is
//     contiguous for the MFMA operand);
//   - S^T = K_j Q^T on v_mfma_f32_32x32x16_bf16, fp32 accumulate.  In the
//     S^T layout a lane holds 16 keys of one query per 32-key tile, so the
//     row maximum is an in-lane max plus one exchange with lane^32;
//   - the restart rule of Alg. 1 and the integer maximum of Sec. 3.3 run per
//     query row (R8 per-row reading), with exact power-of-two rescales;
//   - T = fl32(acc * c - ref) (eq. 3: the scale and the subtraction are one
//     fused operation, rounded once), then P = HiF8(2^HiF8(T)) read from a
//     table indexed by bits 31..19 of T (HiF8 rounding to nearest-away
//     depends on those bits only);
//   - the fp32 accumulator layout of S^T is directly the B operand layout of
//     O^T = V_j^T P^T (the key order inside each 16-key group is permuted
//     consistently on both operands), so P never leaves registers.
#include "common.hpp"

namespace baps {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerWave = 32;
constexpr int kTileRows = kWaves * kRowsPerWave;

template <int D, int BLK>
struct Smem {
    static constexpr int kKStride = D + 8;       // u16 per K row in LDS (pad: 16 B)
    static constexpr int kVStride = BLK + 8;     // u16 per V^T row in LDS
    uint16_t k[BLK * kKStride];
    uint16_t vt[D * kVStride];
    uint16_t tab[kTabEntries];                   // P as bf16, indexed by T >> 19
};

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int D, int BLK>
__global__ __launch_bounds__(kThreads) void baps_attn_fwd_kernel(AttnParams p)
{
    static_assert(D % 32 == 0 && BLK % 32 == 0, "tile shape");
    using SM = Smem<D, BLK>;
    __shared__ __attribute__((aligned(16))) SM sm;

    constexpr int kKT = BLK / 32;                 // 32-key tiles per block
    constexpr int kDK = D / 16;                   // 16-wide d chunks (QK^T contraction)
    constexpr int kDT = D / 32;                   // 32-wide d tiles of O^T
    constexpr int kPC = BLK / 16;                 // 16-key chunks (PV contraction)

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int j32 = lane & 31;
    const int half = lane >> 5;

    const int G = p.Hq / p.Hkv;
    const int flat_rows = p.Sq * G;
    const int ntiles = (flat_rows + kTileRows - 1) / kTileRows;
    const int tile = ntiles - 1 - (int)blockIdx.x;         // longest causal tiles first
    const int g = blockIdx.y;
    const int b = blockIdx.z;

    for (int i = tid; i < kTabEntries; i += kThreads) sm.tab[i] = (uint16_t)(p.tab[i] >> 16);

    // this lane's query row: flat index f = r * G + h_local
    const int f = tile * kTileRows + wave * kRowsPerWave + j32;
    const bool row_ok = f < flat_rows;
    const int r = row_ok ? f / G : 0;
    const int h = g * G + (row_ok ? f % G : 0);
    const int off = p.Sk - p.Sq;                            // bottom-right causal alignment
    const int kmax = p.causal ? min(p.Sk - 1, r + off) : p.Sk - 1;

    // wave / workgroup extents of the key loop
    int kmax_wave_hi = row_ok ? kmax : -1;
    int kmax_wave_lo = row_ok ? kmax : 0x7fffffff;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        kmax_wave_hi = max(kmax_wave_hi, __shfl_xor(kmax_wave_hi, o, 64));
        kmax_wave_lo = min(kmax_wave_lo, __shfl_xor(kmax_wave_lo, o, 64));
    }
    int kmax_tile;
    {
        const int f_last = min(flat_rows - 1, tile * kTileRows + kTileRows - 1);
        int kt_hi = -1;
        // rows of a tile are consecutive positions; the largest position is the last row
        const int r_last = f_last / G;
        kt_hi = p.causal ? min(p.Sk - 1, r_last + off) : p.Sk - 1;
        kmax_tile = kt_hi;
    }
    const int nblk = kmax_tile < 0 ? 0 : kmax_tile / BLK + 1;

    // Q^T as the B operand of S^T = K Q^T: lane holds Q[row][16*kk + 8*half .. +8]
    u32x4 qop[kDK];
    {
        const uint16_t* qrow = p.q + (((long long)b * p.Hq + h) * p.Sq + r) * D;
#pragma unroll
        for (int kk = 0; kk < kDK; ++kk) {
            if (row_ok) qop[kk] = *reinterpret_cast<const u32x4*>(qrow + kk * 16 + half * 8);
            else qop[kk] = u32x4{0, 0, 0, 0};
        }
    }

    const uint16_t* kbase = p.k + ((long long)b * p.Hkv + g) * (long long)p.Sk * D;
    const uint16_t* vbase = p.v + ((long long)b * p.Hkv + g) * (long long)p.Sk * D;
    const float ninf = -__builtin_huge_valf();
    const float c = p.c;

    float m = ninf;                 // running integer maximum of this lane's row
    float dl = 0.0f;                // this lane's share of the denominator
    unsigned n_restart = 0, n_visit = 0;
    f32x16 oacc[kDT];
#pragma unroll
    for (int t = 0; t < kDT; ++t) oacc[t] = f32x16{};

    for (int jb = 0; jb < nblk; ++jb) {
        const int key0 = jb * BLK;
        __syncthreads();                                    // previous block's LDS reads done
        // stage K_j row-major and V_j transposed; rows past Sk are zeros
        for (int i = tid; i < BLK * (D / 8); i += kThreads) {
            const int kr = i / (D / 8);
            const int d8 = i % (D / 8);
            u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
            if (key0 + kr < p.Sk) {
                kv = *reinterpret_cast<const u32x4*>(kbase + (long long)(key0 + kr) * D + d8 * 8);
                vv = *reinterpret_cast<const u32x4*>(vbase + (long long)(key0 + kr) * D + d8 * 8);
            }
            *reinterpret_cast<u32x4*>(&sm.k[kr * SM::kKStride + d8 * 8]) = kv;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                sm.vt[(d8 * 8 + 2 * e) * SM::kVStride + kr] = (uint16_t)(vv[e] & 0xffffu);
                sm.vt[(d8 * 8 + 2 * e + 1) * SM::kVStride + kr] = (uint16_t)(vv[e] >> 16);
            }
        }
        __syncthreads();
        if (key0 > kmax_wave_hi) continue;                  // nothing visible for this wave

        // S^T = K_j Q^T
        f32x16 sacc[kKT];
#pragma unroll
        for (int kt = 0; kt < kKT; ++kt) {
            sacc[kt] = f32x16{};
#pragma unroll
            for (int kk = 0; kk < kDK; ++kk) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(
                    &sm.k[(kt * 32 + j32) * SM::kKStride + kk * 16 + half * 8]);
                sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(qop[kk]),
                                                                    sacc[kt], 0, 0, 0);
            }
        }
        // mask keys past kmax (causal diagonal, ragged tail); key of register
        // i of tile kt: key0 + 32*kt + 8*(i/4) + 4*half + i%4
        if (key0 + BLK - 1 > kmax_wave_lo) {
#pragma unroll
            for (int kt = 0; kt < kKT; ++kt)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = key0 + kt * 32 + 8 * (i / 4) + 4 * half + (i % 4);
                    if (key > kmax) sacc[kt][i] = ninf;
                }
        }
        // row maximum of the raw dot products (the scale c > 0 is monotone)
        float amax = ninf;
#pragma unroll
        for (int kt = 0; kt < kKT; ++kt)
#pragma unroll
            for (int i = 0; i < 16; ++i) amax = fmaxf(amax, sacc[kt][i]);
        amax = fmaxf(amax, __shfl_xor(amax, 32, 64));

        // block-aware precision rescaling (Alg. 1), per row
        float ref, ab, beta;                 // ab = alpha / beta, exact powers of two
        if (amax == ninf) {                  // no visible key in this block: no-op
            ref = 0.0f; ab = 1.0f; beta = 1.0f;
        } else {
            bool restart;
            float tq = 0.0f;
            if (jb < p.n_b0 || m == ninf) {
                restart = true;
            } else {
                tq = hif8::round(__builtin_fmaf(amax, c, -m));   // rowmax of the 8-bit T
                restart = ceilf(tq) > (float)p.lambda;
                ++n_visit;
                n_restart += restart ? 1u : 0u;
            }
            float m_new;
            if (restart) {
                m_new = fmaxf(m, ceilf(amax * c));               // ceil(rowmax S), S in fp32
                ref = m_new;
            } else {
                m_new = m + fmaxf(0.0f, ceilf(tq));
                ref = m;
            }
            ab = (m == ninf) ? 0.0f : exp2_int(m - ref);
            beta = exp2_int(ref - m_new);
            m = m_new;
        }

        // P = HiF8(2^HiF8(T)), T = fl32(acc * c - ref); packed as bf16 B operands
        u32x4 pop[kPC];
        float rs = 0.0f;
#pragma unroll
        for (int kt = 0; kt < kKT; ++kt) {
#pragma unroll
            for (int ch = 0; ch < 2; ++ch) {
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float t0 = __builtin_fmaf(sacc[kt][ch * 8 + 2 * e], c, -ref);
                    const float t1 = __builtin_fmaf(sacc[kt][ch * 8 + 2 * e + 1], c, -ref);
                    const uint32_t p0 = sm.tab[hif8::f2u(t0) >> kTabShift];
                    const uint32_t p1 = sm.tab[hif8::f2u(t1) >> kTabShift];
                    rs += hif8::u2f(p0 << 16);
                    rs += hif8::u2f(p1 << 16);
                    w[e] = p0 | (p1 << 16);
                }
                pop[kt * 2 + ch] = u32x4{w[0], w[1], w[2], w[3]};
            }
        }

        // d = alpha d + beta rowsum and O~ = alpha O~ + beta P V, written as
        // beta * ((alpha/beta) X + Y): identical in fp32, powers of two are exact
        if (__any(ab != 1.0f)) {
#pragma unroll
            for (int t = 0; t < kDT; ++t)
#pragma unroll
                for (int i = 0; i < 16; ++i) oacc[t][i] *= ab;
        }
        dl = dl * ab + rs;

        // O~^T += V_j^T P^T; A operand: lane holds V^T[d][keys] for the same
        // permuted 16-key order as the B operand taken from the S^T layout
#pragma unroll
        for (int pc = 0; pc < kPC; ++pc) {
            const int kb0 = pc * 16 + 4 * half;
#pragma unroll
            for (int t = 0; t < kDT; ++t) {
                const uint16_t* vr = &sm.vt[(t * 32 + j32) * SM::kVStride];
                const u32x2 lo = *reinterpret_cast<const u32x2*>(vr + kb0);
                const u32x2 hi = *reinterpret_cast<const u32x2*>(vr + kb0 + 8);
                const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
                oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(pop[pc]),
                                                                   oacc[t], 0, 0, 0);
            }
        }
        if (__any(beta != 1.0f)) {
#pragma unroll
            for (int t = 0; t < kDT; ++t)
#pragma unroll
                for (int i = 0; i < 16; ++i) oacc[t][i] *= beta;
        }
        dl *= beta;
    }

    // epilogue: O = diag(d)^-1 O~, lse = ln2 (m + log2 d)
    const float d = dl + __shfl_xor(dl, 32, 64);
    if (!row_ok) return;
    float* orow = p.o + (((long long)b * p.Hq + h) * p.Sq + r) * D;
    const bool empty = (m == ninf);
#pragma unroll
    for (int t = 0; t < kDT; ++t)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            f32x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = empty ? 0.0f : oacc[t][q4 * 4 + e] / d;
            *reinterpret_cast<f32x4*>(orow + t * 32 + q4 * 8 + half * 4) = v;
        }
    if (half == 0) {
        if (p.lse) p.lse[((long long)b * p.Hq + h) * p.Sq + r] = empty ? ninf : 0.69314718055994531f * (m + log2f(d));
        if (p.counters && n_visit) {
            atomicAdd(p.counters + 2 * ((long long)b * p.Hq + h) + 0, (unsigned long long)n_restart);
            atomicAdd(p.counters + 2 * ((long long)b * p.Hq + h) + 1, (unsigned long long)n_visit);
        }
    }
}

template <int D, int BLK>
hipError_t launch_one(const AttnParams& p, hipStream_t st)
{
    const int G = p.Hq / p.Hkv;
    const long long flat = (long long)p.Sq * G;
    const dim3 grid((unsigned)((flat + kTileRows - 1) / kTileRows), (unsigned)p.Hkv, (unsigned)p.B);
    hipLaunchKernelGGL((baps_attn_fwd_kernel<D, BLK>), grid, dim3(kThreads), 0, st, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnParams& p, int D, int block, hipStream_t st)
{
    if (D == 64 && block == 64) return launch_one<64, 64>(p, st);
    if (D == 64 && block == 128) return launch_one<64, 128>(p, st);
    if (D == 128 && block == 64) return launch_one<128, 64>(p, st);
    if (D == 128 && block == 128) return launch_one<128, 128>(p, st);
    if (D == 64 && block == 32) return launch_one<64, 32>(p, st);
    if (D == 128 && block == 32) return launch_one<128, 32>(p, st);
    return hipErrorInvalidValue;
}

}  // namespace baps
