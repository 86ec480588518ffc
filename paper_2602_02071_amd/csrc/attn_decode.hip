// Fused BAPS attention forward for few query rows per key/value head
// (batched decode, speculative or chunked short queries).  Same method and
// state machine as the prefill kernel (Alg. 1 per query row, block-aware
// rescaling, HiF8 T and P), shaped for the HBM-bound regime:
//
//   - a workgroup owns up to 16 flattened (query position, query head of the
//     group) rows of one key/value head, on 16x16x32 bf16 MFMAs;
//   - its BLK/32 waves split every key block: wave w takes the 32 keys
//     [32w, 32w + 32) of each block, so the waves stream disjoint parts of
//     the K/V rows concurrently;
//   - per block the waves exchange their partial row maxima through LDS (one
//     barrier) and then all take the same Alg. 1 decision from the same
//     maximum, so every wave holds the same reference; their output and
//     denominator partials are therefore on one scale and are summed once at
//     the end;
//   - each wave streams its K and V slots through its own LDS ring, filled by
//     asynchronous global->LDS loads kept RW slots ahead; a slot is consumed
//     after the vector-memory counter says it landed and refilled right after.
#include "common.hpp"

namespace baps {

namespace {

typedef __bf16 bf16x2 __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef short s16x4 __attribute__((ext_vector_type(4)));
#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

constexpr int kRows = 16;            // query rows per workgroup
constexpr int kSlotKeys = 32;        // keys per ring slot

template <int D, int BLK>
struct DCfg {
    static constexpr int kWaves = BLK / kSlotKeys;              // one wave per 32-key slot of a block
    static constexpr int kRowBytes = 2 * D;
    static constexpr int kCPR = D / 8;                          // 16-byte chunks per row
    static constexpr int kSlotBytes = kSlotKeys * kRowBytes;    // 8 KiB (D=128), 4 KiB (D=64)
    static constexpr int kIPS = kSlotBytes / 1024;              // wave-wide loads per slot
    // ring slots per wave: about 64 KiB of ring per workgroup, at least 2,
    // and at most 63 loads outstanding per wave
    static constexpr int kRW0 = (64 * 1024) / (kWaves * kSlotBytes);
    static constexpr int kRW = kRW0 < 2 ? 2 : (kRW0 * kIPS > 63 ? 63 / kIPS : kRW0);
    static constexpr int kLdsBytes = kWaves * kRW * kSlotBytes;
};

// chunk swizzles (same bank-conflict reasoning as the prefill kernel): K rows
// are read 16 at a time at one logical chunk, V rows 4 at a time, 2 chunks
template <int D>
__device__ __forceinline__ int k_swz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
template <int D>
__device__ __forceinline__ int v_swz(int r) { return D == 128 ? 2 * (r & 3) : 2 * ((r >> 1) & 1); }
// FP8 K rows (D bytes), read 16 rows at a time at one logical chunk
template <int D>
__device__ __forceinline__ int k8_swz(int r) { return D == 128 ? ((r ^ ((r >> 3) & 1)) & 7) : ((r >> 2) & 3); }

typedef int i32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ i32x8 cat8(u32x4 a, u32x4 b)
{
    return i32x8{(int)a[0], (int)a[1], (int)a[2], (int)a[3], (int)b[0], (int)b[1], (int)b[2], (int)b[3]};
}

// One wave-wide asynchronous global->LDS load of 1 KiB, marked non-temporal:
// every K/V byte is read once, so the stream should not displace cached data
__device__ __forceinline__ void lds_dma_16(const void* gptr, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt"
                 :
                 : "v"(gptr), "s"(lds_base)
                 : "memory", "m0");
}

// wait until at most n wave-wide loads of this wave are outstanding (n is
// rounded down to a multiple of 4: waiting longer is always safe)
__device__ __forceinline__ void wait_vm(int n)
{
    switch (n < 0 ? 0 : (n > 60 ? 60 : (n & ~3))) {
#define W(N) case N: __builtin_amdgcn_s_waitcnt(0xF70 | ((N) & 15) | ((((N) >> 4) & 3) << 14)); break;
        W(0) W(4) W(8) W(12) W(16) W(20) W(24) W(28) W(32) W(36) W(40) W(44) W(48) W(52) W(56) W(60)
#undef W
    default: __builtin_amdgcn_s_waitcnt(0xF70); break;
    }
}

// TIE: the 8-bit cast of T rounds ties to even (a second code table covers
// the T whose bits 18..0 are zero).  DUMP: also write the raw dot products and
// block references of the rows the caller marks (AttnParams::dump_slot).
template <int D, int BLK, bool CT, int MODE, bool F8, bool TIE, bool DUMP>
__global__ __launch_bounds__(64 * (BLK / 32)) void baps_attn_decode_kernel(AttnParams p)
{
    static_assert(MODE == kModeE2E || CT, "the eq. (2) setups use the compact table (T <= 0)");
    static_assert(!TIE || (MODE == kModeE2E && CT && !F8), "ties to even: canonical path");
    static_assert(D == 64 || D == 128, "head dimension");
    static_assert(BLK % kSlotKeys == 0 && BLK <= 128, "key block");
    using C = DCfg<D, BLK>;
    constexpr int KW = C::kWaves;
    constexpr int RW = C::kRW;
    // P lookup: the compact code table (lambda <= kCodeMaxLambda), else the
    // bf16 half of the full score table
    __shared__ __attribute__((aligned(16))) uint8_t ctab[CT ? kCodeHi + 1 : 1];
    __shared__ __attribute__((aligned(16))) uint8_t ctab_e[TIE ? kCodeHi + 1 : 1];
    __shared__ __attribute__((aligned(16))) uint16_t tab[CT ? 1 : kTabEntries];
    __shared__ float xch[2][KW][kRows];           // partial row maxima, by block parity
    extern __shared__ __attribute__((aligned(1024))) char ring[];
    const uint32_t ring_lds = (uint32_t)(uintptr_t)LDS_PTR(char, ring);

    constexpr int kDK = D / 32;                   // 32-wide d chunks (QK^T contraction)
    constexpr int kDT = D / 16;                   // 16-wide d tiles of O^T

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c16 = lane & 15;                    // query column of this lane
    const int grp = lane >> 4;                    // lane group 0..3

    const int G = p.Hq / p.Hkv;
    const int flat_rows = p.Sq * G;
    const int tile = blockIdx.x;
    const int g = blockIdx.y;
    const int b = blockIdx.z;
    const uint16_t* kbase = p.k + ((long long)b * p.Hkv + g) * (long long)p.Sk * D;
    const uint8_t* kbase8 = reinterpret_cast<const uint8_t*>(p.k) + ((long long)b * p.Hkv + g) * (long long)p.Sk * D;
    const uint16_t* vbase = p.v + ((long long)b * p.Hkv + g) * (long long)p.Sk * D;
    constexpr int kIPS8 = kSlotKeys * D / 1024;   // loads of an FP8 K slot (half a slot)

    const int off = p.Sk - p.Sq;
    const int f_last = min(flat_rows - 1, tile * kRows + kRows - 1);
    const int kmax_tile = p.causal ? min(p.Sk - 1, f_last / G + off) : p.Sk - 1;
    const int nblk = kmax_tile < 0 ? 0 : kmax_tile / BLK + 1;
    const int nslots = 2 * nblk;                  // this wave's slots: K then V of each block

    // slot n of this wave: block n/2, keys 32*wave .. +32 of the block; K if n is even
    const uint32_t my_ring_lds = ring_lds + (uint32_t)(wave * RW * C::kSlotBytes);
    const char* my_ring = ring + wave * RW * C::kSlotBytes;
    auto issue_slot = [&](int n) {
        const int jb = n >> 1;
        const bool is_v = (n & 1) != 0;
        const int key0 = jb * BLK + wave * kSlotKeys;
        const uint32_t dst = my_ring_lds + (uint32_t)((n % RW) * C::kSlotBytes);
        if (F8 && !is_v) {                        // FP8 K: rows of D bytes
#pragma unroll
            for (int t = 0; t < kIPS8; ++t) {
                const int r = t * (1024 / D) + lane / (D / 16);
                const int ch = (lane % (D / 16)) ^ k8_swz<D>(r);
                const int key = min(key0 + r, p.Sk - 1);
                lds_dma_16(kbase8 + (long long)key * D + ch * 16, dst + t * 1024);
            }
            return;
        }
        const uint16_t* base = is_v ? vbase : kbase;
#pragma unroll
        for (int t = 0; t < C::kIPS; ++t) {
            const int r = t * (1024 / C::kRowBytes) + lane / C::kCPR;
            const int pch = lane % C::kCPR;
            const int ch = pch ^ (is_v ? v_swz<D>(r) : k_swz<D>(r));
            const int key = min(key0 + r, p.Sk - 1);
            lds_dma_16(base + (long long)key * D + ch * 8, dst + t * 1024);
        }
    };
    int issued = 0;
    for (; issued < min(nslots, RW); ++issued) issue_slot(issued);

    if constexpr (MODE == kModeDefault) {
        // fp32 exp2: no table
    } else if constexpr (CT) {
        for (int i = tid; i < kCodeEntries; i += 64 * KW) ctab[kCodeLo + i] = p.ctab[i];
        if constexpr (TIE)
            for (int i = tid; i < kCodeEntries; i += 64 * KW) ctab_e[kCodeLo + i] = p.ctab_even[i];
    } else {
        for (int i = tid; i < kTabEntries; i += 64 * KW) tab[i] = (uint16_t)(p.tab[i] >> 16);
    }

    // this lane's query row
    const int f = tile * kRows + c16;
    const bool row_ok = f < flat_rows;
    const int r = row_ok ? f / G : 0;
    const int h = g * G + (row_ok ? f % G : 0);
    const int kmax = row_ok ? (p.causal ? min(p.Sk - 1, r + off) : p.Sk - 1) : -1;
    int dslot = -1;
    if constexpr (DUMP) dslot = row_ok ? p.dump_slot[((long long)b * p.Hq + h) * p.Sq + r] : -1;
    // tile-level restart (restart_rows > 1, then restart_rows * G <= 16): the
    // rows c16 == h_local (mod G) of an aligned span of restart_rows * G rows
    // of the 16 share each block's decision; a ballot takes it
    const bool tiled = p.restart_rows > 1;
    uint32_t tmask = 0;
    if (tiled) {
        const int RG = p.restart_rows * G;
        uint32_t pat = 0;
        for (int j = 0; j < kRows; j += G) pat |= 1u << j;
        tmask = (pat << (c16 % G)) & (((1u << RG) - 1u) << (RG * (c16 / RG)));
    }
    const bool trep = !tiled || c16 == __builtin_ctz(tmask | 0x10000u);   // this lane counts its tile
    int kmax_lo = row_ok ? kmax : 0x7fffffff;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) kmax_lo = min(kmax_lo, __shfl_xor(kmax_lo, o, 64));
    kmax_lo = __builtin_amdgcn_readfirstlane(kmax_lo);

    // Q^T as the B operand of S^T = K Q^T (16x16x32): lane holds
    // Q[row][32*kk + 8*grp .. +8]; K uses the same d order
    // (FP8: one 16x16x128 MFMA, lane holds Q[row][32*grp .. +32]; zeros past D)
    u32x4 qop[F8 ? 1 : kDK];
    i32x8 qop8 = {};
    if constexpr (F8) {
        const uint8_t* qrow = reinterpret_cast<const uint8_t*>(p.q) + (((long long)b * p.Hq + h) * p.Sq + r) * D;
        if (row_ok && 32 * grp < D)
            qop8 = cat8(*reinterpret_cast<const u32x4*>(qrow + 32 * grp),
                        *reinterpret_cast<const u32x4*>(qrow + 32 * grp + 16));
    } else {
        const uint16_t* qrow = p.q + (((long long)b * p.Hq + h) * p.Sq + r) * D;
#pragma unroll
        for (int kk = 0; kk < kDK; ++kk)
            qop[kk] = row_ok ? *reinterpret_cast<const u32x4*>(qrow + kk * 32 + grp * 8) : u32x4{0, 0, 0, 0};
    }

    const float ninf = -__builtin_huge_valf();
    const float c = p.c;
    const float lam = (float)p.lambda;
    // Alg. 1 state (the same in every wave); output and denominator partials
    // kept relative to the current block reference
    float m = ninf, ref = ninf, dl = 0.0f;
    unsigned n_restart = 0, n_visit = 0;
    f32x4 oacc[kDT];
#pragma unroll
    for (int t = 0; t < kDT; ++t) oacc[t] = f32x4{};

    const int kx = k_swz<D>(c16);                 // K rows 16*t2 + c16
    const uint32_t krow = c16 * C::kRowBytes;
    const int vrow0 = 4 * grp + c16 / 4;          // +16 for slots 4..7
    const int vx = v_swz<D>(vrow0);
    const int vd0 = 4 * (c16 & 3);                // + 16*dt
    const uint32_t vrow = vrow0 * C::kRowBytes + 2 * (vd0 & 7);

    int consumed = 0;
    // loads issued after slot n (K slots are even; FP8 K slots carry kIPS8 loads)
    auto wait_slot = [&](int n) {
        if constexpr (F8) {
            const int nv = issued / 2 - (n + 1) / 2;
            const int nk = issued - 1 - n - nv;
            wait_vm(nv * C::kIPS + nk * kIPS8);
        } else {
            wait_vm((issued - 1 - n) * C::kIPS);
        }
    };
    auto next_slot = [&]() {
        if (issued < nslots) { issue_slot(issued); ++issued; }
        ++consumed;
    };
    __syncthreads();                              // code table published

    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    for (int jb = 0; jb < nblk; ++jb) {
        const int key0 = jb * BLK + wave * kSlotKeys;   // this wave's first key of the block
        // S^T = K Q^T for this wave's 32 keys: two 16-key tiles
        f32x4 sacc[2];
        {
            wait_slot(consumed);
            const char* slot = my_ring + (consumed % RW) * C::kSlotBytes;
            if constexpr (F8) {
                // FP8 E4M3 K rows of D bytes; lane reads bytes [32 grp, +32) of key row 16 t2 + c16
                const int kx8 = k8_swz<D>(c16);   // the same for rows c16 and 16 + c16
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2) {
                    i32x8 a8 = {};
                    if (32 * grp < D) {
                        const char* kr = slot + (16 * t2 + c16) * D;
                        a8 = cat8(*reinterpret_cast<const u32x4*>(kr + 16 * ((2 * grp) ^ kx8)),
                                  *reinterpret_cast<const u32x4*>(kr + 16 * ((2 * grp + 1) ^ kx8)));
                    }
                    sacc[t2] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a8, qop8, f32x4{}, 0, 0, 0, 127, 0, 127);
                }
            } else {
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2) {
                    f32x4 acc = {};
#pragma unroll
                    for (int kk = 0; kk < kDK; ++kk) {
                        const u32x4 a = *reinterpret_cast<const u32x4*>(
                            slot + krow + t2 * 16 * C::kRowBytes + 16 * ((4 * kk + grp) ^ kx));
                        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(qop[kk]), acc, 0, 0, 0);
                    }
                    sacc[t2] = acc;
                }
            }
            next_slot();
        }
        // mask keys past kmax; register i of tile t2 holds key key0 + 16*t2 + 4*grp + i
        if (key0 + kSlotKeys - 1 > kmax_lo) {
            asm volatile("" ::: "memory");
            const int lim = kmax - key0 - 4 * grp;
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (16 * t2 + i > lim) sacc[t2][i] = ninf;
        }
        if constexpr (DUMP) {
            if (dslot >= 0) {
                float* dst = p.dump_acc + (long long)dslot * p.Sk;
#pragma unroll
                for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = key0 + 16 * t2 + 4 * grp + i;
                        if (key <= kmax) dst[key] = sacc[t2][i];
                    }
            }
        }
        // row maximum of the block: this wave's 32 keys, then across the waves
        float pm = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(sacc[0][0], sacc[0][1]), sacc[0][2]),
                                   __builtin_fmaxf(__builtin_fmaxf(sacc[0][3], sacc[1][0]), sacc[1][1]));
        pm = __builtin_fmaxf(pm, __builtin_fmaxf(sacc[1][2], sacc[1][3]));
        pm = __builtin_fmaxf(pm, __shfl_xor(pm, 16, 64));
        pm = __builtin_fmaxf(pm, __shfl_xor(pm, 32, 64));
        float amax = pm;
        if constexpr (KW > 1) {
            if (grp == 0) xch[jb & 1][wave][c16] = pm;
            __syncthreads();
            amax = xch[jb & 1][0][c16];
#pragma unroll
            for (int w = 1; w < KW; ++w) amax = __builtin_fmaxf(amax, xch[jb & 1][w][c16]);
        }

        float nref;
        if constexpr (MODE == kModeE2E) {
            // block-aware precision rescaling (Alg. 1), per row or per tile (see
            // the prefill kernel)
            const bool vis = row_ok && amax != ninf;
            const bool in_b0 = (jb < p.n_b0) || (p.b0_last && jb == kmax / BLK);
            const bool forced = in_b0 || (m == ninf);
            const float tq = hif8::round(__builtin_fmaf(amax, c, -m), true, TIE);
            bool restart = forced || (ceilf(tq) > lam);
            bool b1 = vis && !in_b0;
            if (tiled) {
                const uint32_t wantb = (uint32_t)__ballot(vis && restart) & tmask;
                const uint32_t visb = (uint32_t)__ballot(vis) & tmask;
                const uint32_t b0b = (uint32_t)__ballot(vis && in_b0) & tmask;
                restart = wantb != 0u;
                b1 = visb != 0u && b0b == 0u;
            }
            const float m_hi = __builtin_fmaxf(m, ceilf(amax * c));
            const float m_new = vis ? (restart ? m_hi : m + __builtin_fmaxf(0.0f, ceilf(tq))) : m;
            const float ref_new = vis ? (restart ? m_hi : m) : ref;
            n_visit += (b1 && trep) ? 1u : 0u;
            n_restart += (b1 && trep && restart) ? 1u : 0u;
            const float fac = (ref == ninf) ? 1.0f : exp2_int(ref - ref_new);
            if (__any(fac != 1.0f)) {
    #pragma unroll
                for (int t = 0; t < kDT; ++t)
    #pragma unroll
                    for (int i = 0; i < 4; ++i) oacc[t][i] *= fac;
            }
            dl *= fac;
            m = m_new;
            ref = ref_new;
            nref = (ref == ninf) ? 0.0f : -ref;
            if constexpr (DUMP) {
                if (dslot >= 0 && grp == 0 && wave == 0 && vis) p.dump_ref[(long long)dslot * p.dump_nblk + jb] = ref;
            }
        } else {
            // eq. (2): real-valued running maximum (see the prefill kernel)
            const bool vis = amax != ninf;
            const float m_new = vis ? __builtin_fmaxf(m, amax * c) : m;
            float fac = 1.0f;
            if (m != ninf) {
                const float x = m - m_new;
                if constexpr (MODE == kModeDefault) {
                    fac = __builtin_amdgcn_exp2f(x);
                } else {
                    const uint32_t ix = min(max(hif8::f2u(x) >> kTabShift, (uint32_t)kCodeLo), (uint32_t)kCodeHi);
                    fac = hif8::u2f((uint32_t)ctab[ix] << 20) * 0x1p104f;
                }
            }
            if (__any(fac != 1.0f)) {
#pragma unroll
                for (int t = 0; t < kDT; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) oacc[t][i] *= fac;
            }
            dl *= fac;
            m = m_new;
            ref = m_new;
            nref = (m == ninf) ? 0.0f : -m;
            if constexpr (DUMP) {
                if (dslot >= 0 && grp == 0 && wave == 0 && vis) p.dump_ref[(long long)dslot * p.dump_nblk + jb] = ref;
            }
        }

        // P = HiF8(2^HiF8(T)) of the 32 keys as one B operand: slots 0..3 =
        // keys 4*grp + i, slots 4..7 = keys 16 + 4*grp + i
        u32x4 pop;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t2 = e >> 1;
            uint32_t w;
            if constexpr (MODE == kModeDefault) {
                const float p0 = __builtin_amdgcn_exp2f(sacc[t2][2 * (e & 1)] * c + nref);
                const float p1 = __builtin_amdgcn_exp2f(sacc[t2][2 * (e & 1) + 1] * c + nref);
                const bf16x2 pb = {(__bf16)p0, (__bf16)p1};
                pop[e] = __builtin_bit_cast(uint32_t, pb);
                dl += p0 + p1;
                continue;
            }
            const float t0 = MODE == kModeE2E ? __builtin_fmaf(sacc[t2][2 * (e & 1)], c, nref)
                                              : sacc[t2][2 * (e & 1)] * c + nref;
            const float t1 = MODE == kModeE2E ? __builtin_fmaf(sacc[t2][2 * (e & 1) + 1], c, nref)
                                              : sacc[t2][2 * (e & 1) + 1] * c + nref;
            if constexpr (TIE) {
                // a T with bits 18..0 zero reads the ties-to-even table
                const uint32_t u0 = hif8::f2u(t0), u1 = hif8::f2u(t1);
                const uint32_t i0 = min(max(u0 >> kTabShift, (uint32_t)kCodeLo), (uint32_t)kCodeHi);
                const uint32_t i1 = min(max(u1 >> kTabShift, (uint32_t)kCodeLo), (uint32_t)kCodeHi);
                const uint32_t c0 = (u0 & 0x7ffffu) ? ctab[i0] : ctab_e[i0];
                const uint32_t c1 = (u1 & 0x7ffffu) ? ctab[i1] : ctab_e[i1];
                w = (c0 | (c1 << 16)) << 4;
            } else if constexpr (CT) {
                const uint32_t i0 = min(max(hif8::f2u(t0) >> kTabShift, (uint32_t)kCodeLo), (uint32_t)kCodeHi);
                const uint32_t i1 = min(max(hif8::f2u(t1) >> kTabShift, (uint32_t)kCodeLo), (uint32_t)kCodeHi);
                w = ((uint32_t)ctab[i0] | ((uint32_t)ctab[i1] << 16)) << 4;
            } else {
                w = (uint32_t)tab[hif8::f2u(t0) >> kTabShift] | ((uint32_t)tab[hif8::f2u(t1) >> kTabShift] << 16);
            }
            pop[e] = w;
            dl = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, dl, false);
        }
        // X^T += V^T P^T for these 32 keys
        {
            wait_slot(consumed);
            const char* slot = my_ring + (consumed % RW) * C::kSlotBytes;
#pragma unroll
            for (int t = 0; t < kDT; ++t) {
                const char* pa = slot + vrow + 16 * (((16 * t + vd0) >> 3) ^ vx);
                const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, pa));
                const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, pa + 16 * C::kRowBytes));
                const u32x4 a = {__builtin_bit_cast(u32x2, va)[0], __builtin_bit_cast(u32x2, va)[1],
                                 __builtin_bit_cast(u32x2, vb)[0], __builtin_bit_cast(u32x2, vb)[1]};
                oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(pop), oacc[t], 0, 0, 0);
            }
            next_slot();
        }
    }

    // sum the waves' partials (one reference scale) through the ring, then
    // O = X / dX, lse = ln2 (ref + log2 dX); the 4 lanes of a query hold
    // disjoint d rows 16*t + 4*grp + i
    float dw = dl + __shfl_xor(dl, 16, 64);
    dw += __shfl_xor(dw, 32, 64);
    if constexpr (KW > 1) {
        float* mb = reinterpret_cast<float*>(ring);             // [KW-1][kRows][D]
        float* db = mb + (KW - 1) * kRows * D;                  // [KW-1][kRows]
        __syncthreads();                                        // every wave is done with its ring
        if (wave > 0) {
            float* mine = mb + (wave - 1) * kRows * D + c16 * D;
#pragma unroll
            for (int t = 0; t < kDT; ++t) *reinterpret_cast<f32x4*>(mine + 16 * t + 4 * grp) = oacc[t];
            if (grp == 0) db[(wave - 1) * kRows + c16] = dw;
        }
        __syncthreads();
        if (wave > 0) return;
#pragma unroll
        for (int w = 1; w < KW; ++w) {
            const float* theirs = mb + (w - 1) * kRows * D + c16 * D;
#pragma unroll
            for (int t = 0; t < kDT; ++t) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(theirs + 16 * t + 4 * grp);
#pragma unroll
                for (int e = 0; e < 4; ++e) oacc[t][e] += v[e];
            }
            dw += db[(w - 1) * kRows + c16];
        }
    }
    if (!row_ok) return;
    const long long orow_off = (((long long)b * p.Hq + h) * p.Sq + r) * D;
    const bool empty = (ref == ninf);
    const float inv = empty ? 0.0f : 1.0f / dw;
    if (p.out_bf16) {
        uint16_t* orow = reinterpret_cast<uint16_t*>(p.o) + orow_off;
#pragma unroll
        for (int t = 0; t < kDT; ++t) {
            const bf16x2 lo = {(__bf16)(oacc[t][0] * inv), (__bf16)(oacc[t][1] * inv)};
            const bf16x2 hi = {(__bf16)(oacc[t][2] * inv), (__bf16)(oacc[t][3] * inv)};
            *reinterpret_cast<u32x2*>(orow + 16 * t + 4 * grp) =
                u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
        }
    } else {
        float* orow = p.o + orow_off;
#pragma unroll
        for (int t = 0; t < kDT; ++t) {
            f32x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = oacc[t][e] * inv;
            *reinterpret_cast<f32x4*>(orow + 16 * t + 4 * grp) = v;
        }
    }
    if (grp == 0) {
        const float dbias = (CT && MODE != kModeDefault) ? (float)kCodeBiasLog2 : 0.0f;
        if (p.lse) p.lse[((long long)b * p.Hq + h) * p.Sq + r] = empty ? ninf : 0.69314718055994531f * (ref + (log2f(dw) + dbias));
        if (n_visit) {
            if (p.counters) {
                atomicAdd(p.counters + 2 * ((long long)b * p.Hq + h) + 0, (unsigned long long)n_restart);
                atomicAdd(p.counters + 2 * ((long long)b * p.Hq + h) + 1, (unsigned long long)n_visit);
            }
            if (p.tile_counts) {
                const int R = p.restart_rows;
                unsigned long long* tc =
                    p.tile_counts + 2 * (((long long)b * p.Hq + h) * ((p.Sq + R - 1) / R) + r / R);
                atomicAdd(tc + 0, (unsigned long long)n_restart);
                atomicAdd(tc + 1, (unsigned long long)n_visit);
            }
        }
    }
}

template <int D, int BLK, bool CT, int MODE, bool F8, bool TIE, bool DUMP>
hipError_t launch_dec(const AttnParams& p, hipStream_t st)
{
    using C = DCfg<D, BLK>;
    static_assert(C::kLdsBytes >= (C::kWaves - 1) * kRows * (D + 1) * 4, "merge buffer fits the ring");
    static DeviceOnce attr_set;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (!attr_set.is_done(dev)) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&baps_attn_decode_kernel<D, BLK, CT, MODE, F8, TIE, DUMP>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, C::kLdsBytes);
        if (e != hipSuccess) return e;
        attr_set.mark(dev);
    }
    const long long flat = (long long)p.Sq * (p.Hq / p.Hkv);
    const dim3 grid((unsigned)((flat + kRows - 1) / kRows), (unsigned)p.Hkv, (unsigned)p.B);
    hipLaunchKernelGGL((baps_attn_decode_kernel<D, BLK, CT, MODE, F8, TIE, DUMP>), grid, dim3(64 * C::kWaves),
                       C::kLdsBytes, st, p);
    return hipGetLastError();
}

template <int D, int BLK, bool DUMP>
hipError_t launch_dec_ct(const AttnParams& p, hipStream_t st)
{
    if (p.tie_even) return launch_dec<D, BLK, true, kModeE2E, false, true, DUMP>(p, st);
    if (p.qk_f8) {                                 // FP8 Q/K
        if (p.mode == kModeDefault) return launch_dec<D, BLK, true, kModeDefault, true, false, DUMP>(p, st);
        if (p.mode == kModeExp2) return launch_dec<D, BLK, true, kModeExp2, true, false, DUMP>(p, st);
        if (p.lambda <= kCodeMaxLambda) return launch_dec<D, BLK, true, kModeE2E, true, false, DUMP>(p, st);
        return launch_dec<D, BLK, false, kModeE2E, true, false, DUMP>(p, st);
    }
    if (p.mode == kModeDefault) return launch_dec<D, BLK, true, kModeDefault, false, false, DUMP>(p, st);
    if (p.mode == kModeExp2) return launch_dec<D, BLK, true, kModeExp2, false, false, DUMP>(p, st);
    if (p.lambda <= kCodeMaxLambda) return launch_dec<D, BLK, true, kModeE2E, false, false, DUMP>(p, st);
    return launch_dec<D, BLK, false, kModeE2E, false, false, DUMP>(p, st);
}

template <int D, int BLK>
hipError_t launch_dec_any(const AttnParams& p, hipStream_t st)
{
    return p.dump_slot ? launch_dec_ct<D, BLK, true>(p, st) : launch_dec_ct<D, BLK, false>(p, st);
}

}  // namespace

hipError_t launch_attention_decode(const AttnParams& p, int D, int block, hipStream_t st)
{
    if (D == 64 && block == 32) return launch_dec_any<64, 32>(p, st);
    if (D == 64 && block == 64) return launch_dec_any<64, 64>(p, st);
    if (D == 64 && block == 128) return launch_dec_any<64, 128>(p, st);
    if (D == 128 && block == 32) return launch_dec_any<128, 32>(p, st);
    if (D == 128 && block == 64) return launch_dec_any<128, 64>(p, st);
    if (D == 128 && block == 128) return launch_dec_any<128, 128>(p, st);
    return hipErrorInvalidValue;
}

}  // namespace baps
