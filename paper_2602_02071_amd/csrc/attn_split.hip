// Split-key passes of the fused BAPS attention forward, for few query rows
// per key/value head and few (batch, key/value head) streams (single-sequence
// or small-batch decode over long contexts), where one workgroup per stream
// would leave most of the GPU idle.
//
// Alg. 1 visits the key blocks of a row in order, but its state after block j
// (the integer running maximum m and the block reference) depends on the keys
// only through each block's row maximum.  So:
//   1. scores: every key split in parallel streams K and writes the raw dot
//      products acc = q.k (fp32, as the MFMA accumulates them) and the raw
//      row maximum of every block;
//   2. pv: every split in parallel first replays Alg. 1's B0 / restart rule
//      and integer maximum over the block maxima of its rows, from block 0 to
//      its own last block -- the same per-block decision as the one-pass
//      kernels, 16 blocks per step, serial only where m changes -- then
//      streams V, forms P = HiF8(2^HiF8(T)) with T = fl32(acc*c - ref_j), and
//      accumulates X and dX relative to its latest reference;
//   3. combine: per row, the splits' X and dX brought to the largest
//      reference with exact powers of two (references never decrease along a
//      row) and summed: O = sum X / sum dX, and lse.
// Every T, P and reference equals the one-pass kernels'; O differs only by
// the order of the fp32 additions.

#include "common.hpp"

namespace baps {

namespace {

typedef __bf16 bf16x2 __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef short s16x4 __attribute__((ext_vector_type(4)));
#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

constexpr int kRows = 16;            // query rows per workgroup (16x16x32 MFMA columns)
constexpr int kSlotKeys = 32;        // keys per wave and block, and per ring slot

template <int D, int BLK>
struct SCfg {
    static constexpr int kWaves = BLK / kSlotKeys;              // one wave per 32-key slot of a block
    static constexpr int kRowBytes = 2 * D;
    static constexpr int kCPR = D / 8;                          // 16-byte chunks per row
    static constexpr int kSlotBytes = kSlotKeys * kRowBytes;
    static constexpr int kIPS = kSlotBytes / 1024;              // wave-wide loads per slot
    static constexpr int kRW0 = (64 * 1024) / (kWaves * kSlotBytes);
    static constexpr int kRW = kRW0 < 2 ? 2 : (kRW0 * kIPS > 63 ? 63 / kIPS : kRW0);
    static constexpr int kLdsBytes = kWaves * kRW * kSlotBytes;
};

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

// one wave-wide non-temporal global->LDS load of 1 KiB (every byte read once)
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
    asm volatile("" ::: "memory");            // LDS written by the loads is read after this
}

// Rows of the workgroup: flat index f = r * G + h_local of its 16-row tile.
struct RowInfo {
    int f, r, h, kmax;
    bool ok;
};

__device__ __forceinline__ RowInfo row_info(const AttnParams& p, int tile, int g, int c16)
{
    const int G = p.Hq / p.Hkv;
    const int flat = p.Sq * G;
    RowInfo ri;
    ri.f = tile * kRows + c16;
    ri.ok = ri.f < flat;
    ri.r = ri.ok ? ri.f / G : 0;
    ri.h = g * G + (ri.ok ? ri.f % G : 0);
    ri.kmax = ri.ok ? (p.causal ? min(p.Sk - 1, ri.r + (p.Sk - p.Sq)) : p.Sk - 1) : -1;
    return ri;
}

// ---------------------------------------------------------------------------
// 1. scores: acc and block maxima of one key split
// ---------------------------------------------------------------------------
template <int D, int BLK, bool F8>
__global__ __launch_bounds__(64 * (BLK / 32)) void split_scores_kernel(SplitParams sp)
{
    using C = SCfg<D, BLK>;
    constexpr int KW = C::kWaves;
    constexpr int RW = C::kRW;
    constexpr int kDK = D / 32;
    __shared__ float xch[2][KW][kRows];
    extern __shared__ __attribute__((aligned(1024))) char ring[];
    const uint32_t ring_lds = (uint32_t)(uintptr_t)LDS_PTR(char, ring);
    const AttnParams& p = sp.a;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c16 = lane & 15;
    const int grp = lane >> 4;
    const int split = blockIdx.x % sp.nsplit;
    const int tile = blockIdx.x / sp.nsplit;
    const int g = blockIdx.y;
    const int b = blockIdx.z;
    const int flat = p.Sq * (p.Hq / p.Hkv);
    const long long bg = (long long)b * p.Hkv + g;
    const uint16_t* kbase = p.k + bg * (long long)p.Sk * D;
    const uint8_t* kbase8 = reinterpret_cast<const uint8_t*>(p.k) + bg * (long long)p.Sk * D;
    const int j0 = split * sp.bps;
    const int j1 = min(sp.nblk, j0 + sp.bps);
    const int nslots = max(0, j1 - j0);
    constexpr int kIPS = F8 ? kSlotKeys * D / 1024 : C::kIPS;     // loads per slot (FP8 K: rows of D bytes)

    const uint32_t my_ring_lds = ring_lds + (uint32_t)(wave * RW * C::kSlotBytes);
    const char* my_ring = ring + wave * RW * C::kSlotBytes;
    auto issue_slot = [&](int n) {               // K keys [32*wave, +32) of block j0 + n
        const int key0 = (j0 + n) * BLK + wave * kSlotKeys;
        const uint32_t dst = my_ring_lds + (uint32_t)((n % RW) * C::kSlotBytes);
        if constexpr (F8) {
#pragma unroll
            for (int t = 0; t < kIPS; ++t) {
                const int rr = t * (1024 / D) + lane / (D / 16);
                const int ch = (lane % (D / 16)) ^ k8_swz<D>(rr);
                const int key = min(key0 + rr, p.Sk - 1);
                lds_dma_16(kbase8 + (long long)key * D + ch * 16, dst + t * 1024);
            }
            return;
        }
#pragma unroll
        for (int t = 0; t < C::kIPS; ++t) {
            const int rr = t * (1024 / C::kRowBytes) + lane / C::kCPR;
            const int ch = (lane % C::kCPR) ^ k_swz<D>(rr);
            const int key = min(key0 + rr, p.Sk - 1);
            lds_dma_16(kbase + (long long)key * D + ch * 8, dst + t * 1024);
        }
    };
    int issued = 0;
    for (; issued < min(nslots, RW); ++issued) issue_slot(issued);

    const RowInfo ri = row_info(p, tile, g, c16);
    int kmax_lo = ri.ok ? ri.kmax : 0x7fffffff;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) kmax_lo = min(kmax_lo, __shfl_xor(kmax_lo, o, 64));
    kmax_lo = __builtin_amdgcn_readfirstlane(kmax_lo);
    u32x4 qop[F8 ? 1 : kDK];
    i32x8 qop8 = {};                              // FP8: Q[row][32*grp .. +32], zeros past D
    if constexpr (F8) {
        const uint8_t* qrow = reinterpret_cast<const uint8_t*>(p.q) + (((long long)b * p.Hq + ri.h) * p.Sq + ri.r) * D;
        if (ri.ok && 32 * grp < D)
            qop8 = cat8(*reinterpret_cast<const u32x4*>(qrow + 32 * grp),
                        *reinterpret_cast<const u32x4*>(qrow + 32 * grp + 16));
    } else {
        const uint16_t* qrow = p.q + (((long long)b * p.Hq + ri.h) * p.Sq + ri.r) * D;
#pragma unroll
        for (int kk = 0; kk < kDK; ++kk)
            qop[kk] = ri.ok ? *reinterpret_cast<const u32x4*>(qrow + kk * 32 + grp * 8) : u32x4{0, 0, 0, 0};
    }
    const float ninf = -__builtin_huge_valf();
    const int kx = k_swz<D>(c16);
    const uint32_t krow = c16 * C::kRowBytes;
    const long long nkeys = (long long)sp.nblk * BLK;
    float* acc_row = sp.acc + (bg * flat + (ri.ok ? ri.f : 0)) * nkeys;
    float* bmax_row = sp.bmax + (bg * flat + (ri.ok ? ri.f : 0)) * sp.bstride;

    for (int n = 0; n < nslots; ++n) {
        const int jb = j0 + n;
        const int key0 = jb * BLK + wave * kSlotKeys;
        f32x4 sacc[2];
        wait_vm((issued - 1 - n) * kIPS);
        const char* slot = my_ring + (n % RW) * C::kSlotBytes;
        if constexpr (F8) {
            const int kx8 = k8_swz<D>(c16);
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
                f32x4 a4 = {};
#pragma unroll
                for (int kk = 0; kk < kDK; ++kk) {
                    const u32x4 a = *reinterpret_cast<const u32x4*>(
                        slot + krow + t2 * 16 * C::kRowBytes + 16 * ((4 * kk + grp) ^ kx));
                    a4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(qop[kk]), a4, 0, 0, 0);
                }
                sacc[t2] = a4;
            }
        }
        if (issued < nslots) { issue_slot(issued); ++issued; }
        // mask keys past kmax; register i of tile t2 holds key key0 + 16*t2 + 4*grp + i
        if (key0 + kSlotKeys - 1 > kmax_lo) {
            asm volatile("" ::: "memory");
            const int lim = ri.kmax - key0 - 4 * grp;
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (16 * t2 + i > lim) sacc[t2][i] = ninf;
        }
        if (ri.ok) {
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2)
                *reinterpret_cast<f32x4*>(acc_row + key0 + 16 * t2 + 4 * grp) = sacc[t2];
        }
        float pm = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(sacc[0][0], sacc[0][1]), sacc[0][2]),
                                   __builtin_fmaxf(__builtin_fmaxf(sacc[0][3], sacc[1][0]), sacc[1][1]));
        pm = __builtin_fmaxf(pm, __builtin_fmaxf(sacc[1][2], sacc[1][3]));
        pm = __builtin_fmaxf(pm, __shfl_xor(pm, 16, 64));
        pm = __builtin_fmaxf(pm, __shfl_xor(pm, 32, 64));
        if constexpr (KW > 1) {
            if (grp == 0) xch[jb & 1][wave][c16] = pm;
            __syncthreads();
            if (wave == 0) {
                float am = xch[jb & 1][0][c16];
#pragma unroll
                for (int w = 1; w < KW; ++w) am = __builtin_fmaxf(am, xch[jb & 1][w][c16]);
                pm = am;
            }
        }
        if (wave == 0 && grp == 0 && ri.ok) bmax_row[jb] = pm;
    }
}

// ---------------------------------------------------------------------------
// 2. pv: Alg. 1's per-block decisions up to the split, then P V of the split
// ---------------------------------------------------------------------------
constexpr int kWinBlocks = 256;      // block maxima per LDS window of the scan (one row)

template <int D, int BLK>
struct PCfg {
    using C = SCfg<D, BLK>;
    static constexpr int kWaves = C::kWaves;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int kPS = D + 4;                            // floats per part row: X, dX, reference
    static constexpr int kLdsBytes = C::kLdsBytes;               // dynamic: the V ring (64 KiB at most)
};

template <int D, int BLK>
__global__ __launch_bounds__(64 * (BLK / 32)) void split_pv_kernel(SplitParams sp)
{
    using C = SCfg<D, BLK>;
    using PC = PCfg<D, BLK>;
    constexpr int KW = C::kWaves;
    constexpr int RW = C::kRW;
    constexpr int kDT = D / 16;
    constexpr int NT = PC::kThreads;
    constexpr int PS = PC::kPS;
    __shared__ __attribute__((aligned(1024))) uint8_t ctab[kCodeTableBytes];   // entry i at [i - kCodeLo]
    __shared__ unsigned s_cnt[kRows][2];
    __shared__ __attribute__((aligned(1024))) float s_win[KW][2][kWinBlocks];       // scan windows
    __shared__ float refs_l[kRows * kSplitMaxBps];                                   // block references
    extern __shared__ __attribute__((aligned(1024))) char ring[];
    const uint32_t ring_lds = (uint32_t)(uintptr_t)LDS_PTR(char, ring);
    const AttnParams& p = sp.a;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c16 = lane & 15;
    const int grp = lane >> 4;
    const int split = blockIdx.x % sp.nsplit;
    const int tile = blockIdx.x / sp.nsplit;
    const int g = blockIdx.y;
    const int b = blockIdx.z;
    const int flat = p.Sq * (p.Hq / p.Hkv);
    const long long bg = (long long)b * p.Hkv + g;
    const uint16_t* vbase = p.v + bg * (long long)p.Sk * D;
    const int j0 = split * sp.bps;
    const int j1 = min(sp.nblk, j0 + sp.bps);
    const int nslots = max(0, j1 - j0);
    const float ninf = -__builtin_huge_valf();
    const float c = p.c;

    // -- block-maximum windows of the scan: one wave-wide 1 KiB DMA each, the
    //    maxima of blocks [256 w, 256 w + 256) of one row of the tile
    const uint32_t win_lds = (uint32_t)(uintptr_t)LDS_PTR(float, &s_win[wave][0][0]);
    const float* win = &s_win[wave][0][0];
    const int nwin = (j1 + kWinBlocks - 1) / kWinBlocks;
    const int nr = min(kRows, flat - tile * kRows);         // rows of the tile (at least one)
    const int npass = (nr + KW - 1) / KW;                   // the scan takes one row per wave at a time
    int ndma = 0;                                 // DMA ops of this wave issued so far
    int tag0 = 0, tag1 = 0;                       // ndma after the DMA of each window buffer
    int tagc = 0;                                 // ndma after this wave's part of the code table
    {
        const uint32_t ctab_lds = (uint32_t)(uintptr_t)LDS_PTR(uint8_t, ctab);
        for (int i = wave; i < kCodeTableBytes / 1024; i += KW) {
            lds_dma_16(p.ctab + i * 1024 + 16 * lane, ctab_lds + (uint32_t)(i * 1024));
            tagc = ++ndma;
        }
    }
    auto issue_win = [&](int pass, int w) {
        const int srow = min(pass * KW + wave, nr - 1);
        const float* src = sp.bmax + (bg * flat + tile * kRows + srow) * sp.bstride + w * kWinBlocks + 4 * lane;
        lds_dma_16(src, win_lds + (uint32_t)((w & 1) * 1024));
        ++ndma;
        if (w & 1) tag1 = ndma; else tag0 = ndma;
    };
    issue_win(0, 0);
    if (nwin > 1) issue_win(0, 1);

    // -- the V ring of this split
    const uint32_t my_ring_lds = ring_lds + (uint32_t)(wave * RW * C::kSlotBytes);
    const char* my_ring = ring + wave * RW * C::kSlotBytes;
    auto issue_slot = [&](int n) {               // V keys [32*wave, +32) of block j0 + n
        const int key0 = (j0 + n) * BLK + wave * kSlotKeys;
        const uint32_t dst = my_ring_lds + (uint32_t)((n % RW) * C::kSlotBytes);
#pragma unroll
        for (int t = 0; t < C::kIPS; ++t) {
            const int rr = t * (1024 / C::kRowBytes) + lane / C::kCPR;
            const int ch = (lane % C::kCPR) ^ v_swz<D>(rr);
            const int key = min(key0 + rr, p.Sk - 1);
            lds_dma_16(vbase + (long long)key * D + ch * 8, dst + t * 1024);
        }
        ndma += C::kIPS;
    };
    int issued = 0;
    for (; issued < min(nslots, RW); ++issued) issue_slot(issued);

    // -- the scan: Alg. 1's decision for every block of [0, j1) of a row, 64
    //    blocks (one per lane) evaluated per step at the current m; the blocks
    //    up to the first one that changes m are settled, and the step repeats
    //    from there with the new m (wave-uniform: a scalar register)
    const float lam = (float)p.lambda;
    for (int pass = 0; pass < npass; ++pass) {
        const int srow = pass * KW + wave;
        const bool row_ok = srow < nr;
        const int last_blk = row_ok ? row_info(p, tile, g, srow).kmax / BLK : -1;   // B0 with b0_last
        float m = ninf;
        unsigned n_restart = 0, n_visit = 0;
        if (pass > 0) {                           // this pass's first windows (the V ring is already in flight)
            issue_win(pass, 0);
            if (nwin > 1) issue_win(pass, 1);
        }
        for (int w = 0; w < nwin; ++w) {
            wait_vm(ndma - ((w & 1) ? tag1 : tag0));
            const float* wl = win + (w & 1) * kWinBlocks;
#pragma unroll 1
            for (int kk = 0; kk < kWinBlocks / 64; ++kk) {
                const int cb = w * kWinBlocks + 64 * kk;
                if (cb >= j1) break;
                const int jb = cb + lane;
                float amax = wl[64 * kk + lane];
                if (!(row_ok && jb < j1)) amax = ninf;
                const bool vis = amax != ninf;
                const float ceil_ac = ceilf(amax * c);
                const bool in_b0 = jb < p.n_b0 || (p.b0_last && jb == last_blk);
                const bool mine = row_ok && jb >= j0 && jb < j1;
                int lo = 0;
                for (;;) {
                    const bool forced = in_b0 || (m == ninf);
                    const float tq = hif8::round(__builtin_fmaf(amax, c, -m));
                    const bool restart = forced || (ceilf(tq) > lam);
                    const float m_hi = __builtin_fmaxf(m, ceil_ac);
                    const float m_new = vis ? (restart ? m_hi : m + __builtin_fmaxf(0.0f, ceilf(tq))) : m;
                    const float ref_new = vis ? (restart ? m_hi : m) : ninf;
                    const bool pend = lane >= lo;
                    const unsigned long long bal = __ballot(pend && hif8::f2u(m_new) != hif8::f2u(m));
                    const int f = bal ? (int)__builtin_ctzll(bal) : 64;
                    if (pend && lane <= f && mine) {
                        refs_l[srow * kSplitMaxBps + (jb - j0)] = ref_new;   // -inf: no visible key
                        const bool b1 = vis && !in_b0;
                        n_visit += b1 ? 1u : 0u;
                        n_restart += (b1 && restart) ? 1u : 0u;
                    }
                    if (f >= 63) {
                        if (f == 63) m = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                              __builtin_bit_cast(int, m_new), 63));
                        break;
                    }
                    m = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, m_new), f));
                    lo = f + 1;
                }
            }
            if (w + 2 < nwin) issue_win(pass, w + 2);
        }
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            n_visit += __shfl_xor(n_visit, o, 64);
            n_restart += __shfl_xor(n_restart, o, 64);
        }
        if (lane == 0 && row_ok) {
            s_cnt[srow][0] = n_restart;
            s_cnt[srow][1] = n_visit;
        }
    }
    wait_vm(ndma - tagc);                         // this wave's part of the code table has landed

    const RowInfo ri = row_info(p, tile, g, c16);
    const long long nkeys = (long long)sp.nblk * BLK;
    const long long rowoff = bg * flat + (ri.ok ? ri.f : 0);
    const float* acc_row = sp.acc + rowoff * nkeys;
    float cur = ninf, dl = 0.0f;                  // X and dX are relative to the reference cur
    f32x4 oacc[kDT];
#pragma unroll
    for (int t = 0; t < kDT; ++t) oacc[t] = f32x4{};
    const int vrow0 = 4 * grp + c16 / 4;
    const int vx = v_swz<D>(vrow0);
    const int vd0 = 4 * (c16 & 3);
    const uint32_t vrow = vrow0 * C::kRowBytes + 2 * (vd0 & 7);
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    __syncthreads();                              // code table, references and counts published

    // The raw dot products of kAccRun blocks are loaded together at the start
    // of each run of blocks: the first use of a load waits for every older
    // memory operation of the wave, which includes the V ring's loads in
    // flight, so one load per block would let only one slot of the ring fly.
    constexpr int kAccRun = 4;
    for (int n0 = 0; n0 < nslots; n0 += kAccRun) {
    f32x4 accr[kAccRun][2];
#pragma unroll
    for (int u = 0; u < kAccRun; ++u) {
        const int key0 = (j0 + n0 + u) * BLK + wave * kSlotKeys;
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
            accr[u][t2] = (ri.ok && n0 + u < nslots) ? *reinterpret_cast<const f32x4*>(acc_row + key0 + 16 * t2 + 4 * grp)
                                                     : f32x4{ninf, ninf, ninf, ninf};
    }
#pragma unroll
    for (int u = 0; u < kAccRun; ++u) {
        const int n = n0 + u;
        if (n >= nslots) break;
        const int jb = j0 + n;
        const int key0 = jb * BLK + wave * kSlotKeys;
        // this block's reference; the partials follow it with exact rescales
        const float rj = ri.ok ? refs_l[c16 * kSplitMaxBps + n] : ninf;
        const float fac = (cur == ninf || rj == ninf) ? 1.0f : exp2_int(cur - rj);
        if (__any(fac != 1.0f)) {
#pragma unroll
            for (int t = 0; t < kDT; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) oacc[t][i] *= fac;
        }
        dl *= fac;
        if (rj != ninf) cur = rj;
        const float nref = (cur == ninf) ? 0.0f : -cur;
        const f32x4* sacc = accr[u];
        u32x4 pop;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t2 = e >> 1;
            const float t0 = __builtin_fmaf(sacc[t2][2 * (e & 1)], c, nref);
            const float t1 = __builtin_fmaf(sacc[t2][2 * (e & 1) + 1], c, nref);
            const uint32_t i0 = min(max(hif8::f2u(t0) >> kTabShift, (uint32_t)kCodeLo), (uint32_t)kCodeHi);
            const uint32_t i1 = min(max(hif8::f2u(t1) >> kTabShift, (uint32_t)kCodeLo), (uint32_t)kCodeHi);
            const uint32_t w = ((uint32_t)ctab[i0 - kCodeLo] | ((uint32_t)ctab[i1 - kCodeLo] << 16)) << 4;
            pop[e] = w;
            dl = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, dl, false);
        }
        wait_vm((issued - 1 - n) * C::kIPS);
        const char* slot = my_ring + (n % RW) * C::kSlotBytes;
#pragma unroll
        for (int t = 0; t < kDT; ++t) {
            const char* pa = slot + vrow + 16 * (((16 * t + vd0) >> 3) ^ vx);
            const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, pa));
            const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, pa + 16 * C::kRowBytes));
            const u32x4 a = {__builtin_bit_cast(u32x2, va)[0], __builtin_bit_cast(u32x2, va)[1],
                             __builtin_bit_cast(u32x2, vb)[0], __builtin_bit_cast(u32x2, vb)[1]};
            oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(pop), oacc[t], 0, 0, 0);
        }
        if (issued < nslots) { issue_slot(issued); ++issued; }
    }
    }

    // -- one sum over the waves (they share the references), then this
    //    split's part: X, dX and the reference cur they are relative to
    float dw = dl + __shfl_xor(dl, 16, 64);
    dw += __shfl_xor(dw, 32, 64);
    if constexpr (KW > 1) {
        float* mb = reinterpret_cast<float*>(ring);             // [KW-1][kRows][D]
        float* db = mb + (KW - 1) * kRows * D;                  // [KW-1][kRows]
        __syncthreads();
        if (wave > 0) {
            float* mine = mb + (wave - 1) * kRows * D + c16 * D;
#pragma unroll
            for (int t = 0; t < kDT; ++t) *reinterpret_cast<f32x4*>(mine + 16 * t + 4 * grp) = oacc[t];
            if (grp == 0) db[(wave - 1) * kRows + c16] = dw;
        }
        __syncthreads();
        if (wave == 0) {
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
    }
    const long long rows_all = (long long)p.B * p.Hkv * flat;
    if (wave == 0 && ri.ok) {
        float* prow = sp.part + ((long long)split * rows_all + rowoff) * PS;
#pragma unroll
        for (int t = 0; t < kDT; ++t) *reinterpret_cast<f32x4*>(prow + 16 * t + 4 * grp) = oacc[t];
        if (grp == 0) {
            prow[D] = dw;
            prow[D + 1] = cur;
        }
    }
    // restart counters of this split's blocks (a tile is one row here)
    if (tid < kRows) {
        const RowInfo cr = row_info(p, tile, g, tid);
        if (cr.ok && s_cnt[tid][1]) {
            if (p.counters) {
                unsigned long long* cp = p.counters + 2 * ((long long)b * p.Hq + cr.h);
                atomicAdd(cp + 0, (unsigned long long)s_cnt[tid][0]);
                atomicAdd(cp + 1, (unsigned long long)s_cnt[tid][1]);
            }
            if (p.tile_counts) {
                unsigned long long* tc = p.tile_counts + 2 * (((long long)b * p.Hq + cr.h) * p.Sq + cr.r);
                atomicAdd(tc + 0, (unsigned long long)s_cnt[tid][0]);
                atomicAdd(tc + 1, (unsigned long long)s_cnt[tid][1]);
            }
        }
    }
}


// ---------------------------------------------------------------------------
// 3. combine: one workgroup per row; groups of threads take every SG-th split
//    of 4 values of d each, and their sums meet in LDS
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void split_combine_kernel(SplitParams sp)
{
    constexpr int QD = D / 4;                     // threads per split group (4 values of d each)
    constexpr int SG = 256 / QD;                  // split groups
    constexpr int PS = D + 4;
    constexpr int kU = 8;                         // splits in flight per thread
    __shared__ float red[256][6];
    const AttnParams& p = sp.a;
    const int tid = threadIdx.x;
    const int q4 = tid % QD;
    const int sg = tid / QD;
    const int f = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int G = p.Hq / p.Hkv;
    const int flat = p.Sq * G;
    const long long row = ((long long)b * p.Hkv + g) * flat + f;
    const long long pstride = (long long)p.B * p.Hkv * flat * PS;
    const float* pcol = sp.part + row * PS;
    const float ninf = -__builtin_huge_valf();
    float rr = ninf, dx = 0.0f;
    f32x4 xs = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int s0 = sg; s0 < sp.nsplit; s0 += kU * SG) {
        float rv[kU], dv[kU];
        f32x4 xv[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {           // straight-line loads (a clamped split, masked below)
            const float* prow = pcol + min(s0 + u * SG, sp.nsplit - 1) * pstride;
            xv[u] = *reinterpret_cast<const f32x4*>(prow + 4 * q4);
            dv[u] = prow[D];
            rv[u] = prow[D + 1];
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
            if (s0 + u * SG >= sp.nsplit) rv[u] = ninf;
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            if (rv[u] == ninf) continue;          // no visible key in that split
            if (rv[u] > rr) {
                const float fa = exp2_int(rr - rv[u]);   // 0 while rr is -inf (nothing summed yet)
#pragma unroll
                for (int e = 0; e < 4; ++e) xs[e] *= fa;
                dx *= fa;
                rr = rv[u];
            }
            const float fb = exp2_int(rv[u] - rr);
#pragma unroll
            for (int e = 0; e < 4; ++e) xs[e] += fb * xv[u][e];
            dx += fb * dv[u];
        }
    }
    red[tid][0] = rr;
    red[tid][1] = dx;
    red[tid][2] = xs[0];
    red[tid][3] = xs[1];
    red[tid][4] = xs[2];
    red[tid][5] = xs[3];
    __syncthreads();
    if (sg != 0) return;
    for (int o = 1; o < SG; ++o) {
        const float* th = red[tid + o * QD];
        const float r2 = th[0];
        if (r2 == ninf) continue;
        const float top = __builtin_fmaxf(rr, r2);
        const float fa = (rr == ninf) ? 0.0f : exp2_int(rr - top);
        const float fb = exp2_int(r2 - top);
        dx = dx * fa + th[1] * fb;
#pragma unroll
        for (int e = 0; e < 4; ++e) xs[e] = xs[e] * fa + th[2 + e] * fb;
        rr = top;
    }
    const int r = f / G;
    const int h = g * G + f % G;
    const bool empty = rr == ninf;
    const float inv = empty ? 0.0f : 1.0f / dx;
    const long long orow_off = (((long long)b * p.Hq + h) * p.Sq + r) * D + 4 * q4;
    if (p.out_bf16) {
        typedef __bf16 bf16x2 __attribute__((__vector_size__(2 * sizeof(__bf16))));
        const bf16x2 lo = {(__bf16)(xs[0] * inv), (__bf16)(xs[1] * inv)};
        const bf16x2 hi = {(__bf16)(xs[2] * inv), (__bf16)(xs[3] * inv)};
        *reinterpret_cast<u32x2*>(reinterpret_cast<uint16_t*>(p.o) + orow_off) =
            u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
    } else {
        *reinterpret_cast<f32x4*>(p.o + orow_off) = f32x4{xs[0] * inv, xs[1] * inv, xs[2] * inv, xs[3] * inv};
    }
    if (q4 == 0 && p.lse)
        p.lse[((long long)b * p.Hq + h) * p.Sq + r] =
            empty ? ninf : 0.69314718055994531f * (rr + (log2f(dx) + (float)kCodeBiasLog2));
}

template <int D, int BLK>
hipError_t launch_split_db(const SplitParams& sp, hipStream_t st)
{
    using C = SCfg<D, BLK>;
    using PC = PCfg<D, BLK>;
    static_assert(C::kLdsBytes >= (C::kWaves - 1) * kRows * (D + 1) * 4, "merge buffer fits the ring");
    static DeviceOnce attr_set;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (!attr_set.is_done(dev)) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&split_scores_kernel<D, BLK, false>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, C::kLdsBytes);
        if (e == hipSuccess)
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(&split_scores_kernel<D, BLK, true>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, C::kLdsBytes);
        if (e == hipSuccess)
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(&split_pv_kernel<D, BLK>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, PC::kLdsBytes);
        if (e != hipSuccess) return e;
        attr_set.mark(dev);
    }
    const AttnParams& p = sp.a;
    if (sp.bps < 1 || sp.bps > kSplitMaxBps || sp.bstride % kWinBlocks || sp.bstride < sp.nblk ||
        (long long)sp.nsplit * sp.bps < sp.nblk || (long long)(sp.nsplit - 1) * sp.bps >= sp.nblk)
        return hipErrorInvalidValue;
    const long long flat = (long long)p.Sq * (p.Hq / p.Hkv);
    const unsigned tiles = (unsigned)((flat + kRows - 1) / kRows);
    const dim3 grid(tiles * (unsigned)sp.nsplit, (unsigned)p.Hkv, (unsigned)p.B);
    if (p.qk_f8)
        hipLaunchKernelGGL((split_scores_kernel<D, BLK, true>), grid, dim3(64 * C::kWaves), C::kLdsBytes, st, sp);
    else
        hipLaunchKernelGGL((split_scores_kernel<D, BLK, false>), grid, dim3(64 * C::kWaves), C::kLdsBytes, st, sp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((split_pv_kernel<D, BLK>), grid, dim3(PC::kThreads), PC::kLdsBytes, st, sp);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((split_combine_kernel<D>), dim3((unsigned)flat, (unsigned)p.Hkv, (unsigned)p.B), dim3(256), 0,
                       st, sp);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_split(const SplitParams& sp, int D, int block, hipStream_t st)
{
    if (D == 64 && block == 32) return launch_split_db<64, 32>(sp, st);
    if (D == 64 && block == 64) return launch_split_db<64, 64>(sp, st);
    if (D == 64 && block == 128) return launch_split_db<64, 128>(sp, st);
    if (D == 128 && block == 32) return launch_split_db<128, 32>(sp, st);
    if (D == 128 && block == 64) return launch_split_db<128, 64>(sp, st);
    if (D == 128 && block == 128) return launch_split_db<128, 128>(sp, st);
    return hipErrorInvalidValue;
}

}  // namespace baps
