// Fused BAPS attention forward (Alg. 1, the "E2E HiF8" workflow) for gfx950.
//
// Work split: a work item is 32*NW query rows of one key/value head.  The
// rows are the flattened (query position, query head of the group) pairs, so
// the Hq/Hkv query heads that share K/V share the item, and single-position
// decode packs its heads into one tile.  Each wave owns 32 rows.  At D = 128
// the grid is persistent: one workgroup per CU takes a sequence of items
// (item_at); the first K/V block of the next item loads during the last
// block of the current one, and its Q right after that block's Q^T reads;
// at D = 64 a workgroup takes one item and two of them share a CU.
//
// Per key block j (the paper's key tile, visited in ascending order):
//   - K_j and V_j arrive in LDS through asynchronous global->LDS loads into a
//     double buffer: the loads of block j+1 are in flight while block j is
//     computed.  Both tiles keep their natural [key][d] layout with the
//     16-byte chunks of each row XOR-swizzled, so that the ds_read_b128 K
//     operand reads are free of bank conflicts (and the transposing V reads
//     nearly so);
//   - S^T = K_j Q^T on v_mfma_f32_32x32x16_bf16 with fp32 accumulation (Q
//     stays in registers).  In the S^T layout a lane holds 16 keys of one
//     query per 32-key tile, so a row maximum is an in-lane max plus one
//     exchange with lane^32;
//   - block-aware precision rescaling per query row: the restart rule of
//     Alg. 1 with threshold lambda, the integer running maximum of Sec. 3.3
//     and exact power-of-two rescale factors;
//   - T = fl32(acc * c - ref): the scale and the subtraction of eq. (3) are
//     one fused multiply-add, rounded once; P = HiF8(2^HiF8(T)) is read from
//     a 8192-entry LDS table indexed by bits 31..19 of T (HiF8 rounding to
//     nearest-away depends on those bits only) and is exact in bf16;
//   - the S^T accumulator layout is already the B operand layout of
//     O^T += V_j^T P^T once the keys inside each 16-key group are taken in a
//     fixed permuted order; the A operand (V^T fragments) comes straight from
//     the [key][d] tile through ds_read_b64_tr_b16 transposing reads, in the
//     same key order.  P never leaves registers.  The table reads of the
//     whole block are issued ahead of the PV loop; the packing of 32-key tile
//     t+1 runs on the VALU while the PV MFMAs of tile t execute.
#include "common.hpp"

namespace baps {

namespace {

constexpr int kRowsPerWave = 32;

typedef __bf16 bf16x2 __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef short s16x4 __attribute__((ext_vector_type(4)));
#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// 16-byte chunk swizzles.  K: rows read 16 at a time at one logical chunk
// (ds_read_b128).  V: rows read 4 at a time, two logical chunks (transposing
// reads of 16 lanes).
template <int D>
__device__ __forceinline__ int k_swz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
template <int D>
__device__ __forceinline__ int v_swz(int r) { return D == 128 ? 2 * (r & 3) : 2 * ((r >> 1) & 1); }
// FP8 K rows (D bytes): 16 rows read at one logical chunk hit distinct banks,
// and the swizzle of row 32*kt + j32 depends on j32 only
template <int D>
__device__ __forceinline__ int k8_swz(int r) { return D == 128 ? ((r ^ ((r >> 3) & 1)) & 7) : ((r >> 2) & 3); }

typedef int i32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ i32x8 cat8(u32x4 a, u32x4 b)
{
    return i32x8{(int)a[0], (int)a[1], (int)a[2], (int)a[3], (int)b[0], (int)b[1], (int)b[2], (int)b[3]};
}

template <int D, int BLK, int NW>
struct Cfg {
    static constexpr int kThreads = 64 * NW;
    static constexpr int kTileRows = kRowsPerWave * NW;
    static constexpr int kRowBytes = 2 * D;
    static constexpr int kCPR = D / 8;                       // 16-byte chunks per row
    static constexpr int kTileBytes = BLK * kRowBytes;       // one K or V block
    static constexpr int kLoadsPerTile = kTileBytes / 1024;  // 1 KiB per wave-wide load
    static constexpr int kRowsPerLoad = 1024 / kRowBytes;
    // dynamic LDS: [K0][V0][K1][V1]; the score table is a static LDS array
    static constexpr int kLdsBytes = 4 * kTileBytes;
};

// maximum of n values as a tree of 3-input maxima (short dependency chain)
template <int N>
__device__ __forceinline__ float tree_max(float* v)
{
    int n = N;
#pragma unroll
    for (int lvl = 0; lvl < 6; ++lvl) {
        if (n == 1) break;
        const int m = (n + 2) / 3;
#pragma unroll
        for (int i = 0; i < m; ++i) {
            const int a = 3 * i, b = 3 * i + 1, c = 3 * i + 2;
            v[i] = c < n ? __builtin_fmaxf(__builtin_fmaxf(v[a], v[b]), v[c]) : (b < n ? __builtin_fmaxf(v[a], v[b]) : v[a]);
        }
        n = m;
    }
    return v[0];
}

// value of lane l^32 (v_permlane32_swap: no LDS round trip)
__device__ __forceinline__ float swap_halves(float x)
{
    const uint32_t u = __builtin_bit_cast(uint32_t, x);
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    // element 0: lanes 0..31 keep their value, lanes 32..63 receive lanes 0..31;
    // element 1: lanes 0..31 receive lanes 32..63, lanes 32..63 keep theirs
    const uint32_t r0 = r[0], r1 = r[1];
    return __builtin_bit_cast(float, (threadIdx.x & 32) ? r0 : r1);
}

// One wave-wide asynchronous global->LDS load: lane l's 16 bytes at gptr land
// at LDS byte lds_base + 16*l.  Issued as inline assembly so that the compiler
// does not guard every later LDS read with a wait on these loads; the kernel
// waits for them explicitly (vmcnt) before the barrier that publishes a tile.
__device__ __forceinline__ void lds_dma_16(const void* gptr, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gptr), "s"(lds_base)
                 : "memory", "m0");
}

// Issue the asynchronous loads of K (or V) rows [key0, key0 + BLK) into an
// LDS tile; rows past the end re-read the last row (finite values that the
// key mask removes).  Wave w issues loads w, w+NW, ...
template <int D, int BLK, int NW, bool IS_V>
__device__ __forceinline__ void load_tile(const uint16_t* base, int key0, int Sk, uint32_t lds_tile, int wave, int lane)
{
    using C = Cfg<D, BLK, NW>;
#pragma unroll
    for (int t = wave; t < C::kLoadsPerTile; t += NW) {
        const int r = t * C::kRowsPerLoad + lane / C::kCPR;
        const int p = lane % C::kCPR;
        const int c = p ^ (IS_V ? v_swz<D>(r) : k_swz<D>(r));
        const int key = min(key0 + r, Sk - 1);
        const uint16_t* src = base + (long long)key * D + c * 8;
        lds_dma_16(src, __builtin_amdgcn_readfirstlane(lds_tile + t * 1024));
    }
}

// The wave's loads of a block that lies entirely before Sk (no clamp) with
// the scalar-base form: lane offsets from the block's first row are fixed
// per wave (precomputed once), the block's base address is wave-uniform, so
// a load costs no vector instruction.
__device__ __forceinline__ void lds_dma_16_sb(uint32_t voff, uint64_t sbase, uint32_t lds_base)
{
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(sbase), "s"(lds_base)
                 : "memory", "m0");
}

__device__ __forceinline__ uint64_t uniform_addr(const void* p)
{
    const uint64_t a = (uint64_t)(uintptr_t)p;
    return ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
           (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
}

// per-load lane offsets (bytes from the block's first row) of this wave's
// loads t = wave, wave + NW, ...; rows of RB bytes, CPR chunks of 16 bytes
template <int NJ, int NW, int LOADS, int RB, int SWZ_KIND, int D>
__device__ __forceinline__ void tile_offsets(uint32_t (&ofs)[NJ], int wave, int lane)
{
    constexpr int CPR = RB / 16;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int t = wave + j * NW;
        const int r = t * (1024 / RB) + lane / CPR;
        const int sw = SWZ_KIND == 0 ? k_swz<D>(r) : (SWZ_KIND == 1 ? v_swz<D>(r) : k8_swz<D>(r));
        ofs[j] = (uint32_t)(r * RB + 16 * ((lane % CPR) ^ sw));
    }
}

template <int NJ, int NW, int LOADS>
__device__ __forceinline__ void load_tile_sb(const void* block_base, const uint32_t (&ofs)[NJ], uint32_t lds_tile, int wave)
{
    const uint64_t sb = uniform_addr(block_base);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int t = wave + j * NW;
        if (t < LOADS) lds_dma_16_sb(ofs[j], sb, __builtin_amdgcn_readfirstlane(lds_tile + t * 1024));
    }
}

// The same for K in FP8 (rows of D bytes, half a bf16 tile).
template <int D, int BLK, int NW>
__device__ __forceinline__ void load_tile_k8(const uint8_t* base, int key0, int Sk, uint32_t lds_tile, int wave, int lane)
{
    constexpr int kCPR8 = D / 16;
    constexpr int kLoads = BLK * D / 1024;
#pragma unroll
    for (int t = wave; t < kLoads; t += NW) {
        const int r = t * (1024 / D) + lane / kCPR8;
        const int c = (lane % kCPR8) ^ k8_swz<D>(r);
        const int key = min(key0 + r, Sk - 1);
        lds_dma_16(base + (long long)key * D + c * 16, __builtin_amdgcn_readfirstlane(lds_tile + t * 1024));
    }
}

// Work items are (query tile, key/value head, batch) triples with a linear
// id L.  When the (batch, key/value head) count is a multiple of 8, L % 8 is
// the head class: workgroups are dealt to the 8 XCDs round-robin by id, each
// XCD with its own L2, and the schedule below keeps every item of a class on
// the workgroups of one XCD, so that a head's K/V is fetched into one L2
// only.  Otherwise L runs over the tiles of all heads.  Either way the
// longest causal tiles come first.
__device__ __forceinline__ void decode_item(int L, int ntiles, int heads, int Hkv, int& tile, int& g, int& b)
{
    int t_rev, hk;
    if (heads % 8 == 0) {
        const int hpx = heads / 8;                      // heads per class
        const int k = L >> 3;
        hk = (L & 7) + 8 * (k % hpx);
        t_rev = k / hpx;
    } else {
        t_rev = L / heads;
        hk = L % heads;
    }
    tile = ntiles - 1 - t_rev;
    g = hk % Hkv;
    b = hk / Hkv;
}

// The persistent schedule: nwg resident workgroups share nitems items.  With
// nwg a multiple of 8, workgroup w serves class w % 8 alone: in round r it
// takes item r*nwg/8 + k of the class (k = w / 8) on even rounds and
// r*nwg/8 + nwg/8 - 1 - k on odd rounds.  Items come longest first, so the
// back-and-forth order pairs long tiles with short ones (a causal workload
// with two items per workgroup gets the same number of key blocks on every
// workgroup).  Returns -1 past the last item.
__device__ __forceinline__ int item_at(int r, int w, int nwg, int nitems)
{
    if (nwg >= nitems) return r == 0 ? w : -1;
    int L;
    if (nwg % 8 == 0) {
        const int g8 = nwg >> 3, k = w >> 3;
        L = 8 * (r * g8 + ((r & 1) ? g8 - 1 - k : k)) + (w & 7);
    } else {
        L = r * nwg + ((r & 1) ? nwg - 1 - w : w);
    }
    return L < nitems ? L : -1;
}

// A value the compiler must take as new at this point (keeps computations
// derived from it where they are written)
__device__ __forceinline__ void opaque_v(int& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void opaque_s(int& x) { asm volatile("" : "+s"(x)); }

typedef __attribute__((address_space(4))) const AttnParams* kargs_ptr;

// The kernel's arguments through a pointer the compiler cannot see through:
// loads from it stay where they are written (once per work item) instead of
// holding those fields in scalar registers across the key-block loop.
__device__ __forceinline__ kargs_ptr fresh_args()
{
    kargs_ptr a = (kargs_ptr)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(a));
    return a;
}

// An item's tile, key/value head, batch and key blocks (its last row sees
// the most keys).
struct ItemGeo {
    int tile, g, b, nblk;
};

template <int BLK, int TILE_ROWS>
__device__ __forceinline__ ItemGeo item_geo(int L, int Hq, int Hkv, int B, int Sq, int Sk, int causal)
{
    const int G = Hq / Hkv;
    const int flat_rows = Sq * G;
    const int ntiles = (flat_rows + TILE_ROWS - 1) / TILE_ROWS;
    ItemGeo e;
    decode_item(L, ntiles, B * Hkv, Hkv, e.tile, e.g, e.b);
    const int f_last = min(flat_rows - 1, e.tile * TILE_ROWS + TILE_ROWS - 1);
    const int kmax_tile = causal ? min(Sk - 1, f_last / G + Sk - Sq) : Sk - 1;
    e.nblk = kmax_tile < 0 ? 0 : kmax_tile / BLK + 1;
    return e;
}

// The item a workgroup takes in round r, with its geometry; false past the last
template <int BLK, int TILE_ROWS>
__device__ __forceinline__ bool item_of_round(kargs_ptr a, int r, ItemGeo& e)
{
    const int ntiles = (a->Sq * (a->Hq / a->Hkv) + TILE_ROWS - 1) / TILE_ROWS;
    const int L = item_at(r, blockIdx.x, gridDim.x, ntiles * a->B * a->Hkv);
    if (L < 0) return false;
    e = item_geo<BLK, TILE_ROWS>(L, a->Hq, a->Hkv, a->B, a->Sq, a->Sk, a->causal);
    return true;
}

// PERSIST: the grid holds at most as many workgroups as the GPU runs at once
// and each takes a sequence of items (item_at); otherwise one item per
// workgroup.  TIE: the 8-bit cast of T rounds ties to even (a second code
// table covers the T whose bits 18..0 are zero, the only ones that can sit
// exactly halfway).  DUMP: also write the raw dot products and the block
// references of the rows the caller marks (AttnParams::dump_slot).
template <int D, int BLK, int NW, bool CT, int MODE, bool TILE, bool F8, bool PERSIST, bool TIE, bool DUMP>
__global__ __launch_bounds__(64 * NW) void baps_attn_fwd_kernel(AttnParams p)
{
    static_assert(MODE == kModeE2E || CT, "the eq. (2) setups use the compact table (T <= 0)");
    static_assert(MODE == kModeE2E || !TILE, "tile-level restart belongs to Alg. 1");
    static_assert(!TIE || (MODE == kModeE2E && CT && !TILE && !F8), "ties to even: canonical per-row path");
    static_assert(D == 64 || D == 128, "head dimension");
    static_assert(BLK % 32 == 0 && BLK <= 128, "key block");
    using C = Cfg<D, BLK, NW>;
    // P lookup: with the code table (lambda <= kCodeMaxLambda) the table
    // expanded to all 8192 indices (no lookup needs a clamp); else the bf16
    // half of the full score table
    __shared__ __attribute__((aligned(1024))) uint8_t ctab[CT ? (TIE ? 2 : 1) * kTabEntries : 1];
    // restart test of Alg. 1 against the threshold T >= dec_x0 and the
    // branch-free increment (CT kernels with ties away: lambda <= 8); the
    // others round T in registers
    constexpr bool kDec = CT && MODE == kModeE2E && !TIE;
    __shared__ __attribute__((aligned(16))) uint16_t tab[CT ? 1 : kTabEntries];
    __shared__ uint32_t tflag[TILE ? NW : 1][3];  // per wave: rows that restart, see the block, are in B0
    extern __shared__ __attribute__((aligned(1024))) char tiles[];
    const uint32_t tiles_lds = (uint32_t)(uintptr_t)LDS_PTR(char, tiles);

    constexpr int kKT = BLK / 32;                 // 32-key tiles per block
    constexpr int kDK = D / 16;                   // 16-wide d chunks (QK^T contraction)
    constexpr int kDT = D / 32;                   // 32-wide d tiles of O^T
    constexpr int kDK8 = D / 64;                  // 64-wide d chunks (FP8 QK^T)

    static_assert((NW & (NW - 1)) == 0, "waves per workgroup");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // (the mask states the bound wave < NW, which folds the per-wave load
    // counts of the K/V tiles to constants)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (NW - 1);
    const int j32 = lane & 31;
    const int half = lane >> 5;

    const int G = p.Hq / p.Hkv;
    const int flat_rows = p.Sq * G;
    const int off = p.Sk - p.Sq;                            // bottom-right causal alignment

    // Tile-level restart (the paper's granularity, Sec. 3.2): the rows of one
    // head at restart_rows consecutive query positions share each block's
    // decision.  With G and R powers of two and R*G <= 256 a tile is the
    // rows j32 == h_local (mod G) of an aligned span of R*G flattened rows:
    // inside one wave when R*G <= 32 (a ballot decides), else across
    // R*G/32 consecutive waves (per-wave masks meet in LDS).
    // tmask: this lane's tile within the wave's 32 rows (all rows of its
    // head when the tile spans waves tw0 .. tw0 + twn - 1)
    uint32_t tmask = 0;
    int tw0 = 0, twn = 1;
    bool xwave = false, trep = false;             // trep: this lane counts its tile's blocks
    if constexpr (TILE) {
        const int RG = p.restart_rows * G;
        uint32_t pat = 0;
        for (int j = 0; j < 32; j += G) pat |= 1u << j;
        tmask = pat << (j32 % G);
        xwave = RG > 32;
        if (!xwave) {
            tmask &= (RG == 32 ? 0xffffffffu : ((1u << RG) - 1u) << (RG * (j32 / RG)));
            trep = half == 0 && j32 == __builtin_ctz(tmask);
        } else {
            twn = RG / 32;
            tw0 = wave - wave % twn;
            trep = half == 0 && wave == tw0 && j32 < G;
        }
    }

    // per-lane LDS byte offsets of the operand reads inside a tile
    uint32_t koff[F8 ? 2 * kDK8 : kDK];
    if constexpr (F8) {
        const int kx = k8_swz<D>(j32);           // FP8 rows of D bytes; two chunks per MFMA
#pragma unroll
        for (int kk = 0; kk < kDK8; ++kk)
#pragma unroll
            for (int e = 0; e < 2; ++e) koff[2 * kk + e] = j32 * D + 16 * ((4 * kk + 2 * half + e) ^ kx);
    } else {
        const int kx = k_swz<D>(j32);            // swizzle of row kt*32 + j32 depends on j32 only
#pragma unroll
        for (int kk = 0; kk < kDK; ++kk) koff[kk] = j32 * C::kRowBytes + 16 * ((2 * kk + half) ^ kx);
    }
    // lane offsets of the scalar-base K / V loads (blocks inside Sk)
    constexpr int kLoadsK = F8 ? BLK * D / 1024 : C::kLoadsPerTile;
    constexpr int kNJK = (kLoadsK + NW - 1) / NW;
    constexpr int kNJV = (C::kLoadsPerTile + NW - 1) / NW;
    uint32_t kdofs[kNJK], vdofs[kNJV];
    tile_offsets<kNJK, NW, kLoadsK, F8 ? D : C::kRowBytes, F8 ? 2 : 0, D>(kdofs, wave, lane);
    tile_offsets<kNJV, NW, C::kLoadsPerTile, C::kRowBytes, 1, D>(vdofs, wave, lane);

    uint32_t voff[kDT];
    {
        // transposing reads: lane l of a 16-lane group points at row
        // 16*pc + 4*half + (l%16)/4 (+8 for slots 4..7) and at 4 values of d
        const int s16 = lane & 15;
        const int row0 = 4 * half + s16 / 4;
        const int vx = v_swz<D>(row0);          // invariant under +16*pc and +8
#pragma unroll
        for (int t = 0; t < kDT; ++t) {
            const int d = 32 * t + 16 * ((lane >> 4) & 1) + 4 * (s16 & 3);
            voff[t] = row0 * C::kRowBytes + 16 * ((d >> 3) ^ vx) + 2 * (d & 7);
        }
    }

    // key/value head offset (elements; bytes for FP8 K) of an item
    auto kv_off = [&](const ItemGeo& e) { return ((long long)e.b * p.Hkv + e.g) * (long long)p.Sk * D; };
    // Asynchronous loads of key block jb of the key/value head at hoff into K/V buffer sel
    auto issue_block = [&](long long hoff, int jb, int sel) {
        const uint8_t* kb8 = reinterpret_cast<const uint8_t*>(p.k) + hoff;
        const uint16_t* kb = p.k + hoff;
        const uint16_t* vb = p.v + hoff;
        const uint32_t nk = tiles_lds + sel * 2 * C::kTileBytes;
        const int k1 = jb * BLK;
        if (k1 + BLK <= p.Sk) {                             // the whole block lies before Sk
            if constexpr (F8) load_tile_sb<kNJK, NW, kLoadsK>(kb8 + (long long)k1 * D, kdofs, nk, wave);
            else load_tile_sb<kNJK, NW, kLoadsK>(kb + (long long)k1 * D, kdofs, nk, wave);
            load_tile_sb<kNJV, NW, C::kLoadsPerTile>(vb + (long long)k1 * D, vdofs, nk + C::kTileBytes, wave);
        } else {
            if constexpr (F8) load_tile_k8<D, BLK, NW>(kb8, k1, p.Sk, nk, wave, lane);
            else load_tile<D, BLK, NW, false>(kb, k1, p.Sk, nk, wave, lane);
            load_tile<D, BLK, NW, true>(vb, k1, p.Sk, nk + C::kTileBytes, wave, lane);
        }
    };

    // Q^T as the B operand of S^T = K Q^T: lane holds Q[row][16*kk + 8*half .. +8]
    // (FP8: 32 bytes Q[row][64*kk + 32*half .. +32] per 32x32x64 MFMA)
    u32x4 qop[F8 ? 1 : kDK];
    i32x8 qop8[F8 ? kDK8 : 1];
    auto load_q = [&](kargs_ptr a, const ItemGeo& e) {
        int ln = lane, Gi = G;
        opaque_v(ln);
        opaque_s(Gi);
        const int hf = ln >> 5;
        const int f = e.tile * C::kTileRows + wave * kRowsPerWave + (ln & 31);
        const bool ok = f < flat_rows;
        const int r = ok ? f / Gi : 0;
        const int h = e.g * Gi + (ok ? f % Gi : 0);
        if constexpr (F8) {
            const uint8_t* qrow = reinterpret_cast<const uint8_t*>(a->q) + (((long long)e.b * a->Hq + h) * a->Sq + r) * D;
#pragma unroll
            for (int kk = 0; kk < kDK8; ++kk) {
                const u32x4 lo = ok ? *reinterpret_cast<const u32x4*>(qrow + 64 * kk + 32 * hf) : u32x4{0, 0, 0, 0};
                const u32x4 hi = ok ? *reinterpret_cast<const u32x4*>(qrow + 64 * kk + 32 * hf + 16) : u32x4{0, 0, 0, 0};
                qop8[kk] = cat8(lo, hi);
            }
        } else {
            const uint16_t* qrow = a->q + (((long long)e.b * a->Hq + h) * a->Sq + r) * D;
#pragma unroll
            for (int kk = 0; kk < kDK; ++kk)
                qop[kk] = ok ? *reinterpret_cast<const u32x4*>(qrow + kk * 16 + hf * 8) : u32x4{0, 0, 0, 0};
        }
    };

    ItemGeo cur;
    if (!item_of_round<BLK, C::kTileRows>(fresh_args(), 0, cur)) return;   // (the grid holds at most one workgroup per item)
    if (cur.nblk > 0) issue_block(kv_off(cur), 0, 0);
    if constexpr (MODE != kModeDefault) {                  // (Default evaluates exp2 in fp32: no table)
        if constexpr (CT) {
            // asynchronous copy (the LDS address handed to the loads is the
            // table's: the compiler sees it written)
            const uint32_t ct_lds = (uint32_t)(uintptr_t)LDS_PTR(uint8_t, ctab);
            for (int i = wave; i < kTabEntries / 1024; i += NW)
                lds_dma_16(p.ctabx + i * 1024 + 16 * lane, __builtin_amdgcn_readfirstlane(ct_lds + i * 1024));
            if constexpr (TIE) {
                for (int i = wave; i < kTabEntries / 1024; i += NW)
                    lds_dma_16(p.ctabx_even + i * 1024 + 16 * lane,
                               __builtin_amdgcn_readfirstlane(ct_lds + kTabEntries + i * 1024));
            }
        } else {
            for (int i = tid; i < kTabEntries; i += C::kThreads) tab[i] = (uint16_t)(p.tab[i] >> 16);
        }
    }
    load_q(fresh_args(), cur);

    const float ninf = -__builtin_huge_valf();
    const float c = p.c;
    const float lam = (float)p.lambda;
    const bool count_blocks = p.counters || p.tile_counts;   // restart / visit counts requested
    int sel = 0;                        // K/V buffer of the current key block

    for (int rnd = 0;; ++rnd) {
        const long long hoff_cur = kv_off(cur);

        // this lane's query row: flat index f = r * G + h_local (computed
        // afresh per item, from values the compiler cannot hoist out of the
        // item loop)
        int ln = lane, Gi = G;
        opaque_v(ln);
        opaque_s(Gi);
        const int f = cur.tile * C::kTileRows + wave * kRowsPerWave + (ln & 31);
        const bool row_ok = f < flat_rows;
        const int r = row_ok ? f / Gi : 0;
        const int h = cur.g * Gi + (row_ok ? f % Gi : 0);
        const int kmax = row_ok ? (p.causal ? min(p.Sk - 1, r + off) : p.Sk - 1) : -1;
        int dslot = -1;
        if constexpr (DUMP) dslot = row_ok ? p.dump_slot[((long long)cur.b * p.Hq + h) * p.Sq + r] : -1;
        int kmax_wave_hi = kmax, kmax_wave_lo = row_ok ? kmax : 0x7fffffff;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            kmax_wave_hi = max(kmax_wave_hi, __shfl_xor(kmax_wave_hi, o, 64));
            kmax_wave_lo = min(kmax_wave_lo, __shfl_xor(kmax_wave_lo, o, 64));
        }
        // wave-uniform from here on: keeps the skip and mask branches scalar
        kmax_wave_hi = __builtin_amdgcn_readfirstlane(kmax_wave_hi);
        kmax_wave_lo = __builtin_amdgcn_readfirstlane(kmax_wave_lo);

        // Alg. 1 state of this lane's row.  The output and the denominator are
        // kept relative to the current block reference ref_j instead of the
        // running maximum m_j: X_j = sum_{i<=j} 2^(ref_i - ref_j) P_i V_i and
        // dX_j likewise, so O~_j = 2^(ref_j - m_j) X_j and d_j = 2^(ref_j - m_j) dX_j.
        // The two power-of-two rescales of a block (2^(m_{j-1}-m_j) on the old
        // state, 2^(ref_j - m_j) on the new block) fold into one exact rescale by
        // 2^(ref_{j-1} - ref_j), needed only when the reference moves, and the
        // normalisation O = O~/d = X/dX is unchanged.
        bool q_ready = false;           // the next item's Q was loaded during the last block
        float m = ninf;                 // running integer maximum m_j
        float ref = ninf;               // current block reference
        float dl = 0.0f;                // this lane's share of dX
        unsigned n_restart = 0, n_visit = 0;
        f32x16 oacc[kDT];
#pragma unroll
        for (int t = 0; t < kDT; ++t) oacc[t] = f32x16{};

        for (int jb = 0; jb < cur.nblk; ++jb, sel ^= 1) {
            const int key0 = jb * BLK;
            const char* kt_lds = tiles + sel * 2 * C::kTileBytes;
            const char* vt_lds = kt_lds + C::kTileBytes;
            __builtin_amdgcn_s_waitcnt(0);                  // this wave's loads of block jb (and Q) landed
            __syncthreads();                                // everyone's did; block jb-1 fully consumed
            // the next block of this item, or the first block of the next
            // item while the last one is computed
            const bool last = jb + 1 == cur.nblk;
            ItemGeo e_next;
            bool has_next = false;
            if (!last) {
                issue_block(hoff_cur, jb + 1, sel ^ 1);
            } else if constexpr (PERSIST) {
                has_next = item_of_round<BLK, C::kTileRows>(fresh_args(), rnd + 1, e_next);
                if (has_next && e_next.nblk > 0) issue_block(kv_off(e_next), 0, sel ^ 1);
            }
            // A wave that sees nothing of the block skips it.  In a tile that
            // spans waves it still takes part in the tile's exchange below, with
            // no visible row (its row maximum stays -inf): the exchange has one
            // barrier on one path, and the tile's representative lane counts the
            // block whenever any row of the tile sees it.
            const bool live = key0 <= kmax_wave_hi;
            if (!live && !(TILE && xwave)) continue;

            f32x16 sacc[kKT];
#pragma unroll
            for (int kt = 0; kt < kKT; ++kt) sacc[kt] = f32x16{};
            float amax = ninf;
            if (live) {
            // S^T = K_j Q^T.  The wave raises its priority for the MFMA burst so
            // that the two waves sharing a SIMD drift apart: one runs its QK^T
            // MFMAs while the other runs the VALU softmax of its block.
            __builtin_amdgcn_s_setprio(2);
            if constexpr (F8) {
                // FP8 E4M3 on both sides, unit block scales (E8M0 127): the
                // dequantisation scales are folded into c
#pragma unroll
                for (int kk = 0; kk < kDK8; ++kk) {
#pragma unroll
                    for (int kt = 0; kt < kKT; ++kt) {
                        const char* kp = kt_lds + kt * 32 * D;
                        const u32x4 lo = *reinterpret_cast<const u32x4*>(kp + koff[2 * kk]);
                        const u32x4 hi = *reinterpret_cast<const u32x4*>(kp + koff[2 * kk + 1]);
                        sacc[kt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(cat8(lo, hi), qop8[kk], sacc[kt],
                                                                                   0, 0, 0, 127, 0, 127);
                    }
                }
            } else {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int kk = 0; kk < kDK; ++kk) {
                    const char* kp = kt_lds + koff[kk];
#pragma unroll
                    for (int kt = 0; kt < kKT; ++kt) {
                        const u32x4 a = *reinterpret_cast<const u32x4*>(kp + kt * 32 * C::kRowBytes);
                        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(qop[kk]), sacc[kt],
                                                                           0, 0, 0);
                    }
                }
                // keep kKReads operand reads in flight ahead of the MFMAs that
                // consume them (the default schedule keeps two, and the MFMAs
                // wait on LDS latency)
                constexpr int kKReads = 4;
                __builtin_amdgcn_sched_group_barrier(0x100, kKReads, 0);          // LDS reads
#pragma unroll
                for (int i = 0; i < kDK * kKT - kKReads; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // one MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);            // one LDS read
                }
                __builtin_amdgcn_sched_group_barrier(0x008, kKReads, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_setprio(0);
            if constexpr (PERSIST) {
                // the last block's Q^T reads are done: the next item's Q loads
                // behind this block's softmax and PV
                if (has_next) {
                    load_q(fresh_args(), e_next);
                    q_ready = true;
                }
            }
            // mask keys past kmax (causal diagonal, ragged tail); key of register
            // i of tile kt: key0 + 32*kt + 8*(i/4) + 4*half + i%4
            if (key0 + BLK - 1 > kmax_wave_lo) {
                asm volatile("" ::: "memory");          // keep this a real branch (no if-conversion)
                const int lim = kmax - key0 - 4 * half;
#pragma unroll
                for (int kt = 0; kt < kKT; ++kt)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (kt * 32 + 8 * (i / 4) + (i % 4) > lim) sacc[kt][i] = ninf;
            }
            if constexpr (DUMP) {
                if (dslot >= 0) {
                    float* dst = p.dump_acc + (long long)dslot * p.Sk;
#pragma unroll
                    for (int kt = 0; kt < kKT; ++kt)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const int key = key0 + 32 * kt + 8 * (i / 4) + 4 * half + i % 4;
                            if (key <= kmax) dst[key] = sacc[kt][i];
                        }
                }
            }
            // row maximum of the raw dot products (the scale c > 0 is monotone):
            // a 3-way tree over this lane's 16*kKT scores, then lanes l and l^32
            {
                float mx[16 * kKT];
#pragma unroll
                for (int kt = 0; kt < kKT; ++kt)
#pragma unroll
                    for (int i = 0; i < 16; ++i) mx[16 * kt + i] = sacc[kt][i];
                amax = tree_max<16 * kKT>(mx);
                amax = __builtin_fmaxf(amax, swap_halves(amax));
            }
            }  // live
            float nref;
            if constexpr (MODE == kModeE2E) {
                // block-aware precision rescaling (Alg. 1), per row, branch-free.
                // B0 blocks (and a first block with m = -inf) take the high-precision
                // path; B1 blocks restart when ceil(rowmax T) > lambda, where rowmax of
                // the 8-bit T = fl32(acc*c - m) is the 8-bit cast of the raw maximum's
                // T (the cast is monotone).
                const bool vis = (!TILE || row_ok) && amax != ninf;
                const bool in_b0 = (jb < p.n_b0) || (p.b0_last && jb == kmax / BLK);
                const bool forced = in_b0 || (m == ninf);
                // ceil(rowmax T) of the 8-bit T = fl32(acc*c - m): the 8-bit cast
                // of the raw maximum's T (the cast is monotone), then ceil
                const float xt = __builtin_fmaf(amax, c, -m);
                float ctq;
                bool restart;
                if constexpr (kDec) {
                    restart = forced || (xt >= p.dec_x0);
                    ctq = hif8_ceil_below9(xt);            // used only without a restart
                } else {
                    ctq = ceilf(hif8::round(xt, true, TIE));
                    restart = forced || (ctq > lam);
                }
                if constexpr (TILE) {
                    // the tile restarts when any of its rows that see the block would
                    const uint32_t wantb = (uint32_t)__ballot(vis && restart);
                    const uint32_t visb = (uint32_t)__ballot(vis);
                    const uint32_t b0b = (uint32_t)__ballot(vis && in_b0);
                    uint32_t tw, tv, tb;
                    if (!xwave) {
                        tw = wantb & tmask;
                        tv = visb & tmask;
                        tb = b0b & tmask;
                    } else {
                        if (lane == 0) {
                            tflag[wave][0] = wantb;
                            tflag[wave][1] = visb;
                            tflag[wave][2] = b0b;
                        }
                        __syncthreads();
                        uint32_t a = 0, vv = 0, z = 0;
                        for (int w = tw0; w < tw0 + twn; ++w) {
                            a |= tflag[w][0];
                            vv |= tflag[w][1];
                            z |= tflag[w][2];
                        }
                        tw = a & tmask;
                        tv = vv & tmask;
                        tb = z & tmask;
                    }
                    restart = tw != 0u;
                    if (trep && tv && !tb) {                    // a B1 tile-block
                        ++n_visit;
                        n_restart += restart ? 1u : 0u;
                    }
                } else if (count_blocks) {
                    const bool b1 = vis && !in_b0;
                    n_visit += b1 ? 1u : 0u;
                    n_restart += (b1 && restart) ? 1u : 0u;
                }
                const float m_hi = __builtin_fmaxf(m, ceilf(amax * c));    // ceil(rowmax S), S in fp32
                // (kDec, per row: a row that does not see the block has amax =
                // -inf, so T = -inf (m finite: no restart unless forced, ctq = 0)
                // or m = -inf (forced: m_hi = m), and m stays as it is)
                const float m_new = (kDec && !TILE) ? (restart ? m_hi : m + ctq)
                                                    : (vis ? (restart ? m_hi : m + __builtin_fmaxf(0.0f, ctq)) : m);
                const float ref_new = vis ? (restart ? m_hi : m) : ref;
                // (ref_new >= ref: the reference never decreases)
                const float f = (ref == ninf) ? 1.0f : exp2_nonpos_int(ref - ref_new);
                if (__any(f != 1.0f)) {
        #pragma unroll
                    for (int t = 0; t < kDT; ++t)
        #pragma unroll
                        for (int i = 0; i < 16; ++i) oacc[t][i] *= f;
                }
                dl *= f;
                m = m_new;
                ref = ref_new;
                if constexpr (DUMP) {
                    if (dslot >= 0 && half == 0 && vis) p.dump_ref[(long long)dslot * p.dump_nblk + jb] = ref;
                }
    
                // a row with no visible key so far keeps ref = -inf; its masked scores
                // (acc = -inf) must still give T = -inf and P = 0
                nref = (ref == ninf) ? 0.0f : -ref;
            } else {
                // eq. (2): real-valued running maximum m, rescale factor
                // 2^(m_old - m) in fp32 (Default) or HiF8(2^HiF8(m_old - m)) (Exp2 HiF8)
                const bool vis = amax != ninf;
                const float m_new = vis ? __builtin_fmaxf(m, amax * c) : m;   // fl32(max acc * c) = max S
                float f = 1.0f;
                if (m != ninf) {
                    const float x = m - m_new;
                    if constexpr (MODE == kModeDefault) {
                        f = __builtin_amdgcn_exp2f(x);
                    } else {
                        f = hif8::u2f((uint32_t)ctab[hif8::f2u(x) >> kTabShift] << 20) * 0x1p104f;
                    }
                }
                if (__any(f != 1.0f)) {
#pragma unroll
                    for (int t = 0; t < kDT; ++t)
#pragma unroll
                        for (int i = 0; i < 16; ++i) oacc[t][i] *= f;
                }
                dl *= f;
                m = m_new;
                ref = m_new;
                nref = (m == ninf) ? 0.0f : -m;
                if constexpr (DUMP) {
                    if (dslot >= 0 && half == 0 && vis) p.dump_ref[(long long)dslot * p.dump_nblk + jb] = ref;
                }
            }
    
            if (!live) continue;
            const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
            // T and the table entry of every score of the block first, written
            // ahead of the PV loop so that the gathers are in flight well
            // before the packing that reads them (T = fl32(acc*c - ref) rounded
            // once for Alg. 1; fl32(S - m) with S = fl32(acc*c) for Exp2 HiF8;
            // under ties to even a T with bits 18..0 zero reads the second half
            // of the table)
            uint32_t cd[kKT][16];
            if constexpr (MODE != kModeDefault) {
#pragma unroll
                for (int kt = 0; kt < kKT; ++kt)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const float t = MODE == kModeE2E ? __builtin_fmaf(sacc[kt][i], c, nref) : sacc[kt][i] * c + nref;
                        const uint32_t u = hif8::f2u(t);
                        uint32_t idx = u >> kTabShift;
                        if constexpr (TIE) idx |= (u & 0x7ffffu) ? 0u : (uint32_t)kTabEntries;
                        cd[kt][i] = CT ? (uint32_t)ctab[idx] : (uint32_t)tab[idx];
                    }
            }
#pragma unroll
            for (int kt = 0; kt < kKT; ++kt) {
                // P = HiF8(2^HiF8(T)), T = fl32(acc*c - ref), for this 32-key tile,
                // packed as two bf16 B operands
                u32x4 pop[2];
#pragma unroll
                for (int ch = 0; ch < 2; ++ch) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        uint32_t w;
                        if constexpr (MODE == kModeDefault) {
                            // P = 2^fl32(S - m) in fp32; bf16 into P V, fp32 into the sum
                            const float p0 = __builtin_amdgcn_exp2f(sacc[kt][ch * 8 + 2 * e] * c + nref);
                            const float p1 = __builtin_amdgcn_exp2f(sacc[kt][ch * 8 + 2 * e + 1] * c + nref);
                            const bf16x2 pb = {(__bf16)p0, (__bf16)p1};
                            w = __builtin_bit_cast(uint32_t, pb);
                            dl += p0 + p1;
                            pop[ch][e] = w;
                            continue;
                        }
                        // two bf16 of P * 2^-kCodeBiasLog2 (code table), or of P (score table)
                        if constexpr (CT) w = (cd[kt][ch * 8 + 2 * e] | (cd[kt][ch * 8 + 2 * e + 1] << 16)) << 4;
                        else w = cd[kt][ch * 8 + 2 * e] | (cd[kt][ch * 8 + 2 * e + 1] << 16);
                        pop[ch][e] = w;
                        dl = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, dl, false);
                    }
                }
                // X^T += V_j^T P^T over this tile's two 16-key chunks
#pragma unroll
                for (int ch = 0; ch < 2; ++ch) {
                    const int pc = 2 * kt + ch;
#pragma unroll
                    for (int t = 0; t < kDT; ++t) {
                        const char* pa = vt_lds + voff[t] + pc * 16 * C::kRowBytes;
                        const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, pa));
                        const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, pa + 8 * C::kRowBytes));
                        const u32x4 a = {__builtin_bit_cast(u32x2, va)[0], __builtin_bit_cast(u32x2, va)[1],
                                         __builtin_bit_cast(u32x2, vb)[0], __builtin_bit_cast(u32x2, vb)[1]};
                        oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(pop[ch]), oacc[t], 0, 0, 0);
                    }
                }
            }
        }

        // epilogue: O = X / dX, lse = ln2 (ref + log2 dX) = ln2 (m + log2 d);
        // with the compact table X and dX carry the factor 2^-kCodeBiasLog2
        const float d = dl + __shfl_xor(dl, 32, 64);
        const float dbias = (CT && MODE != kModeDefault) ? (float)kCodeBiasLog2 : 0.0f;
        const kargs_ptr a = fresh_args();
        if (row_ok) {
            const long long orow_off = (((long long)cur.b * a->Hq + h) * a->Sq + r) * D;
            const bool empty = (ref == ninf);
            const float inv = empty ? 0.0f : 1.0f / d;
            if (a->out_bf16) {
                uint16_t* orow = reinterpret_cast<uint16_t*>(a->o) + orow_off;
#pragma unroll
                for (int t = 0; t < kDT; ++t)
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const bf16x2 lo = {(__bf16)(oacc[t][q4 * 4 + 0] * inv), (__bf16)(oacc[t][q4 * 4 + 1] * inv)};
                        const bf16x2 hi = {(__bf16)(oacc[t][q4 * 4 + 2] * inv), (__bf16)(oacc[t][q4 * 4 + 3] * inv)};
                        *reinterpret_cast<u32x2*>(orow + t * 32 + q4 * 8 + half * 4) =
                            u32x2{__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
                    }
            } else {
                float* orow = a->o + orow_off;
#pragma unroll
                for (int t = 0; t < kDT; ++t)
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        f32x4 v;
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] = oacc[t][q4 * 4 + e] * inv;
                        *reinterpret_cast<f32x4*>(orow + t * 32 + q4 * 8 + half * 4) = v;
                    }
            }
            if (half == 0) {
                if (a->lse)
                    a->lse[((long long)cur.b * a->Hq + h) * a->Sq + r] =
                        empty ? ninf : 0.69314718055994531f * (ref + (log2f(d) + dbias));
                if ((TILE ? trep : true) && n_visit) {
                    if (a->counters) {
                        atomicAdd(a->counters + 2 * ((long long)cur.b * a->Hq + h) + 0, (unsigned long long)n_restart);
                        atomicAdd(a->counters + 2 * ((long long)cur.b * a->Hq + h) + 1, (unsigned long long)n_visit);
                    }
                    if (a->tile_counts) {
                        const int R = a->restart_rows;
                        unsigned long long* tc =
                            a->tile_counts + 2 * (((long long)cur.b * a->Hq + h) * ((a->Sq + R - 1) / R) + r / R);
                        atomicAdd(tc + 0, (unsigned long long)n_restart);
                        atomicAdd(tc + 1, (unsigned long long)n_visit);
                    }
                }
            }
        }
        // the next item: its first key block is on its way (loaded during
        // this item's last block); its Q is loaded now, behind the O stores
        // (the first block waits for both)
        ItemGeo nxt;
        if (!PERSIST || !item_of_round<BLK, C::kTileRows>(a, rnd + 1, nxt)) break;
        if (cur.nblk == 0 && nxt.nblk > 0) issue_block(kv_off(nxt), 0, sel);
        if (!q_ready) load_q(a, nxt);
        cur = nxt;
    }
}

template <int D, int BLK, int NW, bool CT, int MODE, bool TILE, bool F8, bool TIE, bool DUMP>
hipError_t launch_one(const AttnParams& p, hipStream_t st)
{
    using C = Cfg<D, BLK, NW>;
    // D = 128 takes the persistent grid (one workgroup per CU, whose LDS it
    // fills); D = 64 keeps one item per workgroup, which leaves the registers
    // for two resident workgroups per CU, and so does tile-level restart,
    // whose extra state would spill across the item loop
    constexpr bool kPersist = D == 128 && !TILE;
    const int lds = 4 * C::kTileBytes;
    const void* fn =
        reinterpret_cast<const void*>(&baps_attn_fwd_kernel<D, BLK, NW, CT, MODE, TILE, F8, kPersist, TIE, DUMP>);
    int dev = 0, ncu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    // resident workgroups per CU, found once per device ordinal below 64
    // (the kernel's resources do not depend on the call; 0: not yet found)
    static std::atomic<int> per_cu_of[64] = {};
    int per_cu = (dev >= 0 && dev < 64) ? per_cu_of[dev].load(std::memory_order_relaxed) : 0;
    if (per_cu == 0) {
        e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        if (e != hipSuccess) return e;
        int n = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, C::kThreads, lds);
        if (e != hipSuccess) return e;
        per_cu = n > 0 ? n : 1;
        if (dev >= 0 && dev < 64) per_cu_of[dev].store(per_cu, std::memory_order_relaxed);
    }
    // persistent grid: every work item (query tile, key/value head, batch)
    // on at most as many workgroups as the GPU holds at once
    const long long flat = (long long)p.Sq * (p.Hq / p.Hkv);
    const long long items = (flat + C::kTileRows - 1) / C::kTileRows * p.Hkv * p.B;
    const long long slots = (long long)ncu * per_cu;
    const unsigned grid = (unsigned)(kPersist && items > slots ? slots : items);
    hipLaunchKernelGGL((baps_attn_fwd_kernel<D, BLK, NW, CT, MODE, TILE, F8, kPersist, TIE, DUMP>), dim3(grid),
                       dim3(C::kThreads), lds, st, p);
    return hipGetLastError();
}

template <int D, int BLK, bool DUMP>
hipError_t launch_d_blk_dump(const AttnParams& p, hipStream_t st)
{
    // few rows per key/value head (decode, short queries): the HBM-streaming
    // kernel, which holds a tile of restart_rows query positions when it fits
    // in its 16 rows
    const int G = p.Hq / p.Hkv;
    const long long flat = (long long)p.Sq * G;
    if (flat <= 64 && (long long)p.restart_rows * G <= 16) return launch_attention_decode(p, D, BLK, st);
    if (p.tie_even)                                // ties to even (canonical per-row path only)
        return launch_one<D, BLK, 8, true, kModeE2E, false, false, true, DUMP>(p, st);
    if (p.qk_f8) {                                 // FP8 Q/K (per-row restart only)
        if (p.mode == kModeDefault) return launch_one<D, BLK, 8, true, kModeDefault, false, true, false, DUMP>(p, st);
        if (p.mode == kModeExp2) return launch_one<D, BLK, 8, true, kModeExp2, false, true, false, DUMP>(p, st);
        if (p.lambda <= kCodeMaxLambda) return launch_one<D, BLK, 8, true, kModeE2E, false, true, false, DUMP>(p, st);
        return launch_one<D, BLK, 8, false, kModeE2E, false, true, false, DUMP>(p, st);
    }
    if (p.mode == kModeDefault) return launch_one<D, BLK, 8, true, kModeDefault, false, false, false, DUMP>(p, st);
    if (p.mode == kModeExp2) return launch_one<D, BLK, 8, true, kModeExp2, false, false, false, DUMP>(p, st);
    if (p.restart_rows > 1) {
        if (p.lambda <= kCodeMaxLambda) return launch_one<D, BLK, 8, true, kModeE2E, true, false, false, DUMP>(p, st);
        return launch_one<D, BLK, 8, false, kModeE2E, true, false, false, DUMP>(p, st);
    }
    if (p.lambda <= kCodeMaxLambda) return launch_one<D, BLK, 8, true, kModeE2E, false, false, false, DUMP>(p, st);
    return launch_one<D, BLK, 8, false, kModeE2E, false, false, false, DUMP>(p, st);
}

template <int D, int BLK>
hipError_t launch_d_blk(const AttnParams& p, hipStream_t st)
{
    return p.dump_slot ? launch_d_blk_dump<D, BLK, true>(p, st) : launch_d_blk_dump<D, BLK, false>(p, st);
}

}  // namespace

hipError_t launch_attention(const AttnParams& p, int D, int block, hipStream_t st)
{
    if (D == 64 && block == 32) return launch_d_blk<64, 32>(p, st);
    if (D == 64 && block == 64) return launch_d_blk<64, 64>(p, st);
    if (D == 64 && block == 128) return launch_d_blk<64, 128>(p, st);
    if (D == 128 && block == 32) return launch_d_blk<128, 32>(p, st);
    if (D == 128 && block == 64) return launch_d_blk<128, 64>(p, st);
    if (D == 128 && block == 128) return launch_d_blk<128, 128>(p, st);
    return hipErrorInvalidValue;
}

}  // namespace baps
