// Shared device-side helpers and launch descriptors of the BAPS HIP library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "hif8.hpp"

namespace baps {

// Host-side set-up done once per device and kernel (a launch attribute, an
// occupancy query): one bit per device ordinal below 64, set once the step
// succeeded there.  Concurrent first calls may both run the step, which is
// idempotent.  Ordinals from 64 up run it on every call.
struct DeviceOnce {
    std::atomic<unsigned long long> done{0};
    bool is_done(int dev) const
    {
        return dev >= 0 && dev < 64 && (done.load(std::memory_order_acquire) >> dev & 1ull);
    }
    void mark(int dev)
    {
        if (dev >= 0 && dev < 64) done.fetch_or(1ull << dev, std::memory_order_release);
    }
};

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Entries of the score table, indexed by bits 31..19 of an fp32 value T:
// P = HiF8(2^HiF8(T)) as fp32 bits in bits 31..8, and the HiF8 code of P in
// bits 7..0 (every HiF8 value has at most 3 mantissa bits, so bits 19..0 of
// its fp32 pattern are zero).  The upper 16 bits are P in bf16, exactly.
constexpr int kTabEntries = 8192;
constexpr int kTabShift = 19;

// Compact code table of the fused attention kernels, for thresholds lambda
// <= kCodeMaxLambda.  Indexed like the score table (bits 31..19 of T) but
// clamped to [kCodeLo, kCodeHi]: every T <= lambda lands on an entry with the
// same P, since P = 1 for |T| < 2^-5 (either sign; the clamp sends positive T
// below 2^-5 to the entry of 2^-5) and P = 0 for T <= -32 (the clamp sends
// -inf and every T <= -32 to the entry of -32).  An entry is the byte
// c = ((e + 23) << 3) | m of P = 2^e (1 + m/8) (c = 0 for P = 0), chosen so
// that c << 4 is the bf16 pattern of P * 2^-kCodeBiasLog2, exactly: e runs
// over [-22, kCodeMaxLambda] and HiF8 keeps at most 3 mantissa bits.  In
// practice the hit entries sit in a few dozen LDS dwords: the gathers are
// nearly free of bank conflicts.  The prefill kernel expands the table in LDS
// to all 8192 indices (entry kCodeLo below, kCodeHi above the range), which
// takes the clamp off every lookup.
constexpr int kCodeLo = 0x7A0;           // T = +2^-5
constexpr int kCodeHi = 0x1840;          // T = -32
constexpr int kCodeEntries = kCodeHi - kCodeLo + 1;
constexpr int kCodeTableBytes = (kCodeEntries + 1023) / 1024 * 1024;   // device copy, zero-padded to whole KiB
constexpr int kCodeBiasLog2 = 104;
constexpr int kCodeMaxLambda = 8;

// max(0, ceil(HiF8(x))) (ties away) for x below 8.75, branch-free: below
// 2^-23 the cast gives 0 or less; from 2^-23 up to 16 it keeps at most 3
// mantissa bits, so with h half the spacing of x's binade (2^(e-4) in
// [2^e, 2^(e+1)) for e >= 0, below the spacing for e < 0) the cast exceeds an
// integer k exactly when x >= k + h (ties go away from zero), and
// ceil(HiF8(x)) = floor(x - h) + 1; x - h is exact (h is at least one unit in
// the last place of x).  Alg. 1's increment of the integer maximum when a
// block does not restart (T <= lambda <= 8).
__device__ __forceinline__ float hif8_ceil_below9(float x)
{
    const float h = hif8::u2f((hif8::f2u(x) & 0x7f800000u) - (4u << 23));
    const float r = floorf(x - h) + 1.0f;
    return x >= 0x1p-23f ? r : 0.0f;
}

// 2^k for an integer-valued k <= 0 (0 below the fp32 range)
__device__ __forceinline__ float exp2_nonpos_int(float k)
{
    return ldexpf(1.0f, (int)__builtin_fmaxf(k, -200.0f));
}

// Softmax setups of the fused attention kernels: the proposed workflow
// (Alg. 1, "E2E HiF8") and two setups of eq. (2) with a real-valued running
// maximum, "Default" (fp32 exp2) and "Exp2 HiF8" (the exp2 evaluated on 8-bit
// input and rounded to 8 bits), for comparison on the same tiling.
constexpr int kModeE2E = 0;
constexpr int kModeDefault = 1;
constexpr int kModeExp2 = 2;

struct AttnParams {
    const uint16_t* q;          // [B, Hq, Sq, D] bf16
    const uint16_t* k;          // [B, Hkv, Sk, D] bf16
    const uint16_t* v;          // [B, Hkv, Sk, D] bf16
    float* o;                   // [B, Hq, Sq, D]
    float* lse;                 // [B, Hq, Sq] or null
    const uint32_t* tab;        // score table (device)
    const uint8_t* ctab;        // compact code table (device), kCodeTableBytes bytes (entries, then zeros)
    const uint8_t* ctabx;       // the compact code table expanded to all kTabEntries indices (device)
    float dec_x0;               // the least fp32 T with ceil(HiF8(T)) > lambda (ties away): Alg. 1's
                                // restart test is T >= dec_x0
    unsigned long long* counters;  // [B*Hq][2] restarted / visited B1 tile-blocks, or null
    unsigned long long* tile_counts;  // [B*Hq][ceil(Sq/R)][2] the same per tile, or null
    int B, Hq, Hkv, Sq, Sk;
    int causal, lambda, n_b0;
    int mode;                   // kModeE2E, kModeDefault or kModeExp2
    int restart_rows;           // R: query positions of one head sharing the restart decision
    int b0_last;                // B0 also holds each row's last visible key block
    int qk_f8;                  // q and k hold FP8 E4M3 codes (c already holds the scales)
    float c;                    // log2(e)/sqrt(D) as fp32 (or the caller's override)
    int out_bf16;               // o holds bf16 (round to nearest even of the fp32 result)
    int tie_even;               // the 8-bit cast of T rounds ties to even (kernels built with TIE)
    const uint8_t* ctab_even;   // compact code table for exact ties under ties-to-even (device)
    const uint8_t* ctabx_even;  // the same expanded to all kTabEntries indices (device)
    // Score dump (kernels built with DUMP only): a query row whose
    // dump_slot[(b*Hq + h)*Sq + r] is s >= 0 writes its raw dot products q.k
    // to dump_acc[s*Sk + key] for every key it sees, and its reference (Alg.
    // 1's m~; the running maximum in the eq. (2) setups) after every key block
    // j it sees to dump_ref[s*dump_nblk + j]
    const int* dump_slot;
    float* dump_acc;
    float* dump_ref;
    int dump_nblk;
};

struct SoftmaxBlockParams {
    const float* s;
    long long rows, cols, ld;
    int block, lambda, n_b0;
    uint8_t* codes;
    int32_t* ref_shift;
    float* m_final;
    float* d_final;
    uint8_t* restarted;
    const uint32_t* tab;
};

// The split-key path of the few-rows kernels (decode with few (batch, KV
// head) streams and many keys).  Alg. 1's state after block j depends on the
// key blocks only through their row maxima, so the path runs in passes over
// a caller-provided workspace: the raw dot products and block maxima of every
// key split in parallel; then, per split in parallel, a per-row scan of Alg.
// 1's restart rule and integer maximum up to the split and P V at the
// references of that scan; last, per row, an exact power-of-two combine.
// The result is the sequential one up to the order of fp32 additions.
struct SplitParams {
    AttnParams a;               // the attention call (mode kModeE2E, lambda <= kCodeMaxLambda)
    float* acc;                 // [B*Hkv][flat][nblk*BLK] raw dot products q.k (-inf when masked)
    float* bmax;                // [B*Hkv][flat][bstride] raw row maximum of every key block
    float* part;                // [nsplit][B*Hkv][flat][D + 4] X, dX and the reference they are relative to
    int nblk, bstride;          // key blocks, and the block-maximum row stride (a multiple of 256)
    int nsplit, bps;            // splits, blocks per split (at most kSplitMaxBps)
};

constexpr int kSplitMaxBps = 32;  // key blocks per split of the split-key path

// exact 2^k for an integer-valued float k (0 below the fp32 range)
__device__ __forceinline__ float exp2_int(float k)
{
    if (k < -160.0f) return 0.0f;
    return ldexpf(1.0f, (int)k);
}

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// Wave-uniform maximum with DPP row ops (quad permutes and mirrors inside
// each row of 16 lanes, then row broadcasts): no LDS round trips.
__device__ __forceinline__ float dpp_max_step(float v, int ctrl, int row_mask)
{
    const int o = __builtin_bit_cast(int, v);
    switch (ctrl) {   // the DPP control must be a compile-time constant
    case 0xB1: return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0xB1, 0xF, 0xF, false)));
    case 0x4E: return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x4E, 0xF, 0xF, false)));
    case 0x141: return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x141, 0xF, 0xF, false)));
    case 0x140: return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x140, 0xF, 0xF, false)));
    case 0x142: return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x142, 0xA, 0xF, false)));
    default: return fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(o, o, 0x143, 0xC, 0xF, false)));
    }
}

__device__ __forceinline__ float wave_max_uniform(float v)
{
    v = dpp_max_step(v, 0xB1, 0xF);     // lane ^ 1
    v = dpp_max_step(v, 0x4E, 0xF);     // lane ^ 2
    v = dpp_max_step(v, 0x141, 0xF);    // mirror within 8
    v = dpp_max_step(v, 0x140, 0xF);    // mirror within 16
    v = dpp_max_step(v, 0x142, 0xA);    // row 0 -> 1, row 2 -> 3
    v = dpp_max_step(v, 0x143, 0xC);    // row 1 -> 2 and 3
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Host launchers (one per kernel family); return a hipError_t.
hipError_t launch_hif8_encode(const float* x, uint8_t* codes, long long n, bool saturate, bool even, hipStream_t st);
hipError_t launch_hif8_decode(const uint8_t* codes, float* x, long long n, hipStream_t st);
hipError_t launch_softmax_block(const SoftmaxBlockParams& p, hipStream_t st);
hipError_t launch_attention(const AttnParams& p, int D, int block, hipStream_t st);
hipError_t launch_attention_decode(const AttnParams& p, int D, int block, hipStream_t st);
hipError_t launch_attention_split(const SplitParams& sp, int D, int block, hipStream_t st);

}  // namespace baps
