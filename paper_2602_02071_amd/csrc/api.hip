// C ABI of the BAPS HIP library: argument validation, the read-only score
// table, and dispatch to the kernels.  No allocation on any call path.
#include <cmath>
#include <cstring>
#include <mutex>

#include "../../include/baps.h"
#include "common.hpp"

namespace {

using namespace baps;

// The score table: entry i covers every fp32 value whose bits 31..19 equal
// i.  P = HiF8(2^HiF8(T)) (App. A: the power of two evaluated on the 8-bit
// input and rounded back to 8 bits), as fp32 bits with the HiF8 code of P
// in the low byte.  Lives in static device memory, one copy per device.
__device__ uint32_t g_score_table[kTabEntries];
// The compact code table of the fused attention kernels (see common.hpp).
__device__ __attribute__((aligned(256))) uint8_t g_code_table[kCodeTableBytes];
// The same table expanded to every score-table index (indices below kCodeLo
// take the entry of kCodeLo, above kCodeHi that of kCodeHi), so that a lookup
// needs no clamp; the prefill kernel copies it into LDS as it is.
__device__ __attribute__((aligned(1024))) uint8_t g_code_table_x[kTabEntries];
// Both tables for ties to even: the entry of an index is the P of the T whose
// bits 31..19 are the index and whose bits 18..0 are zero (the one T of the
// index that can be a tie); every other T reads the tables above.
__device__ __attribute__((aligned(256))) uint8_t g_code_table_even[kCodeTableBytes];
__device__ __attribute__((aligned(1024))) uint8_t g_code_table_x_even[kTabEntries];

// HiF8 value of a double, rounded once: truncating to fp32 toward zero keeps
// the sign, the exponent and the leading mantissa bits that decide a
// round-to-nearest-away HiF8 result.
float hif8_round_double(double y)
{
    if (std::isnan(y)) return std::nanf("");
    float f = (float)y;
    if (std::isinf(y)) return f;
    if (std::fabs((double)f) > std::fabs(y)) f = std::nextafterf(f, 0.0f);
    return hif8::round(f, true);
}

// 2^t for a HiF8 value t, rounded to HiF8 (saturating: 2^t beyond 2^15 gives 2^15)
float hif8_exp2(float t)
{
    if (std::isnan(t)) return t;
    if (t == -INFINITY) return 0.0f;
    if (t == INFINITY) return t;
    double y = std::exp2((double)t);
    if (std::isinf(y)) y = 1.0e300;
    return hif8_round_double(y);
}

// byte c = ((e + 23) << 3) | m of a HiF8 value p = 2^e (1 + m/8) >= 0 (0 for
// p = 0); values beyond 2^kCodeMaxLambda (unreachable for lambda <=
// kCodeMaxLambda) saturate to 255
uint8_t linear_code(float p)
{
    if (p == 0.0f) return 0;
    int e = 0;
    const float fr = std::frexp(p, &e);              // p = fr * 2^e, fr in [0.5, 1)
    e -= 1;
    const int m = (int)std::lround((2.0f * fr - 1.0f) * 8.0f);
    if (e > kCodeMaxLambda) return 255;
    return (uint8_t)(((e + 23) << 3) | m);
}

struct Table {
    uint32_t e[kTabEntries];
    uint8_t code[kCodeEntries], code_even[kCodeEntries];
    uint8_t codex[kTabEntries], codex_even[kTabEntries];
    Table()
    {
        for (uint32_t i = 0; i < (uint32_t)kTabEntries; ++i) {
            const float T = hif8::u2f(i << kTabShift);
            const float p = hif8_exp2(hif8::round(T, true));
            const uint32_t pb = hif8::f2u(p);
            e[i] = (pb & 0xffffff00u) | hif8::encode(p, true);
        }
        for (int i = 0; i < kCodeEntries; ++i) {
            code[i] = linear_code(hif8::u2f(e[kCodeLo + i] & 0xffffff00u));
            const float T = hif8::u2f((uint32_t)(kCodeLo + i) << kTabShift);
            code_even[i] = linear_code(hif8_exp2(hif8::round(T, true, true)));
        }
        for (int i = 0; i < kTabEntries; ++i) {
            const int ci = (i < kCodeLo ? kCodeLo : (i > kCodeHi ? kCodeHi : i)) - kCodeLo;
            codex[i] = code[ci];
            codex_even[i] = code_even[ci];
        }
    }
};

const Table& host_table()
{
    static Table t;
    return t;
}

constexpr int kMaxDevices = 64;
std::mutex g_mutex;

// Scratch of baps_attention_fwd_split_noalloc: the split-key workspace in
// static device memory, one copy per device (held until the process ends).
// In host code this name is a host-side stand-in, never a device address:
// g_dev_scratch[dev] holds the device's own address of it, taken once per
// device with that device current.
static __device__ __attribute__((aligned(256))) char scratch[BAPS_SPLIT_SCRATCH_BYTES];
void* g_dev_scratch[kMaxDevices] = {};
const uint32_t* g_dev_table[kMaxDevices] = {};
const uint8_t* g_dev_code[kMaxDevices] = {};
const uint8_t* g_dev_codex[kMaxDevices] = {};
const uint8_t* g_dev_code_even[kMaxDevices] = {};
const uint8_t* g_dev_codex_even[kMaxDevices] = {};


// the last HIP failure a call of this library met on the calling thread
thread_local hipError_t g_last_hip = hipSuccess;

int status_of(hipError_t e)
{
    if (e == hipSuccess) return BAPS_OK;
    g_last_hip = e;
    return BAPS_HIP_ERROR;
}

// HIP keeps the last failed call's error until it is read, whoever made the
// call (the runtime's own start-up included); the launchers read it after
// their launches, so it is cleared first: a launch is judged on its own.
void clear_stale_error() { (void)hipGetLastError(); }

// Upload one table to its device symbol; returns the symbol's device address.
template <typename T, size_t N>
int upload(const void* symbol, const T (&host)[N], const void** dev_addr)
{
    if (int st = status_of(hipMemcpyToSymbol(symbol, host, sizeof(host), 0, hipMemcpyHostToDevice))) return st;
    void* ptr = nullptr;
    if (int st = status_of(hipGetSymbolAddress(&ptr, symbol))) return st;
    if (!ptr) return BAPS_HIP_ERROR;
    *dev_addr = ptr;
    return BAPS_OK;
}

struct DevTables {
    const uint32_t* tab;
    const uint8_t *code, *codex, *code_even, *codex_even;
    void* scratch;
};

int table_on_current_device(const uint32_t** out, const uint8_t** code = nullptr, const uint8_t** codex = nullptr,
                            DevTables* all = nullptr)
{
    int dev = 0;
    if (int st = status_of(hipGetDevice(&dev))) return st;
    if (dev < 0 || dev >= kMaxDevices) return BAPS_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_mutex);
    if (!g_dev_table[dev]) {
        const Table& t = host_table();
        if (int st = status_of(hipMemcpyToSymbol(HIP_SYMBOL(g_score_table), t.e, sizeof(t.e), 0,
                                                 hipMemcpyHostToDevice)))
            return st;
        void* ptr = nullptr;
        if (int st = status_of(hipGetSymbolAddress(&ptr, HIP_SYMBOL(g_score_table)))) return st;
        if (int st = status_of(hipMemcpyToSymbol(HIP_SYMBOL(g_code_table), t.code, sizeof(t.code), 0,
                                                 hipMemcpyHostToDevice)))
            return st;
        void* cptr = nullptr;
        if (int st = status_of(hipGetSymbolAddress(&cptr, HIP_SYMBOL(g_code_table)))) return st;
        if (int st = status_of(hipMemcpyToSymbol(HIP_SYMBOL(g_code_table_x), t.codex, sizeof(t.codex), 0,
                                                 hipMemcpyHostToDevice)))
            return st;
        void* xptr = nullptr;
        if (int st = status_of(hipGetSymbolAddress(&xptr, HIP_SYMBOL(g_code_table_x)))) return st;
        if (!ptr || !cptr || !xptr) return BAPS_HIP_ERROR;
        const void *eptr = nullptr, *exptr = nullptr;
        if (int st = upload(HIP_SYMBOL(g_code_table_even), t.code_even, &eptr)) return st;
        if (int st = upload(HIP_SYMBOL(g_code_table_x_even), t.codex_even, &exptr)) return st;
        void* sptr = nullptr;
        if (int st = status_of(hipGetSymbolAddress(&sptr, HIP_SYMBOL(scratch)))) return st;
        if (!sptr) return BAPS_HIP_ERROR;
        g_dev_scratch[dev] = sptr;

        g_dev_code_even[dev] = static_cast<const uint8_t*>(eptr);
        g_dev_codex_even[dev] = static_cast<const uint8_t*>(exptr);
        g_dev_code[dev] = static_cast<const uint8_t*>(cptr);
        g_dev_codex[dev] = static_cast<const uint8_t*>(xptr);
        g_dev_table[dev] = static_cast<const uint32_t*>(ptr);
    }
    *out = g_dev_table[dev];
    if (code) *code = g_dev_code[dev];
    if (codex) *codex = g_dev_codex[dev];
    if (all) *all = DevTables{g_dev_table[dev], g_dev_code[dev], g_dev_codex[dev], g_dev_code_even[dev],
                              g_dev_codex_even[dev], g_dev_scratch[dev]};
    return BAPS_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// The least fp32 value T with ceil(HiF8(T)) > lambda (ties away), -inf when
// every T has it: ceil(HiF8(.)) does not decrease with T, so a binary search
// over the fp32 values in order finds the step.  Alg. 1 restarts a block in
// B1 exactly when the 8-bit T of its row maximum reaches it.
float restart_threshold(int lambda)
{
    auto key_value = [](uint32_t key) {              // key order = value order over all non-NaN fp32
        const uint32_t bits = (key & 0x80000000u) ? (key & 0x7fffffffu) : ~key;
        return hif8::u2f(bits);
    };
    auto above = [&](uint32_t key) { return std::ceil(hif8::round(key_value(key), true)) > (float)lambda; };
    uint32_t lo = 0x007fffffu, hi = 0xff800000u;      // keys of -inf and +inf
    if (above(lo)) return -INFINITY;
    if (!above(hi)) return INFINITY;
    while (hi - lo > 1) {                             // above(lo) false, above(hi) true
        const uint32_t mid = lo + (hi - lo) / 2;
        if (above(mid)) hi = mid; else lo = mid;
    }
    return key_value(hi);
}


// Canonical knobs when the caller passes none.
baps_params_t knobs_of(const baps_params_t* prm)
{
    if (prm) return *prm;
    baps_params_t k;
    std::memset(&k, 0, sizeof(k));
    k.lambda = 1;
    k.n_b0 = 1;
    k.mode = BAPS_MODE_E2E_HIF8;
    k.saturate = 1;
    return k;
}

bool pow2(long long x) { return x > 0 && (x & (x - 1)) == 0; }

// The tile height the kernels use: one row per tile unless restart_rows > 1
// and Sq > 1; a tile taller than the query rows is the same single tile as
// the smallest power of two >= Sq.
int effective_rows(int R, int Sq)
{
    if (R <= 1 || Sq <= 1) return 1;
    long long p2 = 1;
    while (p2 < Sq) p2 <<= 1;
    return (int)(R < p2 ? R : p2);
}

// Argument checks and the launch descriptor shared by the one-pass and the
// split-key paths (no HIP call; the device tables are attached by
// attach_tables); returns a status (BAPS_OK with *empty set: nothing to do).
int make_params(const void* q, const void* k, const void* v, float* o, float* lse, int B, int Hq, int Hkv,
                int Sq, int Sk, int D, int causal, int block, const baps_params_t& kn, AttnParams* out,
                bool* empty)
{
    *empty = false;
    const int mode = kn.mode;
    if (mode != BAPS_MODE_E2E_HIF8 && mode != BAPS_MODE_DEFAULT && mode != BAPS_MODE_EXP2_HIF8)
        return BAPS_INVALID_ARGUMENT;
    if (B < 0 || Hq < 0 || Hkv < 0 || Sq < 0 || Sk < 0 || kn.n_b0 < 0 || kn.restart_rows < 0)
        return BAPS_INVALID_ARGUMENT;
    if (!(kn.scale_log2 >= 0.0f) || std::isinf(kn.scale_log2)) return BAPS_INVALID_ARGUMENT;
    if (B == 0 || Hq == 0 || Sq == 0) {
        *empty = true;
        return BAPS_OK;
    }
    if (Hkv == 0 || Hq % Hkv != 0) return BAPS_INVALID_ARGUMENT;
    if (!q || !o || (Sk > 0 && (!k || !v))) return BAPS_INVALID_ARGUMENT;
    if (!aligned16(q) || !aligned16(o) || (Sk > 0 && (!aligned16(k) || !aligned16(v))))
        return BAPS_INVALID_ARGUMENT;
    if (!(D == 64 || D == 128) || !(block == 32 || block == 64 || block == 128)) return BAPS_UNSUPPORTED;
    if ((long long)Sq * (Hq / Hkv) > 0x7fffffffLL || Hkv > 65535 || B > 65535) return BAPS_UNSUPPORTED;
    if (kn.qk_format != BAPS_QK_BF16 && kn.qk_format != BAPS_QK_FP8_E4M3) return BAPS_INVALID_ARGUMENT;
    const bool f8 = kn.qk_format == BAPS_QK_FP8_E4M3;
    if (f8 && !(kn.q_scale > 0.0f && kn.k_scale > 0.0f && std::isfinite(kn.q_scale) && std::isfinite(kn.k_scale)))
        return BAPS_INVALID_ARGUMENT;
    const int G = Hq / Hkv;
    if (kn.restart_rows > 1 && !pow2(kn.restart_rows)) return BAPS_UNSUPPORTED;
    const int R = effective_rows(kn.restart_rows, Sq);
    if (R > 1 && (mode != BAPS_MODE_E2E_HIF8 || !pow2(G) || G > 32 || (long long)R * G > 256 || f8))
        return BAPS_UNSUPPORTED;
    if (kn.tie_mode != BAPS_TIES_AWAY && kn.tie_mode != BAPS_TIES_EVEN) return BAPS_INVALID_ARGUMENT;
    const bool even = kn.tie_mode == BAPS_TIES_EVEN;
    if (even && (mode != BAPS_MODE_E2E_HIF8 || kn.lambda > kCodeMaxLambda || R > 1 || f8)) return BAPS_UNSUPPORTED;
    // without saturation a cast overflows only when an 8-bit P can exceed
    // 2^15, i.e. from lambda 16 up (T <= lambda otherwise, and the eq. (2)
    // setups have T <= 0): below that both settings give the same result
    if (!kn.saturate && mode == BAPS_MODE_E2E_HIF8 && kn.lambda > 15) return BAPS_UNSUPPORTED;
    if (kn.out_bf16 && !aligned16(o)) return BAPS_INVALID_ARGUMENT;
    AttnParams& p = *out;
    p.tab = nullptr;
    p.ctab = nullptr;
    p.ctabx = nullptr;
    p.dec_x0 = restart_threshold(kn.lambda);
    p.q = static_cast<const uint16_t*>(q);
    p.k = static_cast<const uint16_t*>(k);
    p.v = static_cast<const uint16_t*>(v);
    p.o = o;
    p.lse = lse;
    p.counters = kn.restart_counts;
    p.tile_counts = kn.tile_counts;
    p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.Sq = Sq; p.Sk = Sk;
    p.causal = causal ? 1 : 0;
    p.lambda = kn.lambda;
    p.n_b0 = kn.n_b0;
    p.mode = mode;
    p.restart_rows = R;
    p.b0_last = kn.b0_last ? 1 : 0;
    p.qk_f8 = f8 ? 1 : 0;
    p.out_bf16 = kn.out_bf16 ? 1 : 0;
    p.tie_even = even ? 1 : 0;
    p.ctab_even = nullptr;
    p.ctabx_even = nullptr;
    p.dump_slot = nullptr;
    p.dump_acc = nullptr;
    p.dump_ref = nullptr;
    p.dump_nblk = 0;
    // the score scale in log2 units; with FP8 Q/K the dequantisation scales
    // fold into it, in double, rounded once
    const double base = kn.scale_log2 > 0.0f ? (double)kn.scale_log2 : 1.4426950408889634 / std::sqrt((double)D);
    p.c = (float)(f8 ? base * (double)kn.q_scale * (double)kn.k_scale : base);
    if (!(p.c > 0.0f) || std::isinf(p.c)) return BAPS_UNSUPPORTED;
    return BAPS_OK;
}

int attach_tables(AttnParams* p)
{
    const uint32_t* tab = nullptr;
    DevTables t{};
    const int st = table_on_current_device(&tab, nullptr, nullptr, &t);
    p->tab = t.tab;
    p->ctab = t.code;
    p->ctabx = t.codex;

    p->ctab_even = t.code_even;
    p->ctabx_even = t.codex_even;
    return st;
}

int attention_impl(const void* q, const void* k, const void* v, float* o, float* lse, int B, int Hq,
                   int Hkv, int Sq, int Sk, int D, int causal, int block, const baps_params_t& kn, void* stream)
{
    AttnParams p;
    bool empty = false;
    int st = make_params(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, kn, &p, &empty);
    if (st || empty) return st;
    if ((st = attach_tables(&p))) return st;
    clear_stale_error();
    return status_of(launch_attention(p, D, block, static_cast<hipStream_t>(stream)));
}

// The split-key plan of a call: used for few rows per key/value head (the
// decode kernels' regime), few (batch, key/value head) row tiles and many
// key blocks, in the E2E HiF8 setup with the compact code table.
struct SplitPlan {
    bool use = false;
    int nblk = 0, bstride = 0, nsplit = 0, bps = 0;
    long long off_acc = 0, off_bmax = 0, off_part = 0, bytes = 0;
};

long long align256(long long x) { return (x + 255) & ~255LL; }

SplitPlan split_plan(int B, int Hq, int Hkv, int Sq, int Sk, int D, int block, const baps_params_t& kn)
{
    SplitPlan sp;
    if (B <= 0 || Hq <= 0 || Hkv <= 0 || Sq <= 0 || Sk <= 0 || Hq % Hkv) return sp;
    if (!(D == 64 || D == 128) || !(block == 32 || block == 64 || block == 128)) return sp;
    if (kn.mode != BAPS_MODE_E2E_HIF8 || kn.lambda > kCodeMaxLambda || kn.tie_mode != BAPS_TIES_AWAY) return sp;
    if (kn.restart_rows < 0 || effective_rows(kn.restart_rows, Sq) > 1) return sp;   // per-row decisions only
    const long long flat = (long long)Sq * (Hq / Hkv);
    if (flat > 64) return sp;                                   // the prefill kernel's regime
    const long long tiles = (flat + 15) / 16;
    const long long streams = (long long)B * Hkv * tiles;
    const int nblk = (Sk + block - 1) / block;
    if (streams >= 256 || nblk < 4) return sp;                  // already enough workgroups
    long long want = (512 + streams - 1) / streams;             // about two workgroups per CU
    const long long fewest = (nblk + kSplitMaxBps - 1) / kSplitMaxBps;
    if (want < fewest) want = fewest;
    const int ns0 = (int)(want < nblk ? want : nblk);
    sp.bps = (nblk + ns0 - 1) / ns0;
    sp.nsplit = (nblk + sp.bps - 1) / sp.bps;
    if (sp.nsplit < 2) return sp;
    sp.use = true;
    sp.nblk = nblk;
    sp.bstride = (nblk + 255) / 256 * 256;
    const long long rows = (long long)B * Hkv * flat;
    long long off = 0;
    sp.off_acc = off;    off += align256(rows * nblk * (long long)block * 4);
    sp.off_bmax = off;   off += align256(rows * sp.bstride * 4);
    sp.off_part = off;   off += align256((long long)sp.nsplit * rows * (D + 4) * 4);
    sp.bytes = off;
    return sp;
}

// The split-key path of a call whose plan uses it.  workspace == nullptr
// takes the device's static scratch (the caller has checked the size).
int split_impl(const void* q, const void* k, const void* v, float* o, float* lse, int B, int Hq, int Hkv,
               int Sq, int Sk, int D, int causal, int block, const baps_params_t& kn, const SplitPlan& plan,
               void* workspace, long long workspace_bytes, void* stream)
{
    SplitParams sp;
    bool empty = false;
    int st = make_params(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, kn, &sp.a, &empty);
    if (st || empty) return st;
    if (workspace && (workspace_bytes < plan.bytes || ((uintptr_t)workspace & 255u))) return BAPS_INVALID_ARGUMENT;
    DevTables t{};
    const uint32_t* tab = nullptr;
    if ((st = table_on_current_device(&tab, nullptr, nullptr, &t))) return st;
    sp.a.tab = t.tab;
    sp.a.ctab = t.code;
    sp.a.ctabx = t.codex;

    sp.a.ctab_even = t.code_even;
    sp.a.ctabx_even = t.codex_even;
    if (!workspace) workspace = t.scratch;
    char* ws = static_cast<char*>(workspace);
    sp.acc = reinterpret_cast<float*>(ws + plan.off_acc);
    sp.bmax = reinterpret_cast<float*>(ws + plan.off_bmax);
    sp.part = reinterpret_cast<float*>(ws + plan.off_part);
    sp.nblk = plan.nblk;
    sp.bstride = plan.bstride;
    sp.nsplit = plan.nsplit;
    sp.bps = plan.bps;
    clear_stale_error();
    return status_of(launch_attention_split(sp, D, block, static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

long long baps_attention_split_workspace(int B, int Hq, int Hkv, int Sq, int Sk, int D, int block,
                                         const baps_params_t* prm)
{
    const SplitPlan sp = split_plan(B, Hq, Hkv, Sq, Sk, D, block, knobs_of(prm));
    return sp.use ? sp.bytes : 0;
}

int baps_attention_fwd_split(const void* q, const void* k, const void* v, float* o, float* lse, int B, int Hq,
                             int Hkv, int Sq, int Sk, int D, int causal, int block, const baps_params_t* prm,
                             void* workspace, long long workspace_bytes, void* stream)
{
    try {
        const baps_params_t kn = knobs_of(prm);
        const SplitPlan plan = split_plan(B, Hq, Hkv, Sq, Sk, D, block, kn);
        if (!plan.use) return attention_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, kn, stream);
        if (!workspace) return BAPS_INVALID_ARGUMENT;
        return split_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, kn, plan, workspace,
                          workspace_bytes, stream);
    } catch (...) {
        return BAPS_HIP_ERROR;
    }
}

int baps_attention_fwd_split_noalloc(const void* q, const void* k, const void* v, float* o, float* lse, int B,
                                     int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                                     const baps_params_t* prm, void* stream)
{
    try {
        const baps_params_t kn = knobs_of(prm);
        const SplitPlan plan = split_plan(B, Hq, Hkv, Sq, Sk, D, block, kn);
        if (!plan.use) return attention_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, kn, stream);
        if (plan.bytes > BAPS_SPLIT_SCRATCH_BYTES) return BAPS_UNSUPPORTED;
        return split_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, kn, plan, nullptr, 0, stream);
    } catch (...) {
        return BAPS_HIP_ERROR;
    }
}

int baps_attention_fwd(const void* q, const void* k, const void* v, float* o, float* lse, int B, int Hq,
                       int Hkv, int Sq, int Sk, int D, int causal, int block, void* stream)
{
    try {
        return attention_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, knobs_of(nullptr), stream);
    } catch (...) {
        return BAPS_HIP_ERROR;
    }
}

int baps_attention_fwd_ex(const void* q, const void* k, const void* v, float* o, float* lse, int B, int Hq,
                          int Hkv, int Sq, int Sk, int D, int causal, int block, const baps_params_t* prm,
                          void* stream)
{
    if (!prm) return BAPS_INVALID_ARGUMENT;
    try {
        return attention_impl(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, *prm, stream);
    } catch (...) {
        return BAPS_HIP_ERROR;
    }
}

int baps_attention_fwd_dump(const void* q, const void* k, const void* v, float* o, float* lse, int B, int Hq,
                            int Hkv, int Sq, int Sk, int D, int causal, int block, const baps_params_t* prm,
                            const int* row_slot, float* acc_out, float* ref_out, void* stream)
{
    try {
        const baps_params_t kn = knobs_of(prm);
        AttnParams p;
        bool empty = false;
        int st = make_params(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, kn, &p, &empty);
        if (st || empty) return st;
        if (!row_slot || (Sk > 0 && (!acc_out || !ref_out))) return BAPS_INVALID_ARGUMENT;
        if ((st = attach_tables(&p))) return st;
        p.dump_slot = row_slot;
        p.dump_acc = acc_out;
        p.dump_ref = ref_out;
        p.dump_nblk = (Sk + block - 1) / block;
        clear_stale_error();
        return status_of(launch_attention(p, D, block, static_cast<hipStream_t>(stream)));
    } catch (...) {
        return BAPS_HIP_ERROR;
    }
}

int hif8_encode(const float* x, unsigned char* codes, long long n, int flags, void* stream)
{
    if (n < 0 || (flags & ~(BAPS_HIF8_SATURATE | BAPS_HIF8_TIES_EVEN))) return BAPS_INVALID_ARGUMENT;
    if (n == 0) return BAPS_OK;
    if (!x || !codes) return BAPS_INVALID_ARGUMENT;
    clear_stale_error();
    return status_of(launch_hif8_encode(x, codes, n, (flags & BAPS_HIF8_SATURATE) != 0,
                                        (flags & BAPS_HIF8_TIES_EVEN) != 0, static_cast<hipStream_t>(stream)));
}

int hif8_decode(const unsigned char* codes, float* x, long long n, void* stream)
{
    if (n < 0) return BAPS_INVALID_ARGUMENT;
    if (n == 0) return BAPS_OK;
    if (!x || !codes) return BAPS_INVALID_ARGUMENT;
    clear_stale_error();
    return status_of(launch_hif8_decode(codes, x, n, static_cast<hipStream_t>(stream)));
}

int baps_softmax_block(const float* s, long long rows, long long cols, long long ld_s, int block, int lambda,
                       int n_b0, int flags, unsigned char* p_codes, int* ref_shift, float* m_final,
                       float* d_final, unsigned char* restarted, void* stream)
{
    if (rows < 0 || cols < 0 || ld_s < cols || n_b0 < 0 || flags != 0) return BAPS_INVALID_ARGUMENT;
    if (!(block == 64 || block == 128 || block == 256 || block == 512 || block == 1024)) return BAPS_UNSUPPORTED;
    if (rows == 0) return BAPS_OK;
    if (!m_final || !d_final || (cols > 0 && (!s || !p_codes || !ref_shift))) return BAPS_INVALID_ARGUMENT;
    if (rows > 4LL * 0x7fffffffLL) return BAPS_UNSUPPORTED;
    try {
        const uint32_t* tab = nullptr;
        int st = table_on_current_device(&tab);
        if (st) return st;
        SoftmaxBlockParams p;
        p.s = s; p.rows = rows; p.cols = cols; p.ld = ld_s;
        p.block = block; p.lambda = lambda; p.n_b0 = n_b0;
        p.codes = p_codes; p.ref_shift = ref_shift; p.m_final = m_final; p.d_final = d_final;
        p.restarted = restarted; p.tab = tab;
        clear_stale_error();
        return status_of(launch_softmax_block(p, static_cast<hipStream_t>(stream)));
    } catch (...) {
        return BAPS_HIP_ERROR;
    }
}

int baps_get_exp2_lut(unsigned char out_codes[256])
{
    if (!out_codes) return BAPS_INVALID_ARGUMENT;
    for (int c = 0; c < 256; ++c) out_codes[c] = hif8::encode(hif8_exp2(hif8::decode((uint8_t)c)), true);
    return BAPS_OK;
}

int baps_init(void)
{
    try {
        const uint32_t* tab = nullptr;
        return table_on_current_device(&tab);
    } catch (...) {
        return BAPS_HIP_ERROR;
    }
}

const char* baps_last_hip_error(void)
{
    return hipGetErrorName(g_last_hip);
}

const char* baps_status_string(int status)
{
    switch (status) {
    case BAPS_OK: return "ok";
    case BAPS_INVALID_ARGUMENT: return "invalid argument";
    case BAPS_UNSUPPORTED: return "unsupported shape or option";
    case BAPS_HIP_ERROR: return "HIP runtime error";
    default: return "unknown status";
    }
}

}  // extern "C"
