/*
 * BAPS CPU oracle.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU implementation of what the BAPS
 * attention path computes, written from the paper "BAPS: A Fine-Grained
 * Low-Precision Scheme for Softmax in Attention via Block-Aware Precision
 * reScaling" (arXiv 2602.02071):
 *   - eq. (1)   standard attention (the fp64 exact reference),
 *   - eq. (2)   FlashAttention online softmax in base 2 (the "Default",
 *               "Exp2 HiF8", "Naive E2E" and "Exp2 FP8" setups of Sec. 4.1
 *               and Table 1),
 *   - eq. (3)   the offloaded subtraction T = S - rowfill(m~) (Sec. 3.2),
 *   - Sec. 3.3  integer powers of two for the rescale factors,
 *   - Alg. 1    the proposed workflow ("E2E HiF8", Sec. 4.1),
 *   - Alg. 2    (App. A) powers of two in HiF8, simulated through FP16,
 * plus the HiF8 number format the paper cites (Luo et al. 2024, "Ascend
 * HiFloat8 Format for Deep Learning"), decoded from its field layout.
 *
 * Floating point is fp64 unless the paper fixes the precision.  Nothing here
 * is blocked, fused or reordered beyond what those definitions state.  Only
 * the test suite, the smoke check and the benchmark's CPU-baseline leg load
 * this library; it shares no code, header or table with the HIP library.
 *
 * Readings taken where the paper is silent or inconsistent (each one is also
 * listed with its reason in the design notes of the repository):
 *   R1  HiF8 code layout: sign | dot (11,10,01,001,0001,0000) | sign-magnitude
 *       exponent with implicit leading one | mantissa; Inf = 0x6F/0xEF,
 *       NaN = 0x80, zero = 0x00.
 *   R2  rounding to nearest, ties away from zero, straight from the input
 *       value (one rounding, no FP16 intermediate); ties to even on request.
 *       The OCP FP8 formats of the Table 1 setups round ties to even.
 *   R3  finite overflow saturates to +-2^15; +-Inf stays +-Inf.
 *   R5  the 8-bit exp2 is E8(t) = HiF8(exp2(t)) with exp2 in fp64.
 *   R6  the integer row maximum uses ceil (Alg. 1).
 *   R7  the else-branch of Alg. 1 scales the new block by 2^(m~ - m) as well
 *       (the literal text leaves it unscaled; selectable for comparison).
 *   R8  the restart decision is taken per query row (per tile of query rows
 *       in orc_attention_tiles, the paper-literal granularity).
 *   R9  a B0 block is a forced restart: T = S - m and P = E8(HiF8(T)).
 *   R10 B0 = the first n_b0 key blocks (n_b0 = 1), blocks visited in order;
 *       orc_attention_tiles can add each row's last (diagonal) key block.
 *   R11 causal masks are bottom-right aligned: query r sees keys
 *       c <= r + Sk - Sq; masked scores are -inf and drop out.
 *   R13 lse = ln2 * (m + log2 d), natural log of the softmax denominator.
 *   R15 S = fl32(acc * c) with acc = fl32(q.k) (dot product in fp64, rounded
 *       once) and c = fl32(log2(e)/sqrt(d)); in the fused pass the product
 *       and the subtraction of eq. (3) are one operation rounded once:
 *       T = fl32(acc * c - ref).  Any acc within the fp32 summation bound of
 *       the exact q.k is an equally valid high-precision S: the caller may
 *       supply its own (a matrix unit's sums) and get the setup's result on
 *       exactly that S.
 *   R17 query head h reads key/value head h / (Hq/Hkv).
 */
#define _GNU_SOURCE
#include <math.h>
#include <pthread.h>
#include <sched.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

/* ------------------------------------------------------------------------ */
/* Number formats as value sets                                              */
/* ------------------------------------------------------------------------ */

typedef struct {
    int    n;              /* number of non-negative finite values, 0 included */
    double val[256];       /* ascending */
    int    code[256];      /* code of val[i] with a positive sign            */
    int    neg_bit;        /* OR-ed into a code to make it negative          */
    int    inf_code;       /* code of +Inf, -1 if the format has none        */
    int    nan_code;       /* canonical NaN code                             */
    double over_next;      /* nominal value after the maximum: a value rounds
                              to +Inf (non-saturating) when it is at least the
                              midpoint between the maximum and this value    */
    int    ties_even;      /* a value exactly halfway between two neighbours
                              goes to the one with an even significand (else
                              away from zero)                                */
} orc_format;

/* HiF8 decoding from the field layout (R1).  Returns the value of a code;
 * NaN for the NaN code, +-Inf for the infinity codes. */
double orc_hif8_decode(int code)
{
    int s = (code >> 7) & 1;
    int b = code & 0x7f;
    int es = 0, mag = 0, w, man, d_width;
    if ((b >> 5) == 3) {            /* dot 11: D = 4, exponents +-8..+-15, 1 mantissa bit */
        d_width = 4; es = (b >> 4) & 1; mag = 8 | ((b >> 1) & 7); w = 1; man = b & 1;
    } else if ((b >> 5) == 2) {     /* dot 10: D = 3, exponents +-4..+-7, 2 mantissa bits */
        d_width = 3; es = (b >> 4) & 1; mag = 4 | ((b >> 2) & 3); w = 2; man = b & 3;
    } else if ((b >> 5) == 1) {     /* dot 01: D = 2, exponents +-2, +-3, 3 mantissa bits */
        d_width = 2; es = (b >> 4) & 1; mag = 2 | ((b >> 3) & 1); w = 3; man = b & 7;
    } else if ((b >> 4) == 1) {     /* dot 001: D = 1, exponents +-1, 3 mantissa bits */
        d_width = 1; es = (b >> 3) & 1; mag = 1; w = 3; man = b & 7;
    } else if ((b >> 3) == 1) {     /* dot 0001: D = 0, exponent 0, 3 mantissa bits */
        d_width = 0; mag = 0; w = 3; man = b & 7;
    } else {                        /* dot 0000: zero, NaN and the denormals 2^(M-23) */
        man = b & 7;
        if (man == 0) return s ? NAN : 0.0;
        return (s ? -1.0 : 1.0) * ldexp(1.0, man - 23);
    }
    int e = es ? -mag : mag;
    if (d_width == 4 && e == 15 && man == 1) return s ? -INFINITY : INFINITY;
    return (s ? -1.0 : 1.0) * ldexp(1.0 + (double)man / (double)(1 << w), e);
}

/* OCP FP8 E4M3 (no infinities, max 448) and E5M2 (IEEE-like, max 57344),
 * used only by the "Exp2 E4M3/E5M2/E4M3xE5M2" setups of Table 1. */
static double e4m3_decode(int code)
{
    int s = (code >> 7) & 1, e = (code >> 3) & 15, m = code & 7;
    double v;
    if (e == 15 && m == 7) return NAN;
    if (e == 0) v = ldexp((double)m, -9);
    else v = ldexp(1.0 + m / 8.0, e - 7);
    return s ? -v : v;
}

static double e5m2_decode(int code)
{
    int s = (code >> 7) & 1, e = (code >> 2) & 31, m = code & 3;
    double v;
    if (e == 31) return m ? NAN : (s ? -INFINITY : INFINITY);
    if (e == 0) v = ldexp((double)m, -16);
    else v = ldexp(1.0 + m / 4.0, e - 15);
    return s ? -v : v;
}

static orc_format F_HIF8, F_HIF8_EVEN, F_E4M3, F_E5M2;

static void build_format(orc_format* f, double (*dec)(int), int inf_code, int nan_code,
                         double over_next, int ties_even)
{
    int n = 0;
    for (int c = 0; c < 128; ++c) {
        double v = dec(c);
        if (!isfinite(v)) continue;
        /* insertion sort keeps the table ascending */
        int i = n++;
        while (i > 0 && f->val[i - 1] > v) { f->val[i] = f->val[i - 1]; f->code[i] = f->code[i - 1]; --i; }
        f->val[i] = v; f->code[i] = c;
    }
    f->n = n; f->neg_bit = 0x80; f->inf_code = inf_code; f->nan_code = nan_code;
    f->over_next = over_next; f->ties_even = ties_even;
}

__attribute__((constructor)) static void init_formats(void)
{
    /* HiF8: ties away from zero (R2), or to even when asked; OCP E4M3 and
     * E5M2: to nearest even, the rounding of the OCP 8-bit float definition */
    build_format(&F_HIF8, orc_hif8_decode, 0x6f, 0x80, 1.5 * 32768.0, 0);
    build_format(&F_HIF8_EVEN, orc_hif8_decode, 0x6f, 0x80, 1.5 * 32768.0, 1);
    build_format(&F_E4M3, e4m3_decode, -1, 0x7f, 480.0, 1);
    build_format(&F_E5M2, e5m2_decode, 0x7c, 0x7f, 65536.0, 1);
}

/* Round-to-nearest by search over the value set.  At an exact tie the
 * format's rule decides: away from zero (HiF8, R2), or the neighbour whose
 * significand is even, i.e. whose value is an even multiple of the spacing
 * between the two neighbours (this is IEEE's ties-to-even; it sends a tie
 * between the largest value of a binade and the next power of two up, and a
 * tie between zero and the smallest value down to zero).  Returns the index
 * of the chosen non-negative value in f->val, or -1 for an overflow (+Inf,
 * or NaN in a format without Inf).  'a' is a non-negative magnitude (may be
 * +Inf; without saturation +Inf overflows). */
static int nearest_index(const orc_format* f, double a, int saturate)
{
    int top = f->n - 1;
    if (isinf(a)) return (f->inf_code >= 0 || !saturate) ? -1 : top;
    if (a >= f->val[top]) {
        if (saturate) return top;
        const double mid = 0.5 * (f->val[top] + f->over_next);
        if (a == mid && f->ties_even)
            return fmod(f->val[top] / (f->over_next - f->val[top]), 2.0) == 0.0 ? top : -1;
        return a >= mid ? -1 : top;
    }
    /* largest i with val[i] <= a */
    int lo = 0, hi = top;
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (f->val[mid] <= a) lo = mid; else hi = mid;
    }
    double midpoint = 0.5 * (f->val[lo] + f->val[lo + 1]);   /* exact in fp64 */
    if (a == midpoint && f->ties_even)
        return fmod(f->val[lo] / (f->val[lo + 1] - f->val[lo]), 2.0) == 0.0 ? lo : lo + 1;
    return a >= midpoint ? lo + 1 : lo;
}

static int fmt_encode(const orc_format* f, double x, int saturate)
{
    if (isnan(x)) return f->nan_code;
    int i = nearest_index(f, fabs(x), saturate);
    if (i < 0 && f->inf_code < 0) return f->nan_code;         /* overflow of a format without Inf */
    int code = i < 0 ? f->inf_code : f->code[i];
    if (code == 0) return 0;                       /* -0 has no code of its own */
    return signbit(x) ? (code | f->neg_bit) : code;
}

/* the value x rounds to (the 8-bit cast, "in 8-bit" of Alg. 1) */
static double fmt_round(const orc_format* f, double x, int saturate)
{
    if (isnan(x)) return x;
    int i = nearest_index(f, fabs(x), saturate);
    if (i < 0 && f->inf_code < 0) return NAN;
    double a = i < 0 ? INFINITY : f->val[i];
    return signbit(x) ? -a : a;
}

/* flags of the HiF8 cast: ORC_SAT clamps finite overflow to the largest
 * value, ORC_EVEN rounds ties to even (else away from zero) */
#define ORC_SAT 1
#define ORC_EVEN 2
static const orc_format* hif8_fmt(int flags) { return (flags & ORC_EVEN) ? &F_HIF8_EVEN : &F_HIF8; }

int orc_hif8_encode(double x, int flags) { return fmt_encode(hif8_fmt(flags), x, flags & ORC_SAT); }
double orc_hif8_round(double x, int flags) { return fmt_round(hif8_fmt(flags), x, flags & ORC_SAT); }
int orc_e4m3_encode(double x, int saturate) { return fmt_encode(&F_E4M3, x, saturate); }
int orc_e5m2_encode(double x, int saturate) { return fmt_encode(&F_E5M2, x, saturate); }
double orc_e4m3_decode(int c) { return e4m3_decode(c); }
double orc_e5m2_decode(int c) { return e5m2_decode(c); }

/* ------------------------------------------------------------------------ */
/* Threads                                                                   */
/* ------------------------------------------------------------------------ */

typedef void (*range_fn)(void* ctx, int64_t i0, int64_t i1);

typedef struct {
    range_fn fn; void* ctx; int64_t n, chunk; int64_t next;
} pool_job;

static void* pool_worker(void* arg)
{
    pool_job* j = (pool_job*)arg;
    for (;;) {
        int64_t i0 = __atomic_fetch_add(&j->next, j->chunk, __ATOMIC_RELAXED);
        if (i0 >= j->n) break;
        int64_t i1 = i0 + j->chunk < j->n ? i0 + j->chunk : j->n;
        j->fn(j->ctx, i0, i1);
    }
    return NULL;
}

int orc_default_threads(void)
{
    cpu_set_t set;
    if (sched_getaffinity(0, sizeof(set), &set) == 0) return CPU_COUNT(&set);
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

static void parallel_for(int64_t n, int nthreads, int64_t chunk, range_fn fn, void* ctx)
{
    if (n <= 0) return;
    if (nthreads <= 0) nthreads = orc_default_threads();
    if (nthreads > 256) nthreads = 256;
    if (chunk <= 0) chunk = 1;
    pool_job job = { fn, ctx, n, chunk, 0 };
    if (nthreads == 1 || n <= chunk) { fn(ctx, 0, n); return; }
    pthread_t th[256];
    int started = 0;
    for (int t = 0; t < nthreads; ++t)
        if (pthread_create(&th[t], NULL, pool_worker, &job) == 0) ++started;
    if (started == 0) { fn(ctx, 0, n); return; }
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
}

/* ------------------------------------------------------------------------ */
/* Bulk encode and the exhaustive check helper                               */
/* ------------------------------------------------------------------------ */

typedef struct { const float* x; uint8_t* out; int flags; } enc_ctx;

static void enc_range(void* p, int64_t i0, int64_t i1)
{
    enc_ctx* c = (enc_ctx*)p;
    for (int64_t i = i0; i < i1; ++i) c->out[i] = (uint8_t)orc_hif8_encode((double)c->x[i], c->flags);
}

void orc_hif8_encode_f32(const float* x, uint8_t* out, int64_t n, int flags, int nthreads)
{
    enc_ctx c = { x, out, flags };
    parallel_for(n, nthreads, 1 << 16, enc_range, &c);
}

typedef struct { uint64_t start; const uint8_t* got; int flags; int64_t bad; int64_t first_bad; } chk_ctx;

static void chk_range(void* p, int64_t i0, int64_t i1)
{
    chk_ctx* c = (chk_ctx*)p;
    int64_t bad = 0, first = -1;
    for (int64_t i = i0; i < i1; ++i) {
        uint32_t bits = (uint32_t)(c->start + (uint64_t)i);
        float x; memcpy(&x, &bits, 4);
        int want = orc_hif8_encode((double)x, c->flags);
        if (want != c->got[i]) { if (first < 0) first = i; ++bad; }
    }
    if (bad) {
        __atomic_fetch_add(&c->bad, bad, __ATOMIC_RELAXED);
        int64_t cur = __atomic_load_n(&c->first_bad, __ATOMIC_RELAXED);
        while ((cur < 0 || first < cur) &&
               !__atomic_compare_exchange_n(&c->first_bad, &cur, first, 0, __ATOMIC_RELAXED, __ATOMIC_RELAXED)) {}
    }
}

/* Compares codes[i] against the encoding of the fp32 bit pattern start + i,
 * for i < count.  Returns the number of mismatches; *first_bad gets the
 * first mismatching index (or -1). */
int64_t orc_hif8_check_patterns(uint64_t start, int64_t count, const uint8_t* codes, int flags,
                                int nthreads, int64_t* first_bad)
{
    chk_ctx c = { start, codes, flags, 0, -1 };
    parallel_for(count, nthreads, 1 << 18, chk_range, &c);
    if (first_bad) *first_bad = c.first_bad;
    return c.bad;
}

/* ------------------------------------------------------------------------ */
/* Powers of two in 8 bits                                                   */
/* ------------------------------------------------------------------------ */

/* IEEE binary16 rounding (to nearest even, subnormals, overflow to Inf),
 * the FP16 carrier of Alg. 2. */
double orc_round_fp16(double y)
{
    if (isnan(y) || isinf(y) || y == 0.0) return y;
    double a = fabs(y);
    int e;
    frexp(a, &e);                      /* a = f * 2^e with f in [0.5, 1) */
    int ue = e - 1;                    /* unbiased exponent of a */
    if (ue < -14) ue = -14;            /* subnormal spacing is 2^-24 */
    double q = ldexp(1.0, ue - 10);    /* spacing of binary16 at a */
    double r = nearbyint(a / q) * q;   /* default rounding mode: ties to even */
    if (r > 65504.0) r = INFINITY;
    return copysign(r, y);
}

/* E8(t) = HiF8(2^t) for a HiF8 value t (R5). */
static double e8_hif8(double t)
{
    if (isnan(t)) return t;
    if (t == -INFINITY) return 0.0;
    double y = exp2(t);
    if (isinf(y)) y = 1.0e308;         /* a finite overflow, saturated below */
    return fmt_round(&F_HIF8, y, 1);
}

/* The 256-entry table code -> code of HiF8(2^decode(code)).
 * variant 0: fp64 exp2 with one HiF8 rounding (R5).
 * variant 1: Alg. 2 literally, with FP16 as the carrier of the exp2 result. */
void orc_exp2_table(uint8_t out[256], int variant)
{
    for (int c = 0; c < 256; ++c) {
        double x = orc_hif8_decode(c);
        if (isnan(x)) { out[c] = (uint8_t)F_HIF8.nan_code; continue; }
        if (x == INFINITY) { out[c] = (uint8_t)F_HIF8.inf_code; continue; }
        if (x == -INFINITY) { out[c] = 0; continue; }
        if (variant == 0) {
            out[c] = (uint8_t)fmt_encode(&F_HIF8, e8_hif8(x), 1);
        } else {
            /* x is a HiF8 value, so the FP16 -> HiF8 -> FP16 steps leave it unchanged */
            double y16 = orc_round_fp16(exp2(x));       /* exp2 evaluated in FP16 */
            out[c] = (uint8_t)fmt_encode(&F_HIF8, y16, 1);
        }
    }
}

/* Sec. 3.3 and Fig. 2: the error that a running product of rescale factors
 * 2^x_1 * 2^x_2 * ... picks up in the 8-bit pipeline.
 *   integer != 0: each exponent is first raised to an integer, k = ceil(x)
 *     (as the integer running maximum of Alg. 1 does), and the factor 2^k is
 *     exact; the ground truth is 2^(k_1 + ... + k_i).
 *   integer == 0 ("direct" exponents): each factor is the 8-bit pipeline's
 *     E8[Q8(x)], the exponent cast to HiF8 and its power of two cast to HiF8;
 *     the ground truth is 2^(x_1 + ... + x_i).
 * out[i] = log2 of (product of the first i+1 factors / ground truth), both
 * sides summed as log2 in fp64, so the result has no underflow at any
 * length and is exactly 0 when every factor is exact. */
void orc_power_product(const double* x, int64_t n, int integer, double* out)
{
    double lp = 0.0, lt = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        double f, t;
        if (integer) {
            t = ceil(x[i]);
            f = exp2(t);
        } else {
            t = x[i];
            f = e8_hif8(orc_hif8_round(x[i], 1));
        }
        lp += log2(f);
        lt += t;
        out[i] = lp - lt;
    }
}

/* ------------------------------------------------------------------------ */
/* Attention                                                                 */
/* ------------------------------------------------------------------------ */

enum {
    ORC_E2E_HIF8 = 0,       /* Alg. 1 (the "E2E HiF8" setup)                      */
    ORC_DEFAULT = 1,        /* eq. (2), softmax in fp32 ("Default")                */
    ORC_EXP2_HIF8 = 2,      /* eq. (2), every power of two in HiF8 ("Exp2 HiF8")   */
    ORC_NAIVE_E2E = 3,      /* eq. (2) on scores cast to HiF8 first ("Naive E2E")  */
    ORC_EXP2_E4M3 = 4,      /* Table 1 ablations: input/output formats of exp2     */
    ORC_EXP2_E5M2 = 5,
    ORC_EXP2_E4M3xE5M2 = 6,
    ORC_E2E_EXACT = 7       /* Alg. 1 control flow with the 8-bit casts removed and
                               all arithmetic in fp64 (quantizer off)              */
};

typedef struct {
    const uint16_t *q, *k, *v;
    int B, Hq, Hkv, Sq, Sk, D, causal, block;
    int mode, lambda, n_b0, literal_else;
    float c32;              /* log2(e)/sqrt(D) (or the override), as fp32 */
    double c64;             /* the same scale in fp64 (for ORC_E2E_EXACT and eq. (1)) */
    const int64_t* rows;
    double *o, *lse;
    int32_t* nrestart;      /* restarted B1 blocks per row (nullable) */
    double* margin;         /* decision margin per row (nullable), see row_alg1 */
    int pv_bf16;            /* eq. (2) setups: P enters the P V product rounded to bf16 */
    int hif8_flags;         /* the 8-bit cast of T (Alg. 1) and of x (Exp2 HiF8): ORC_SAT,
                               plus ORC_EVEN for ties to even */
    const float* acc_in;    /* nullable: the high-precision q.k of requested row i and key c
                               is acc_in[i * ld_acc + c] instead of fl32(q.k) */
    int64_t ld_acc;
    double* ref_out;        /* nullable: the reference of requested row i at its visible key
                               block j goes to ref_out[i * ld_ref + j] (Alg. 1: the m~ that
                               T = S - m~ is taken against; eq. (2): the running maximum m
                               after block j) */
    int64_t ld_ref;
    int err;                /* set when acc_in lacks a row that a tile decision needs */
} attn_job;

static inline double bf16_to_double(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f; memcpy(&f, &u, 4);
    return (double)f;
}

static inline int last_visible_key(const attn_job* J, int r)
{
    if (!J->causal) return J->Sk - 1;
    int kmax = r + J->Sk - J->Sq;               /* R11: bottom-right alignment */
    return kmax < J->Sk - 1 ? kmax : J->Sk - 1;
}

/* q.k of a query row and a key row, summed in fp64 (exact products) */
static double dot64(const uint16_t* a, const uint16_t* b, int D)
{
    double s = 0.0;
    for (int i = 0; i < D; ++i) s += bf16_to_double(a[i]) * bf16_to_double(b[i]);
    return s;
}

static double abs_dot64(const uint16_t* a, const uint16_t* b, int D)
{
    double s = 0.0;
    for (int i = 0; i < D; ++i) s += fabs(bf16_to_double(a[i]) * bf16_to_double(b[i]));
    return s;
}

/* Error bound of a matrix unit's dot product acc = q.k: the D products are
 * exact in fp32 (a bf16 x bf16 product has at most 16 significant bits), and
 * a sum of D terms formed with fp32 round-to-nearest additions, in any order,
 * lies within gamma_(D-1) * sum_d |q_d k_d| of the exact sum, where
 * gamma_n = n u / (1 - n u) and u = 2^-24 (the standard bound of recursive
 * summation; Higham, Accuracy and Stability of Numerical Algorithms, 2nd
 * ed., Sec. 4.2).  Every S within that bound is an equally valid "S in high
 * precision" of Alg. 1. */
static double acc_err(const uint16_t* a, const uint16_t* b, int D)
{
    const double n = (double)(D > 1 ? D - 1 : 0), u = ldexp(1.0, -24);
    return n * u / (1.0 - n * u) * abs_dot64(a, b, D);
}

/* The high-precision scores of one query row, keys 0 .. kmax (R15):
 * acc[c] = fl32(q.k_c) from the fp64 dot product (exact: the fp64 value
 * itself), or given[c] when the caller supplies the dot products; with eps
 * set, eps[c] = the accumulation error bound of key c in S units. */
static void row_scores(const attn_job* J, const uint16_t* qr, const uint16_t* kb, int kmax,
                       const float* given, int exact, double* acc, double* eps)
{
    const int D = J->D;
    for (int c = 0; c <= kmax; ++c) {
        const uint16_t* kr = kb + (int64_t)c * D;
        if (given) acc[c] = (double)given[c];
        else {
            const double a = dot64(qr, kr, D);
            acc[c] = exact ? a : (double)(float)a;
        }
        if (eps) eps[c] = acc_err(qr, kr, D) * J->c64;
    }
}

/* Distance from x to the nearest point where the HiF8 rounding of x changes. */
static double hif8_boundary_distance(double x)
{
    const orc_format* f = &F_HIF8;
    double a = fabs(x);
    int top = f->n - 1;
    if (a >= f->val[top]) return a - 0.5 * (f->val[top - 1] + f->val[top]);
    int lo = 0, hi = top;
    while (hi - lo > 1) {
        int mid = (lo + hi) / 2;
        if (f->val[mid] <= a) lo = mid; else hi = mid;
    }
    double up = 0.5 * (f->val[lo] + f->val[lo + 1]) - a;
    if (up < 0) up = -up;
    double down = lo > 0 ? a - 0.5 * (f->val[lo - 1] + f->val[lo]) : up;
    if (down < 0) down = -down;
    return up < down ? up : down;
}

static double integer_distance(double x)
{
    double a = x - floor(x), b = ceil(x) - x;
    return a < b ? a : b;
}

typedef struct { double *acc, *eps, *ot, *pv, *ref, *bmargin; } row_scratch;

/* One query row of Alg. 1.  acc_c = fl32(q.k_c) (R15); the block loop is
 * the B0 loop for j < n_b0 and the B1 loop afterwards.
 *
 * With J->margin set, the row also reports how far its 8-bit decisions sit
 * from a boundary, in units of the accumulation error bound of each score:
 * the HiF8 rounding of every T that carries weight >= 2^-12 of the final
 * maximum, the restart test of every B1 block, and the ceil of the row
 * maximum of every block that takes the high-precision path.  A margin of
 * at least 1 means every valid high-precision S gives this same result. */
static void row_alg1(const attn_job* J, int b, int h, int r, row_scratch* W, const float* given,
                     double* o, double* lse, int32_t* nrs, double* margin_out, double* refs_out)
{
    const int D = J->D, blk = J->block;
    const int g = h / (J->Hq / J->Hkv);                                   /* R17 */
    const uint16_t* qr = J->q + (((int64_t)b * J->Hq + h) * J->Sq + r) * D;
    const uint16_t* kb = J->k + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const uint16_t* vb = J->v + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const int exact = (J->mode == ORC_E2E_EXACT);
    const int kmax = last_visible_key(J, r);
    const int nblk = kmax < 0 ? 0 : kmax / blk + 1;
    const int want_margin = margin_out != NULL;
    double m = -INFINITY, d = 0.0;
    int32_t restarts = 0;
    for (int i = 0; i < D; ++i) W->ot[i] = 0.0;

    /* S = Q K^T * log2(e)/sqrt(d): keep acc, the unscaled dot product */
    row_scores(J, qr, kb, kmax, given, exact, W->acc, want_margin ? W->eps : NULL);

    for (int j = 0; j < nblk; ++j) {
        const int c0 = j * blk;
        const int c1 = (c0 + blk <= kmax + 1) ? c0 + blk : kmax + 1;   /* visible keys of block j */
        const double* acc = W->acc + c0;
        const int nc = c1 - c0;
        double bm = INFINITY, eps_blk = 0.0, amax = -INFINITY;
        for (int c = 0; c < nc; ++c) {
            if (want_margin && W->eps[c0 + c] > eps_blk) eps_blk = W->eps[c0 + c];
            if (acc[c] > amax) amax = acc[c];
        }
        int restart;
        double m_new = m, ref = m;
        if (j < J->n_b0) {
            restart = 1;                                                 /* B0 loop (R9) */
        } else {
            /* B1 loop: m~ = m^(j-1); T = S - rowfill(m~) in 8-bit; restart if
             * ceil(rowmax T) > lambda */
            double tmax = -INFINITY;
            for (int c = 0; c < nc; ++c) {
                double t;
                if (exact) t = acc[c] * J->c64 - m;
                else t = orc_hif8_round((double)fmaf((float)acc[c], J->c32, (float)(-m)), J->hif8_flags);
                if (t > tmax) tmax = t;
            }
            restart = ceil(tmax) > (double)J->lambda;
            if (want_margin && m != -INFINITY) {
                double x = amax * J->c64 - m;
                double dist = hif8_boundary_distance(x) / eps_blk;
                if (dist < bm) bm = dist;
            }
            if (!restart) {
                m_new = m + fmax(0.0, ceil(tmax));
                ref = m;                                                 /* m~ stays m^(j-1) */
            } else {
                ++restarts;
            }
        }
        if (restart) {
            /* S in high precision; m^(j) = max(m^(j-1), ceil(rowmax S)); m~ = m^(j) */
            double M = -INFINITY;
            for (int c = 0; c < nc; ++c) {
                double s = exact ? acc[c] * J->c64 : (double)((float)acc[c] * J->c32);
                if (s > M) M = s;
            }
            m_new = fmax(m, ceil(M));
            ref = m_new;
            if (want_margin) {
                double dist = integer_distance(amax * J->c64) / eps_blk;
                if (dist < bm) bm = dist;
            }
        }
        /* P = 2^T in 8-bit, T = S - rowfill(m~) in 8-bit (eq. 3) */
        double rowsum = 0.0;
        for (int i = 0; i < D; ++i) W->pv[i] = 0.0;
        for (int c = 0; c < nc; ++c) {
            double p;
            if (exact) p = exp2(acc[c] * J->c64 - ref);
            else {
                double t = orc_hif8_round((double)fmaf((float)acc[c], J->c32, (float)(-ref)), J->hif8_flags);
                p = e8_hif8(t);
            }
            if (p == 0.0) continue;
            rowsum += p;
            const uint16_t* vr = vb + (int64_t)(c0 + c) * D;
            for (int i = 0; i < D; ++i) W->pv[i] += p * bf16_to_double(vr[i]);
        }
        /* d and O~ with the exact integer powers of two of Sec. 3.3 (R7) */
        const double alpha = (m == -INFINITY) ? 0.0 : exp2(m - m_new);
        const double beta = (J->literal_else && !restart) ? 1.0 : exp2(ref - m_new);
        d = alpha * d + beta * rowsum;
        for (int i = 0; i < D; ++i) W->ot[i] = alpha * W->ot[i] + beta * W->pv[i];
        m = m_new;
        W->ref[j] = ref;
        W->bmargin[j] = bm;
        if (refs_out) refs_out[j] = ref;
    }
    if (margin_out) {
        double mg = INFINITY;
        if (!exact) {
            for (int j = 0; j < nblk; ++j) {
                if (W->bmargin[j] < mg) mg = W->bmargin[j];
                const int c0 = j * blk;
                const int c1 = (c0 + blk <= kmax + 1) ? c0 + blk : kmax + 1;
                for (int c = c0; c < c1; ++c) {
                    double x = W->acc[c] * J->c64 - W->ref[j];
                    double p = e8_hif8(orc_hif8_round((double)fmaf((float)W->acc[c], J->c32, (float)(-W->ref[j])),
                                                      J->hif8_flags));
                    if (ldexp(p, (int)(W->ref[j] - m)) < 1.0 / 4096.0) continue;
                    double dist = hif8_boundary_distance(x) / W->eps[c];
                    if (dist < mg) mg = dist;
                }
            }
        }
        *margin_out = mg;
    }
    if (nblk == 0) {
        for (int i = 0; i < D; ++i) o[i] = 0.0;
        *lse = -INFINITY;
    } else {
        for (int i = 0; i < D; ++i) o[i] = W->ot[i] / d;                 /* O = diag(d)^-1 O~ */
        *lse = M_LN2 * (m + log2(d));                                     /* R13 */
    }
    if (nrs) *nrs = restarts;
}

/* One query row of eq. (2) in the setups of Sec. 4.1 / Table 1 that keep the
 * real-valued running maximum: Default, Exp2 HiF8, Naive E2E, Exp2 FP8.
 * The softmax runs in fp32 as the Default setup states. */
/* p rounded to bf16 (to nearest, ties to even): the precision of the matrix
 * unit's inputs, at which P enters the P V product (pv_bf16) */
static float round_bf16(float p)
{
    uint32_t u;
    memcpy(&u, &p, 4);
    u = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
    memcpy(&p, &u, 4);
    return p;
}

static void row_eq2(const attn_job* J, int b, int h, int r, row_scratch* W, const float* given, double* o,
                    double* lse, double* margin_out, double* refs_out)
{
    const int D = J->D, blk = J->block;
    const int g = h / (J->Hq / J->Hkv);
    const uint16_t* qr = J->q + (((int64_t)b * J->Hq + h) * J->Sq + r) * D;
    const uint16_t* kb = J->k + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const uint16_t* vb = J->v + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const int kmax = last_visible_key(J, r);
    const int nblk = kmax < 0 ? 0 : kmax / blk + 1;
    const int want_margin = margin_out != NULL;
    /* (2^x of an 8-bit x is irrational or an exact power of two, never halfway
     * between two HiF8 values: the output cast needs no tie rule) */
    const orc_format *fin = hif8_fmt(J->hif8_flags), *fout = &F_HIF8;
    if (J->mode == ORC_EXP2_E4M3) { fin = &F_E4M3; fout = &F_E4M3; }
    if (J->mode == ORC_EXP2_E5M2) { fin = &F_E5M2; fout = &F_E5M2; }
    if (J->mode == ORC_EXP2_E4M3xE5M2) { fin = &F_E4M3; fout = &F_E5M2; }
    /* the decisions whose margin is reported: the HiF8 roundings of the Exp2
     * HiF8 setup, and with pv_bf16 the bf16 roundings of P in Default */
    const int hif8_dec = (J->mode == ORC_EXP2_HIF8);
    float m = -INFINITY, d = 0.0f;
    double eps_m = 0.0;                                                  /* error bound of m, in S units */
    double mg = INFINITY;
    float* ot = (float*)W->pv;                                           /* fp32 O~ */
    for (int i = 0; i < D; ++i) ot[i] = 0.0f;

    for (int j = 0; j < nblk; ++j) {
        const int c0 = j * blk;
        const int c1 = (c0 + blk <= kmax + 1) ? c0 + blk : kmax + 1;
        const int nc = c1 - c0;
        float rowmax = -INFINITY;
        double eps_rowmax = 0.0;
        row_scores(J, qr, kb + (int64_t)c0 * D, nc - 1, given ? given + c0 : NULL, 0, W->acc,
                   want_margin ? W->eps : NULL);
        for (int c = 0; c < nc; ++c) {
            float s = (float)W->acc[c] * J->c32;                         /* S = fl32(fl32(q.k) * c) */
            if (J->mode == ORC_NAIVE_E2E) s = (float)fmt_round(fin, s, 1);       /* scores cast first */
            W->acc[c] = s;
            if (s > rowmax) { rowmax = s; eps_rowmax = want_margin ? W->eps[c] : 0.0; }
        }
        const float m_new = m > rowmax ? m : rowmax;                     /* m^(j) */
        const double eps_new = m > rowmax ? eps_m : eps_rowmax;
        float alpha;
        if (m == -INFINITY) alpha = 0.0f;
        else if (J->mode == ORC_DEFAULT) alpha = exp2f(m - m_new);
        else {
            const float x = m - m_new;
            alpha = (float)fmt_round(fout, exp2(fmt_round(fin, (double)x, 1)), 1);
            if (want_margin && hif8_dec && m_new != m) {
                const double dist = hif8_boundary_distance((double)x) / (eps_m + eps_new);
                if (dist < mg) mg = dist;
            }
        }
        float rowsum = 0.0f;
        d *= alpha;
        for (int i = 0; i < D; ++i) ot[i] *= alpha;
        for (int c = 0; c < nc; ++c) {
            float x = (float)W->acc[c] - m_new;
            float p;
            if (J->mode == ORC_DEFAULT) p = exp2f(x);
            else {
                p = (float)fmt_round(fout, exp2(fmt_round(fin, (double)x, 1)), 1);
                /* a score carrying weight >= 2^-12 of the block maximum's whose
                 * rounding sits near a boundary */
                if (want_margin && hif8_dec && x > -12.0f && W->acc[c] != m_new) {
                    const double dist = hif8_boundary_distance((double)x) / (W->eps[c] + eps_new);
                    if (dist < mg) mg = dist;
                }
            }
            /* with pv_bf16, the bf16 rounding of a weighted P is a decision too:
             * its distance to the nearest bf16 midpoint against the change of
             * P that the score error bounds allow (and a few ulps of exp2) */
            if (want_margin && J->pv_bf16 && J->mode == ORC_DEFAULT && x > -12.0f && p > 0.0f) {
                uint32_t u;
                memcpy(&u, &p, 4);
                const uint32_t mu = (u & 0xFFFF0000u) | 0x8000u;
                float mid;
                memcpy(&mid, &mu, 4);
                const double dp = (double)p * (M_LN2 * (W->eps[c] + eps_new) + ldexp(1.0, -21));
                const double dist = fabs((double)p - (double)mid) / dp;
                if (dist < mg) mg = dist;
            }
            rowsum += p;
            const float pv = J->pv_bf16 ? round_bf16(p) : p;
            const uint16_t* vr = vb + (int64_t)(c0 + c) * D;
            for (int i = 0; i < D; ++i) ot[i] += pv * (float)bf16_to_double(vr[i]);
        }
        d += rowsum;
        m = m_new;
        eps_m = eps_new;
        if (refs_out) refs_out[j] = (double)m;
    }
    if (margin_out) *margin_out = mg;
    if (nblk == 0) {
        for (int i = 0; i < D; ++i) o[i] = 0.0;
        *lse = -INFINITY;
    } else {
        for (int i = 0; i < D; ++i) o[i] = (double)(ot[i] / d);
        *lse = M_LN2 * ((double)m + log2((double)d));
    }
}

/* eq. (1) in fp64: O = softmax(Q K^T / sqrt(d)) V (scale from c64 when overridden) */
static void row_exact(const attn_job* J, int b, int h, int r, row_scratch* W, double* o, double* lse)
{
    const int D = J->D;
    const int g = h / (J->Hq / J->Hkv);
    const uint16_t* qr = J->q + (((int64_t)b * J->Hq + h) * J->Sq + r) * D;
    const uint16_t* kb = J->k + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const uint16_t* vb = J->v + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const int kmax = last_visible_key(J, r);
    const double scale = J->c64 * M_LN2;                                 /* natural units */
    if (kmax < 0) {
        for (int i = 0; i < D; ++i) o[i] = 0.0;
        *lse = -INFINITY;
        return;
    }
    double smax = -INFINITY;
    for (int c = 0; c <= kmax; ++c) {
        double s = dot64(qr, kb + (int64_t)c * D, D) * scale;
        W->acc[c] = s;
        if (s > smax) smax = s;
    }
    double z = 0.0;
    for (int i = 0; i < D; ++i) W->ot[i] = 0.0;
    for (int c = 0; c <= kmax; ++c) {
        double w = exp(W->acc[c] - smax);
        z += w;
        const uint16_t* vr = vb + (int64_t)c * D;
        for (int i = 0; i < D; ++i) W->ot[i] += w * bf16_to_double(vr[i]);
    }
    for (int i = 0; i < D; ++i) o[i] = W->ot[i] / z;
    *lse = smax + log(z);
}

typedef struct { attn_job* J; int which; } attn_ctx;   /* which: 0 modes, 1 exact */

static void attn_range(void* p, int64_t i0, int64_t i1)
{
    attn_ctx* C = (attn_ctx*)p;
    attn_job* J = C->J;
    const int D = J->D;
    row_scratch W;
    const size_t nkeys = (size_t)(J->Sk > J->block ? J->Sk : J->block) + 1;
    const size_t nblk = (size_t)(J->Sk / J->block) + 2;
    W.acc = (double*)malloc(sizeof(double) * nkeys);
    W.eps = (double*)malloc(sizeof(double) * nkeys);
    W.ot = (double*)malloc(sizeof(double) * D);
    W.pv = (double*)malloc(sizeof(double) * D);
    W.ref = (double*)malloc(sizeof(double) * nblk);
    W.bmargin = (double*)malloc(sizeof(double) * nblk);
    for (int64_t i = i0; i < i1; ++i) {
        int64_t g = J->rows[i];
        int r = (int)(g % J->Sq);
        int h = (int)((g / J->Sq) % J->Hq);
        int b = (int)(g / ((int64_t)J->Sq * J->Hq));
        double* o = J->o + i * D;
        double* lse = J->lse + i;
        const float* given = J->acc_in ? J->acc_in + i * J->ld_acc : NULL;
        double* refs = J->ref_out ? J->ref_out + i * J->ld_ref : NULL;
        double* mg = J->margin ? J->margin + i : NULL;
        if (C->which) row_exact(J, b, h, r, &W, o, lse);
        else if (J->mode == ORC_E2E_HIF8 || J->mode == ORC_E2E_EXACT)
            row_alg1(J, b, h, r, &W, given, o, lse, J->nrestart ? J->nrestart + i : NULL, mg, refs);
        else row_eq2(J, b, h, r, &W, given, o, lse, mg, refs);
    }
    free(W.acc); free(W.eps); free(W.ot); free(W.pv); free(W.ref); free(W.bmargin);
}

static int attn_check(int B, int Hq, int Hkv, int Sq, int Sk, int D, int block)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Sq < 0 || Sk < 0 || D <= 0 || block <= 0) return 1;
    if (Hq % Hkv) return 1;
    return 0;
}

/* Shared set-up of the attention entry points. */
static void job_init(attn_job* J, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                     int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                     int mode, int lambda, int n_b0, int literal_else, double scale_log2,
                     const int64_t* rows, double* o, double* lse, int32_t* nrestart, double* margin)
{
    memset(J, 0, sizeof(*J));
    J->q = q; J->k = k; J->v = v;
    J->B = B; J->Hq = Hq; J->Hkv = Hkv; J->Sq = Sq; J->Sk = Sk; J->D = D;
    J->causal = causal; J->block = block;
    J->mode = mode; J->lambda = lambda; J->n_b0 = n_b0; J->literal_else = literal_else;
    J->rows = rows; J->o = o; J->lse = lse; J->nrestart = nrestart; J->margin = margin;
    J->hif8_flags = ORC_SAT;
    J->c64 = scale_log2 != 0.0 ? scale_log2 : M_LOG2E / sqrt((double)D);
    J->c32 = (float)J->c64;
    if (mode != ORC_E2E_EXACT) J->c64 = (double)J->c32;
}

/* rows: global query-row indices (b*Hq + h)*Sq + r; outputs o[nrows*D], lse[nrows].
 * scale_log2 = 0 selects log2(e)/sqrt(D).  margin (nullable): per-row decision
 * margin (see row_alg1).  tie_even: the 8-bit casts of T (Alg. 1) and x (Exp2
 * HiF8) round ties to even.  acc_in (nullable): the high-precision dot
 * products of requested row i at acc_in[i*ld_acc + c] for every key c the row
 * sees (another valid S of R15, e.g. a matrix unit's own sums).  ref_out
 * (nullable): per requested row i and visible key block j, the reference at
 * ref_out[i*ld_ref + j] (entries of blocks the row does not see are left as
 * they are).  Returns 0 or 1 (bad arguments). */
int orc_attention_ex(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                     int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                     int mode, int lambda, int n_b0, int literal_else, double scale_log2,
                     const int64_t* rows, int64_t nrows, double* o, double* lse, int32_t* nrestart,
                     double* margin, int nthreads, int pv_bf16, int tie_even,
                     const float* acc_in, int64_t ld_acc, double* ref_out, int64_t ld_ref)
{
    if (attn_check(B, Hq, Hkv, Sq, Sk, D, block) || mode < 0 || mode > 7) return 1;
    if ((acc_in && ld_acc < Sk) || (ref_out && ld_ref < (Sk + block - 1) / block)) return 1;
    attn_job J;
    job_init(&J, q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, mode, lambda, n_b0, literal_else,
             scale_log2, rows, o, lse, nrestart, margin);
    J.pv_bf16 = pv_bf16;
    J.hif8_flags = ORC_SAT | (tie_even ? ORC_EVEN : 0);
    J.acc_in = acc_in; J.ld_acc = ld_acc; J.ref_out = ref_out; J.ld_ref = ld_ref;
    attn_ctx C = { &J, 0 };
    parallel_for(nrows, nthreads, 1, attn_range, &C);
    return 0;
}

int orc_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                  int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                  int mode, int lambda, int n_b0, int literal_else, double scale_log2,
                  const int64_t* rows, int64_t nrows, double* o, double* lse, int32_t* nrestart,
                  int nthreads)
{
    return orc_attention_ex(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, mode, lambda, n_b0,
                            literal_else, scale_log2, rows, nrows, o, lse, nrestart, NULL, nthreads, 0, 0,
                            NULL, 0, NULL, 0);
}

/* ------------------------------------------------------------------------ */
/* Alg. 1 with the restart decision taken per tile of query rows             */
/* ------------------------------------------------------------------------ */

/* The paper decides a restart per tile: the tile of query rows restarts when
 * the maximum entry of rowmax(T) over its rows exceeds lambda (Sec. 3.2,
 * Alg. 1), and the restart rate is counted per tile (Sec. 4.3, Table 4).  A
 * tile here is restart_rows consecutive query positions of one (batch,
 * head); a B0 block forces the whole tile.  B0 is the first n_b0 key blocks
 * and, with b0_last, also the last key block each row sees (the diagonal
 * block under a causal mask; the text names the first and the last tiles as
 * the critical ones).  Rows that see no key of a block take no part in its
 * decision.  On a restart every row of the tile takes the high-precision
 * path of Alg. 1 with its own row maximum; otherwise every row takes the
 * 8-bit path with its own m.  Counters: B1 tile-blocks (a block that some
 * row of the tile sees and that is in B0 for none of them) visited and
 * restarted, the same for every row of the tile.  The margin of each row is
 * the smallest decision margin over its whole tile, since any of them can
 * move the shared decision. */
typedef struct {
    int R;                                  /* rows of the tile */
    double **acc, **eps, **ot, **pv, **ref; /* per row: [keys], [keys], [D], [D], [blocks] */
    double *m, *d, *tmax, *amax, *eps_blk, *mg;
    int *kmax, *nblk;
} tile_scratch;

static void tile_alg1(const attn_job* J, int b0_last, int b, int h, int r0, int nr, tile_scratch* T,
                      const float* const* given, double* o, double* lse, int32_t* nrs, int32_t* nvis,
                      double* margin)
{
    const int D = J->D, blk = J->block;
    const int g = h / (J->Hq / J->Hkv);
    const uint16_t* kb = J->k + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const uint16_t* vb = J->v + ((int64_t)b * J->Hkv + g) * (int64_t)J->Sk * D;
    const int exact = (J->mode == ORC_E2E_EXACT);
    int nblk_t = 0;
    for (int i = 0; i < nr; ++i) {
        const int r = r0 + i;
        const uint16_t* qr = J->q + (((int64_t)b * J->Hq + h) * J->Sq + r) * D;
        T->kmax[i] = last_visible_key(J, r);
        T->nblk[i] = T->kmax[i] < 0 ? 0 : T->kmax[i] / blk + 1;
        if (T->nblk[i] > nblk_t) nblk_t = T->nblk[i];
        T->m[i] = -INFINITY;
        T->d[i] = 0.0;
        T->mg[i] = INFINITY;
        for (int x = 0; x < D; ++x) T->ot[i][x] = 0.0;
        row_scores(J, qr, kb, T->kmax[i], given ? given[i] : NULL, exact, T->acc[i], margin ? T->eps[i] : NULL);
    }
    int32_t t_restart = 0, t_visit = 0;
    double tile_mg = INFINITY;
    for (int j = 0; j < nblk_t; ++j) {
        /* the tile's decision: any visible row in B0, or any visible row whose
         * 8-bit rowmax(T) (at its own m) exceeds lambda */
        int any_vis = 0, any_b0 = 0, restart = 0;
        for (int i = 0; i < nr; ++i) {
            if (j >= T->nblk[i]) continue;
            any_vis = 1;
            const int c0 = j * blk, c1 = (c0 + blk <= T->kmax[i] + 1) ? c0 + blk : T->kmax[i] + 1;
            double amax = -INFINITY, eb = 0.0, tmax = -INFINITY;
            for (int c = c0; c < c1; ++c) {
                if (T->acc[i][c] > amax) amax = T->acc[i][c];
                if (margin && T->eps[i][c] > eb) eb = T->eps[i][c];
                double t;
                if (exact) t = T->acc[i][c] * J->c64 - T->m[i];
                else t = orc_hif8_round((double)fmaf((float)T->acc[i][c], J->c32, (float)(-T->m[i])), J->hif8_flags);
                if (t > tmax) tmax = t;
            }
            T->amax[i] = amax;
            T->eps_blk[i] = eb;
            T->tmax[i] = tmax;
            const int in_b0 = j < J->n_b0 || (b0_last && j == T->nblk[i] - 1);
            if (in_b0) {
                any_b0 = 1;
                restart = 1;
            } else {
                if (ceil(tmax) > (double)J->lambda) restart = 1;
                if (margin && T->m[i] != -INFINITY) {
                    double dist = hif8_boundary_distance(amax * J->c64 - T->m[i]) / eb;
                    if (dist < tile_mg) tile_mg = dist;
                }
            }
        }
        if (!any_vis) continue;
        if (!any_b0) {
            ++t_visit;
            if (restart) ++t_restart;
        }
        for (int i = 0; i < nr; ++i) {
            if (j >= T->nblk[i]) continue;
            const int c0 = j * blk, c1 = (c0 + blk <= T->kmax[i] + 1) ? c0 + blk : T->kmax[i] + 1;
            const double m = T->m[i];
            double m_new, ref;
            if (restart) {
                double M = -INFINITY;
                for (int c = c0; c < c1; ++c) {
                    double sv = exact ? T->acc[i][c] * J->c64 : (double)((float)T->acc[i][c] * J->c32);
                    if (sv > M) M = sv;
                }
                m_new = fmax(m, ceil(M));
                ref = m_new;
                if (margin) {
                    double dist = integer_distance(T->amax[i] * J->c64) / T->eps_blk[i];
                    if (dist < tile_mg) tile_mg = dist;
                }
            } else {
                m_new = m + fmax(0.0, ceil(T->tmax[i]));
                ref = m;
            }
            double rowsum = 0.0;
            for (int x = 0; x < D; ++x) T->pv[i][x] = 0.0;
            for (int c = c0; c < c1; ++c) {
                double p;
                if (exact) p = exp2(T->acc[i][c] * J->c64 - ref);
                else p = e8_hif8(orc_hif8_round((double)fmaf((float)T->acc[i][c], J->c32, (float)(-ref)), J->hif8_flags));
                if (p == 0.0) continue;
                rowsum += p;
                const uint16_t* vr = vb + (int64_t)c * D;
                for (int x = 0; x < D; ++x) T->pv[i][x] += p * bf16_to_double(vr[x]);
            }
            const double alpha = (m == -INFINITY) ? 0.0 : exp2(m - m_new);
            const double beta = (J->literal_else && !restart) ? 1.0 : exp2(ref - m_new);
            T->d[i] = alpha * T->d[i] + beta * rowsum;
            for (int x = 0; x < D; ++x) T->ot[i][x] = alpha * T->ot[i][x] + beta * T->pv[i][x];
            T->m[i] = m_new;
            T->ref[i][j] = ref;
        }
    }
    if (margin && !exact) {
        /* the HiF8 rounding of every T with weight >= 2^-12 of its row's maximum */
        for (int i = 0; i < nr; ++i) {
            for (int j = 0; j < T->nblk[i]; ++j) {
                const int c0 = j * blk, c1 = (c0 + blk <= T->kmax[i] + 1) ? c0 + blk : T->kmax[i] + 1;
                for (int c = c0; c < c1; ++c) {
                    double x = T->acc[i][c] * J->c64 - T->ref[i][j];
                    double p = e8_hif8(orc_hif8_round((double)fmaf((float)T->acc[i][c], J->c32,
                                                                   (float)(-T->ref[i][j])), J->hif8_flags));
                    if (ldexp(p, (int)(T->ref[i][j] - T->m[i])) < 1.0 / 4096.0) continue;
                    double dist = hif8_boundary_distance(x) / T->eps[i][c];
                    if (dist < tile_mg) tile_mg = dist;
                }
            }
        }
    }
    for (int i = 0; i < nr; ++i) {
        if (T->nblk[i] == 0) {
            for (int x = 0; x < D; ++x) o[(int64_t)i * D + x] = 0.0;
            lse[i] = -INFINITY;
        } else {
            for (int x = 0; x < D; ++x) o[(int64_t)i * D + x] = T->ot[i][x] / T->d[i];
            lse[i] = M_LN2 * (T->m[i] + log2(T->d[i]));
        }
        nrs[i] = t_restart;
        nvis[i] = t_visit;
        if (margin) margin[i] = exact ? INFINITY : tile_mg;
    }
}

typedef struct {
    attn_job* J;
    int R, b0_last;
    const int64_t* tiles;       /* unique tile keys (b*Hq + h)*ntq + t, ascending */
    const int64_t* first;       /* [ntiles+1] ranges into order[] */
    const int64_t* order;       /* requested-row indices sorted by tile */
    int32_t* nvisit;
} tiles_ctx;

static void tiles_range(void* p, int64_t t0, int64_t t1)
{
    tiles_ctx* C = (tiles_ctx*)p;
    attn_job* J = C->J;
    const int D = J->D, R = C->R;
    const int64_t ntq = (J->Sq + R - 1) / R;
    const size_t nkeys = (size_t)(J->Sk > J->block ? J->Sk : J->block) + 1;
    const size_t nblk = (size_t)(J->Sk / J->block) + 2;
    tile_scratch T;
    T.R = R;
    T.acc = (double**)malloc(sizeof(double*) * R); T.eps = (double**)malloc(sizeof(double*) * R);
    T.ot = (double**)malloc(sizeof(double*) * R); T.pv = (double**)malloc(sizeof(double*) * R);
    T.ref = (double**)malloc(sizeof(double*) * R);
    for (int i = 0; i < R; ++i) {
        T.acc[i] = (double*)malloc(sizeof(double) * nkeys); T.eps[i] = (double*)malloc(sizeof(double) * nkeys);
        T.ot[i] = (double*)malloc(sizeof(double) * D); T.pv[i] = (double*)malloc(sizeof(double) * D);
        T.ref[i] = (double*)malloc(sizeof(double) * nblk);
    }
    T.m = (double*)malloc(sizeof(double) * R); T.d = (double*)malloc(sizeof(double) * R);
    T.tmax = (double*)malloc(sizeof(double) * R); T.amax = (double*)malloc(sizeof(double) * R);
    T.eps_blk = (double*)malloc(sizeof(double) * R); T.mg = (double*)malloc(sizeof(double) * R);
    T.kmax = (int*)malloc(sizeof(int) * R); T.nblk = (int*)malloc(sizeof(int) * R);
    double* o = (double*)malloc(sizeof(double) * (size_t)R * D);
    double* lse = (double*)malloc(sizeof(double) * R);
    double* mg = (double*)malloc(sizeof(double) * R);
    int32_t* nrs = (int32_t*)malloc(sizeof(int32_t) * R);
    int32_t* nvs = (int32_t*)malloc(sizeof(int32_t) * R);
    const float** given = (const float**)malloc(sizeof(float*) * R);
    for (int64_t t = t0; t < t1; ++t) {
        const int64_t key = C->tiles[t];
        const int tq = (int)(key % ntq);
        const int h = (int)((key / ntq) % J->Hq);
        const int b = (int)(key / (ntq * J->Hq));
        const int r0 = tq * R;
        const int nr = (r0 + R <= J->Sq) ? R : J->Sq - r0;
        if (J->acc_in) {
            /* supplied dot products: every row of the tile takes part in its
             * decisions, so every row of the tile must have been requested */
            for (int i = 0; i < nr; ++i) given[i] = NULL;
            for (int64_t e = C->first[t]; e < C->first[t + 1]; ++e) {
                const int64_t i = C->order[e];
                given[(int)(J->rows[i] % J->Sq) - r0] = J->acc_in + i * J->ld_acc;
            }
            int missing = 0;
            for (int i = 0; i < nr; ++i) missing |= given[i] == NULL;
            if (missing) { __atomic_store_n(&J->err, 1, __ATOMIC_RELAXED); continue; }
        }
        tile_alg1(J, C->b0_last, b, h, r0, nr, &T, J->acc_in ? given : NULL, o, lse, nrs, nvs,
                  J->margin ? mg : NULL);
        for (int64_t e = C->first[t]; e < C->first[t + 1]; ++e) {
            const int64_t i = C->order[e];
            const int r = (int)(J->rows[i] % J->Sq) - r0;
            for (int x = 0; x < D; ++x) J->o[i * D + x] = o[(int64_t)r * D + x];
            J->lse[i] = lse[r];
            if (J->nrestart) J->nrestart[i] = nrs[r];
            if (C->nvisit) C->nvisit[i] = nvs[r];
            if (J->margin) J->margin[i] = mg[r];
            if (J->ref_out)
                for (int j = 0; j < T.nblk[r]; ++j) J->ref_out[i * J->ld_ref + j] = T.ref[r][j];
        }
    }
    free(given);
    for (int i = 0; i < R; ++i) { free(T.acc[i]); free(T.eps[i]); free(T.ot[i]); free(T.pv[i]); free(T.ref[i]); }
    free(T.acc); free(T.eps); free(T.ot); free(T.pv); free(T.ref);
    free(T.m); free(T.d); free(T.tmax); free(T.amax); free(T.eps_blk); free(T.mg); free(T.kmax); free(T.nblk);
    free(o); free(lse); free(mg); free(nrs); free(nvs);
}

static int64_t* g_sort_keys;            /* qsort context (single-threaded section) */
static int cmp_by_key(const void* a, const void* b)
{
    const int64_t ka = g_sort_keys[*(const int64_t*)a], kb = g_sort_keys[*(const int64_t*)b];
    return ka < kb ? -1 : (ka > kb ? 1 : 0);
}

/* Alg. 1 with tile-level restart (restart_rows >= 1 query positions per
 * tile) and optionally B0 = {first n_b0 blocks, each row's last block}.
 * Modes ORC_E2E_HIF8 and ORC_E2E_EXACT.  Besides the outputs of
 * orc_attention_ex: nvisit (nullable), the visited B1 tile-blocks of each
 * requested row's tile; nrestart holds the restarted ones.  Returns 0 or 1. */
int orc_attention_tiles(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                        int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                        int mode, int lambda, int n_b0, int b0_last, int restart_rows, int literal_else,
                        double scale_log2, const int64_t* rows, int64_t nrows, double* o, double* lse,
                        int32_t* nrestart, int32_t* nvisit, double* margin, int nthreads, int tie_even,
                        const float* acc_in, int64_t ld_acc, double* ref_out, int64_t ld_ref)
{
    if (attn_check(B, Hq, Hkv, Sq, Sk, D, block)) return 1;
    if ((mode != ORC_E2E_HIF8 && mode != ORC_E2E_EXACT) || restart_rows < 1 || n_b0 < 0) return 1;
    if ((acc_in && ld_acc < Sk) || (ref_out && ld_ref < (Sk + block - 1) / block)) return 1;
    attn_job J;
    job_init(&J, q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, mode, lambda, n_b0, literal_else,
             scale_log2, rows, o, lse, nrestart, margin);
    J.hif8_flags = ORC_SAT | (tie_even ? ORC_EVEN : 0);
    J.acc_in = acc_in; J.ld_acc = ld_acc; J.ref_out = ref_out; J.ld_ref = ld_ref;
    if (nrows == 0) return 0;
    const int R = restart_rows;
    const int64_t ntq = (Sq + R - 1) / R;
    int64_t* key = (int64_t*)malloc(sizeof(int64_t) * nrows);
    int64_t* order = (int64_t*)malloc(sizeof(int64_t) * nrows);
    int64_t* tiles = (int64_t*)malloc(sizeof(int64_t) * nrows);
    int64_t* first = (int64_t*)malloc(sizeof(int64_t) * (nrows + 1));
    for (int64_t i = 0; i < nrows; ++i) {
        const int64_t g = rows[i];
        key[i] = (g / Sq) * ntq + (g % Sq) / R;
        order[i] = i;
    }
    g_sort_keys = key;
    qsort(order, (size_t)nrows, sizeof(int64_t), cmp_by_key);
    int64_t nt = 0;
    for (int64_t e = 0; e < nrows; ++e) {
        if (e == 0 || key[order[e]] != key[order[e - 1]]) {
            tiles[nt] = key[order[e]];
            first[nt] = e;
            ++nt;
        }
    }
    first[nt] = nrows;
    tiles_ctx C = { &J, R, b0_last ? 1 : 0, tiles, first, order, nvisit };
    parallel_for(nt, nthreads, 1, tiles_range, &C);
    free(key); free(order); free(tiles); free(first);
    return J.err ? 1 : 0;
}

int orc_exact_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                        int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                        double scale_log2, const int64_t* rows, int64_t nrows,
                        double* o, double* lse, int nthreads)
{
    if (attn_check(B, Hq, Hkv, Sq, Sk, D, 1)) return 1;
    attn_job J;
    job_init(&J, q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, 1, ORC_E2E_EXACT, 0, 0, 0, scale_log2, rows, o, lse,
             NULL, NULL);
    attn_ctx C = { &J, 1 };
    parallel_for(nrows, nthreads, 1, attn_range, &C);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* The vector-side steps of Alg. 1 on given scores                           */
/* ------------------------------------------------------------------------ */

typedef struct {
    const float* s; int64_t cols, ld; int block, lambda, n_b0;
    uint8_t* codes; int32_t* ref_shift; double *m_out, *d_out; uint8_t* restarted;
} sb_job;

static void sb_range(void* p, int64_t i0, int64_t i1)
{
    sb_job* J = (sb_job*)p;
    const int64_t nblk = (J->cols + J->block - 1) / J->block;
    double* refs = (double*)malloc(sizeof(double) * (size_t)(nblk ? nblk : 1));
    for (int64_t r = i0; r < i1; ++r) {
        const float* S = J->s + r * J->ld;
        uint8_t* code = J->codes + r * J->cols;
        double m = -INFINITY, d = 0.0;
        for (int64_t j = 0; j < nblk; ++j) {
            const int64_t c0 = j * J->block;
            const int64_t c1 = c0 + J->block < J->cols ? c0 + J->block : J->cols;
            int restart;
            double m_new = m, ref = m;
            if (j < J->n_b0) restart = 1;
            else {
                double tmax = -INFINITY;
                for (int64_t c = c0; c < c1; ++c) {
                    if (S[c] == -INFINITY) continue;                     /* masked score */
                    double t = orc_hif8_round((double)(S[c] - (float)m), 1);
                    if (t > tmax) tmax = t;
                }
                restart = ceil(tmax) > (double)J->lambda;
                if (!restart) m_new = m + fmax(0.0, ceil(tmax));
            }
            if (restart) {
                double M = -INFINITY;
                for (int64_t c = c0; c < c1; ++c) if ((double)S[c] > M) M = S[c];
                m_new = fmax(m, ceil(M));
                ref = m_new;
            }
            double rowsum = 0.0;
            for (int64_t c = c0; c < c1; ++c) {
                double p = 0.0;
                if (ref != -INFINITY && S[c] != -INFINITY)
                    p = e8_hif8(orc_hif8_round((double)(S[c] - (float)ref), 1));
                code[c] = (uint8_t)fmt_encode(&F_HIF8, p, 1);
                rowsum += p;
            }
            const double alpha = (m == -INFINITY) ? 0.0 : exp2(m - m_new);
            const double beta = (ref == -INFINITY) ? 0.0 : exp2(ref - m_new);
            d = alpha * d + beta * rowsum;
            m = m_new;
            refs[j] = ref;
            if (J->restarted) J->restarted[r * nblk + j] = (uint8_t)restart;
        }
        for (int64_t j = 0; j < nblk; ++j)
            J->ref_shift[r * nblk + j] = (refs[j] == -INFINITY) ? INT32_MIN : (int32_t)(refs[j] - m);
        J->m_out[r] = m;
        J->d_out[r] = d;
    }
    free(refs);
}

/* s: rows x cols fp32 scores in log2 units (row stride ld); -inf marks a
 * masked score.  Outputs: codes[rows*cols] (HiF8 code of P relative to its
 * block's reference), ref_shift[rows*nblk] = ref_j - m_final (INT32_MIN for a
 * block with no finite reference), m_final, d_final, restarted[rows*nblk]. */
int orc_softmax_block(const float* s, int64_t rows, int64_t cols, int64_t ld, int block,
                      int lambda, int n_b0, uint8_t* codes, int32_t* ref_shift,
                      double* m_final, double* d_final, uint8_t* restarted, int nthreads)
{
    if (rows < 0 || cols < 0 || block <= 0 || ld < cols) return 1;
    sb_job J = { s, cols, ld, block, lambda, n_b0, codes, ref_shift, m_final, d_final, restarted };
    parallel_for(rows, nthreads, 8, sb_range, &J);
    return 0;
}
