/*
 * BAPS attention on AMD Instinct MI355X (gfx950): C ABI.
 *
 * The library computes the attention forward pass of "BAPS: A Fine-Grained
 * Low-Precision Scheme for Softmax in Attention via Block-Aware Precision
 * reScaling" (arXiv 2602.02071): attention as stated in eq. (1), evaluated
 * blockwise by the base-2 online softmax of eq. (2) reorganised as Alg. 1
 * ("E2E HiF8"): the score minus an integer reference maximum is cast to the
 * 8-bit HiF8 format (eq. 3), its power of two is taken in HiF8 (App. A,
 * Alg. 2), and the running denominator and output are rescaled by exact
 * integer powers of two (Sec. 3.3).
 *
 * Conventions for every entry point:
 *  - Tensor pointers are DEVICE pointers owned by the caller; the library
 *    never allocates, frees or retains them.  Inputs are not modified;
 *    outputs are fully overwritten.
 *  - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL is the default stream) and does not synchronise, except the very
 *    first call on a device, which uploads the library's read-only 32 KiB
 *    score table to that device synchronously (baps_init does it up front).
 *  - Layouts are contiguous row-major: q, o [B][Hq][Sq][D]; k, v
 *    [B][Hkv][Sk][D]; lse [B][Hq][Sq].  bf16 tensors are passed as raw
 *    16-bit patterns.
 *  - Return value: BAPS_OK (0), BAPS_INVALID_ARGUMENT (1: a null pointer
 *    where one is required, a negative size, Hq not a multiple of Hkv),
 *    BAPS_UNSUPPORTED (2: a head dimension or block size without a kernel),
 *    BAPS_HIP_ERROR (3: the HIP runtime reported an error at launch).
 *    baps_status_string() names a status.  No exception crosses the ABI.
 *  - Empty work (B, Hq or Sq zero; n or rows zero) returns BAPS_OK and
 *    touches nothing.
 */
#ifndef BAPS_H
#define BAPS_H

#ifdef __cplusplus
extern "C" {
#endif

#define BAPS_OK 0
#define BAPS_INVALID_ARGUMENT 1
#define BAPS_UNSUPPORTED 2
#define BAPS_HIP_ERROR 3

#define BAPS_HIF8_SATURATE 1
#define BAPS_HIF8_TIES_EVEN 2

/*
 * Fused BAPS attention forward, canonical setup ("E2E HiF8", Sec. 4.1):
 * restart threshold lambda = 1, B0 = the first key block, Alg. 1 per query
 * row, HiF8 rounding to nearest with ties away from zero, saturating.
 *
 * q [B,Hq,Sq,D], k/v [B,Hkv,Sk,D] bf16; o [B,Hq,Sq,D] fp32; lse [B,Hq,Sq]
 * fp32, natural log of the softmax denominator of the scores q.k/sqrt(D),
 * as the HiF8 pipeline estimates it: ln2 * (m + log2 d); may be NULL.
 * Query head h reads key/value head h / (Hq/Hkv).  causal != 0 masks key c
 * from query row r when c > r + Sk - Sq (bottom-right aligned); a row that
 * sees no key gets o = 0 and lse = -inf.  block is the key tile of Alg. 1
 * (the unit of the restart test and of the integer maximum).
 * Supported: D in {64, 128}; block in {32, 64, 128}.  Sk may be 0.
 */
int baps_attention_fwd(const void* q, const void* k, const void* v, float* o, float* lse,
                       int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                       void* stream);

/* Softmax setups (Sec. 4.1, Table 1).  BAPS_MODE_E2E_HIF8 is the proposed
 * workflow (Alg. 1).  The two others follow eq. (2) with the real-valued
 * running maximum m, on the same tiling, for comparison:
 *   BAPS_MODE_DEFAULT    every softmax operation in fp32: P = 2^fl32(S - m),
 *                        rescale 2^(m_old - m); P enters P V rounded to bf16,
 *                        the denominator sums the fp32 P;
 *   BAPS_MODE_EXP2_HIF8  the exp2 on 8-bit input, rounded to 8 bits:
 *                        P = HiF8(2^HiF8(fl32(S - m))), likewise the rescale
 *                        factor; S = fl32(fl32(q.k) * scale).
 * lambda, n_b0 and restart_counts apply to BAPS_MODE_E2E_HIF8 only. */
#define BAPS_MODE_E2E_HIF8 0
#define BAPS_MODE_DEFAULT 1
#define BAPS_MODE_EXP2_HIF8 2

/* Knobs of Alg. 1 and the paper's ablations (Sec. 4.1, Table 4). */
typedef struct {
    int lambda;                          /* restart threshold (integer, Alg. 1); 1 canonical  */
    int n_b0;                            /* key blocks in B0 (taken first, Alg. 1); 1 canonical */
    float scale_log2;                    /* score scale in log2 units; 0 => log2(e)/sqrt(D)    */
    unsigned long long* restart_counts;  /* device [B*Hq][2]: restarted and visited B1 tile-
                                            blocks (a tile is one query row unless
                                            restart_rows > 1; accumulated with atomics; the
                                            caller zeroes it); NULL to skip                   */
    int mode;                            /* BAPS_MODE_*; anything else is an invalid argument  */
    int restart_rows;                    /* query positions of one head that share the restart
                                            decision (the paper's tile, Sec. 3.2); 0 or 1 per
                                            row (canonical).  E2E setup only; a power of two
                                            with restart_rows * (Hq/Hkv) <= 256 and Hq/Hkv a
                                            power of two <= 32, else BAPS_UNSUPPORTED          */
    int b0_last;                         /* nonzero: B0 also holds each row's last visible key
                                            block (the diagonal block when causal)            */
    unsigned long long* tile_counts;     /* device [B*Hq][ceil(Sq/restart_rows)][2]: restarted
                                            and visited B1 blocks per tile (Table 4's restart
                                            rates); caller-zeroed, NULL to skip               */
    int qk_format;                       /* BAPS_QK_BF16 (0) or BAPS_QK_FP8_E4M3 (1): q and k
                                            hold OCP FP8 E4M3 codes (one byte per element,
                                            rows of D bytes) for the values
                                            q_scale * code and k_scale * code; the scales fold
                                            into the score scale, T = fl32(acc * c' - ref) with
                                            c' = fl32(c * q_scale * k_scale) (Sec. 3.2: T is
                                            computed in the dequantisation).  Not with
                                            restart_rows > 1                                  */
    float q_scale, k_scale;              /* FP8 dequantisation scales (finite, > 0)            */
    int tie_mode;                        /* the 8-bit cast of T (eq. 3): BAPS_TIES_AWAY (0,
                                            canonical) or BAPS_TIES_EVEN (1, E2E setup with
                                            lambda <= 8, restart_rows <= 1 and bf16 Q/K; else
                                            BAPS_UNSUPPORTED); anything else is invalid       */
    int saturate;                        /* nonzero: the 8-bit casts clamp finite overflow to
                                            +-2^15 (canonical); 0: they round it to +-Inf.
                                            Identical results unless an 8-bit P can exceed 2^15,
                                            i.e. lambda >= 16 in the E2E setup, which is
                                            BAPS_UNSUPPORTED with saturate = 0                */
    int out_bf16;                        /* nonzero: o receives bf16 (each element the round-to-
                                            nearest-even bf16 of the fp32 result) in place of
                                            fp32: B*Hq*Sq*D 16-bit values at the same 16-byte
                                            aligned address (the float* is reinterpreted)      */
} baps_params_t;

#define BAPS_QK_BF16 0
#define BAPS_QK_FP8_E4M3 1
#define BAPS_TIES_AWAY 0
#define BAPS_TIES_EVEN 1

/* baps_attention_fwd with explicit knobs; p must not be NULL; scale_log2
 * must be >= 0.  A caller that fills the struct by hand sets saturate = 1 for
 * the canonical cast (0 is accepted and gives the same result below lambda 16). */
int baps_attention_fwd_ex(const void* q, const void* k, const void* v, float* o, float* lse,
                          int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                          const baps_params_t* p, void* stream);

/*
 * Verification entry point: baps_attention_fwd_ex (p may be NULL: canonical
 * knobs) on the one-pass kernels of that call, built with a dump of the
 * high-precision scores S that Alg. 1 computes "in high precision" (R15: the
 * matrix unit's own fp32 sums q.k, before the scale) and of the reference of
 * every key block, for the query rows the caller selects.  O, lse and every
 * other output equal those of baps_attention_fwd_ex on the same arguments
 * (the kernels differ only by the extra stores), so an independent
 * implementation of Alg. 1 run on the dumped S must reproduce O bit for bit
 * in its decisions and up to the order of fp32 additions in its sums.
 *   row_slot [B*Hq*Sq] int32 (device): for query row (b*Hq + h)*Sq + r, -1
 *            or a slot s in [0, nslots); distinct rows take distinct slots;
 *   acc_out  [nslots][Sk] fp32 (device): acc_out[s*Sk + c] = q.k_c for every
 *            key c the row sees (under the causal mask); other entries are
 *            left as they are;
 *   ref_out  [nslots][ceil(Sk/block)] fp32 (device): the reference after
 *            every key block j the row sees (Alg. 1's integer m~ that T is
 *            taken against; the running maximum m in the eq. (2) setups);
 *            other entries are left as they are.
 * The caller owns the buffers and sizes them for its nslots.  Status 1 when
 * row_slot, or acc_out / ref_out with Sk > 0, is NULL.
 */
int baps_attention_fwd_dump(const void* q, const void* k, const void* v, float* o, float* lse,
                            int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                            const baps_params_t* p, const int* row_slot, float* acc_out, float* ref_out,
                            void* stream);

/*
 * Split-key path for few query rows per key/value head (single-sequence or
 * small-batch decode over long contexts: few (batch, key/value head) streams,
 * many keys).  Alg. 1's state after a key block depends on the keys only
 * through the block's row maximum, so the call runs as passes over key
 * splits: raw dot products and block maxima of every split in parallel; then,
 * per split in parallel, a per-row replay of the B0 / restart rule and
 * integer maximum in block order up to the split's last block and P V of the
 * split at those references; last, per row, an exact power-of-two combine.  Every T, P and reference equals baps_attention_fwd_ex's;
 * O and lse differ only by the order of fp32 additions.
 *
 * baps_attention_split_workspace: the workspace bytes the call needs for this
 * shape and these knobs (p may be NULL: canonical knobs); 0 when the shape
 * takes the one-pass kernels (more than 64 flattened rows per key/value head,
 * enough streams to fill the GPU, fewer than 4 key blocks, a setup other
 * than BAPS_MODE_E2E_HIF8, or lambda > 8).
 *
 * baps_attention_fwd_split: baps_attention_fwd_ex (p may be NULL: canonical
 * knobs) with a caller-owned device workspace of at least that many bytes,
 * 256-byte aligned, contents undefined on entry and on return; NULL and 0 are
 * fine when the size is 0.  Status 1 when a needed workspace is missing,
 * short or misaligned.  Asynchronous on the stream; the workspace must not be
 * reused before the call completes.
 */
long long baps_attention_split_workspace(int B, int Hq, int Hkv, int Sq, int Sk, int D, int block,
                                         const baps_params_t* p);
int baps_attention_fwd_split(const void* q, const void* k, const void* v, float* o, float* lse,
                             int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                             const baps_params_t* p, void* workspace, long long workspace_bytes,
                             void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * baps_attention_fwd_split with the workspace taken from the library's own
 * static device scratch of BAPS_SPLIT_SCRATCH_BYTES (32 MiB, one copy per
 * device, held until the process ends) instead of a caller's buffer.  The
 * call allocates nothing.  Same arguments, results and kernels as
 * baps_attention_fwd_split; shapes that take the one-pass kernels run them
 * (no scratch).  BAPS_UNSUPPORTED when the shape's workspace
 * (baps_attention_split_workspace) exceeds BAPS_SPLIT_SCRATCH_BYTES.  Every
 * call on a device shares that device's scratch: calls that overlap on one
 * GPU (other streams, other threads) race and must be serialised by the
 * caller; the scratch needs no clearing (its contents are undefined on entry).
 */
#define BAPS_SPLIT_SCRATCH_BYTES (32LL << 20)
int baps_attention_fwd_split_noalloc(const void* q, const void* k, const void* v, float* o, float* lse,
                                     int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, int block,
                                     const baps_params_t* p, void* stream);

/*
 * HiF8 codec (the 8-bit format used by every 8-bit step of the method;
 * Sec. 2, App. A).  hif8_encode: codes[i] = code of the HiF8 value nearest
 * to x[i].  flags: BAPS_HIF8_SATURATE clamps finite overflow to +-2^15 (else
 * values from 1.25*2^15 up become +-Inf); BAPS_HIF8_TIES_EVEN sends a value
 * exactly halfway between two HiF8 values to the one whose significand is
 * even (an even multiple of their spacing: between the last value of a
 * binade and the next power of two, and among the powers of two below
 * 2^-15, that is the upper one; between 0 and 2^-22 it is 0; at the
 * overflow midpoint it is 2^15), else ties go away from zero; no other bit
 * may be set.  +-Inf -> 0x6F/0xEF, NaN -> 0x80, values that round to zero
 * -> 0x00.  hif8_decode: x[i] = value of codes[i] (0x80 -> NaN).
 * n >= 0 elements; any alignment (16-byte aligned buffers stream faster).
 */
int hif8_encode(const float* x, unsigned char* codes, long long n, int flags, void* stream);
int hif8_decode(const unsigned char* codes, float* x, long long n, void* stream);

/*
 * The vector-side steps of Alg. 1 on fp32 score rows already in log2 units
 * (S of eq. 2), one sequential pass over the key blocks of each row:
 * block maximum, B0 / restart rule with threshold lambda, integer running
 * maximum (Sec. 3.3), T = HiF8(S - ref), P = HiF8(2^T), and the running
 * denominator.  s: rows x cols, row stride ld_s >= cols (elements); -inf
 * marks a masked score; scores must be finite or -inf.
 * Outputs (device):
 *   p_codes  [rows, cols]  HiF8 code of P relative to its block's reference
 *   ref_shift[rows, nblk]  ref_j - m_final (<= 0); INT32_MIN for a block
 *                          with no finite reference; nblk = ceil(cols/block)
 *   m_final  [rows]        final integer maximum (-inf for an all-masked row)
 *   d_final  [rows]        final denominator, relative to 2^m_final
 *   restarted[rows, nblk]  1 where the block took the high-precision path
 *                          (B0 or a restart); may be NULL
 * The normalised probability of score c in block j is
 *   decode(p_codes[r,c]) * 2^ref_shift[r,j] / d_final[r].
 * block must be one of 64, 128, 256, 512, 1024.  flags must be 0.
 */
int baps_softmax_block(const float* s, long long rows, long long cols, long long ld_s, int block,
                       int lambda, int n_b0, int flags, unsigned char* p_codes, int* ref_shift,
                       float* m_final, float* d_final, unsigned char* restarted, void* stream);

/* Host copy of the library's 8-bit exp2 table: out_codes[c] = code of
 * HiF8(2^decode(c)) (App. A, Alg. 2, with exp2 in double precision).
 * Needs no GPU. */
int baps_get_exp2_lut(unsigned char out_codes[256]);

/* Uploads the score table to the current device (synchronously).  Optional:
 * the first call of an entry point on a device does it otherwise. */
int baps_init(void);

/* Name of the last HIP runtime error that a call of this library met on the
 * calling thread ("hipSuccess" if none): the detail behind BAPS_HIP_ERROR.
 * Static storage; not cleared by later successful calls. */
const char* baps_last_hip_error(void);

/* Text of a status code (static storage). */
const char* baps_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* BAPS_H */
