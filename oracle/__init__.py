"""CPU oracle for BAPS attention -- TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 implementation of what the BAPS path computes, written
from the paper (arXiv 2602.02071): eq. (1) attention, eq. (2) base-2 online
softmax, eq. (3) offloaded subtraction, Sec. 3.3 integer powers of two,
Alg. 1 (the proposed workflow) and Alg. 2 (App. A, exp2 in HiF8), plus the
HiF8 format the paper cites.  The arithmetic lives in ``baps_oracle.c``
(plain C, compiled with gcc); this module only marshals numpy arrays.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP
library in ``paper_2602_02071_amd``, and that library never imports it.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liborc.so")
SOURCE = os.path.join(_HERE, "baps_oracle.c")

# attention setups (Sec. 4.1 and Table 1 of the paper)
E2E_HIF8 = 0        # Alg. 1, the "E2E HiF8" setup (the canonical BAPS result)
DEFAULT = 1         # eq. (2) with an fp32 softmax ("Default")
EXP2_HIF8 = 2       # eq. (2) with every power of two in HiF8 ("Exp2 HiF8")
NAIVE_E2E = 3       # scores cast to HiF8 before the max subtraction ("Naive E2E")
EXP2_E4M3 = 4
EXP2_E5M2 = 5
EXP2_E4M3xE5M2 = 6
E2E_EXACT = 7       # Alg. 1 control flow with the 8-bit casts removed, fp64 arithmetic

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SOURCE):
        tmp = LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call([
            "gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-ffp-contract=off",
            "-fno-fast-math", "-Wall", "-o", tmp, SOURCE, "-lm", "-lpthread"])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build()
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i64 = ctypes.c_int64
    i32 = ctypes.c_int
    d = ctypes.c_double
    L.orc_hif8_decode.restype = d
    L.orc_hif8_decode.argtypes = [i32]
    L.orc_hif8_encode.restype = i32
    L.orc_hif8_encode.argtypes = [d, i32]
    L.orc_hif8_round.restype = d
    L.orc_hif8_round.argtypes = [d, i32]
    L.orc_e4m3_encode.restype = i32
    L.orc_e4m3_encode.argtypes = [d, i32]
    L.orc_e5m2_encode.restype = i32
    L.orc_e5m2_encode.argtypes = [d, i32]
    L.orc_e4m3_decode.restype = d
    L.orc_e4m3_decode.argtypes = [i32]
    L.orc_e5m2_decode.restype = d
    L.orc_e5m2_decode.argtypes = [i32]
    L.orc_round_fp16.restype = d
    L.orc_round_fp16.argtypes = [d]
    L.orc_default_threads.restype = i32
    L.orc_default_threads.argtypes = []
    L.orc_hif8_encode_f32.restype = None
    L.orc_hif8_encode_f32.argtypes = [P, P, i64, i32, i32]
    L.orc_hif8_check_patterns.restype = i64
    L.orc_hif8_check_patterns.argtypes = [ctypes.c_uint64, i64, P, i32, i32, ctypes.POINTER(i64)]
    L.orc_exp2_table.restype = None
    L.orc_exp2_table.argtypes = [P, i32]
    L.orc_power_product.restype = None
    L.orc_power_product.argtypes = [P, i64, i32, P]
    L.orc_attention.restype = i32
    L.orc_attention.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32,
                                i32, i32, i32, i32, d, P, i64, P, P, P, i32]
    L.orc_attention_ex.restype = i32
    L.orc_attention_ex.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32,
                                   i32, i32, i32, i32, d, P, i64, P, P, P, P, i32, i32, i32, P, i64, P, i64]
    L.orc_attention_tiles.restype = i32
    L.orc_attention_tiles.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32, i32,
                                      i32, i32, i32, i32, i32, i32, d, P, i64, P, P, P, P, P, i32, i32,
                                      P, i64, P, i64]
    L.orc_exact_attention.restype = i32
    L.orc_exact_attention.argtypes = [P, P, P, i32, i32, i32, i32, i32, i32, i32,
                                      d, P, i64, P, P, i32]
    L.orc_softmax_block.restype = i32
    L.orc_softmax_block.argtypes = [P, i64, i64, i64, i32, i32, i32, P, P, P, P, P, i32]
    _lib = L
    return L


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def default_threads() -> int:
    return int(_load().orc_default_threads())


# ---------------------------------------------------------------- HiF8 codec
def hif8_decode(codes) -> np.ndarray:
    """Value of each HiF8 code (NaN / +-Inf for the special codes)."""
    L = _load()
    codes = np.asarray(codes, dtype=np.int64)
    table = np.array([L.orc_hif8_decode(c) for c in range(256)], dtype=np.float64)
    return table[codes]


def _hif8_flags(saturate, ties_even):
    return (1 if saturate else 0) | (2 if ties_even else 0)


def hif8_encode(x, saturate: bool = True, nthreads: int = 0, ties_even: bool = False) -> np.ndarray:
    """Round-to-nearest HiF8 code of each fp32 value (ties away from zero, or
    to even)."""
    L = _load()
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    out = np.empty(x.shape, dtype=np.uint8)
    L.orc_hif8_encode_f32(_ptr(x), _ptr(out), x.size, _hif8_flags(saturate, ties_even), nthreads)
    return out


def hif8_encode_scalar(x: float, saturate: bool = True, ties_even: bool = False) -> int:
    return int(_load().orc_hif8_encode(float(x), _hif8_flags(saturate, ties_even)))


def hif8_round(x, saturate: bool = True, ties_even: bool = False) -> np.ndarray:
    """The value each fp32 input takes after the 8-bit cast."""
    return hif8_decode(hif8_encode(x, saturate, ties_even=ties_even))


def check_patterns(start: int, codes: np.ndarray, saturate: bool = True, nthreads: int = 0,
                   ties_even: bool = False):
    """Compare codes[i] with the oracle's code for fp32 bit pattern start+i.
    Returns (mismatch count, first mismatching index or -1)."""
    L = _load()
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    first = ctypes.c_int64(-1)
    bad = L.orc_hif8_check_patterns(ctypes.c_uint64(start), codes.size, _ptr(codes),
                                    _hif8_flags(saturate, ties_even), nthreads, ctypes.byref(first))
    return int(bad), int(first.value)


def exp2_table(variant: int = 0) -> np.ndarray:
    """code -> code of HiF8(2^x).  variant 0: fp64 exp2, one rounding;
    variant 1: Alg. 2 with its FP16 carrier."""
    out = np.zeros(256, dtype=np.uint8)
    _load().orc_exp2_table(_ptr(out), int(variant))
    return out


def power_product(x, integer: bool) -> np.ndarray:
    """Sec. 3.3 and Fig. 2: log2 of (running product of rescale factors
    2^x_1 ... 2^x_i as the 8-bit pipeline forms them / its ground truth),
    after every step i.  integer=True raises each exponent to an integer
    (ceil, as Alg. 1's integer maximum does) and takes the exact power of
    two; integer=False takes each factor as E8[Q8(x)] (an 8-bit cast of the
    exponent, then of its power of two)."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float64).reshape(-1))
    out = np.empty(x.size, dtype=np.float64)
    _load().orc_power_product(_ptr(x), x.size, int(bool(integer)), _ptr(out))
    return out


def round_fp16(y: float) -> float:
    return float(_load().orc_round_fp16(float(y)))


def e4m3_encode(x: float, saturate: bool = True) -> int:
    """OCP FP8 E4M3 code of x: nearest value, ties to even; beyond the
    largest finite value 448 the NaN code unless saturate."""
    return int(_load().orc_e4m3_encode(float(x), int(bool(saturate))))


def e5m2_encode(x: float, saturate: bool = True) -> int:
    """OCP FP8 E5M2 code of x: nearest value, ties to even; overflow to
    +-Inf unless saturate."""
    return int(_load().orc_e5m2_encode(float(x), int(bool(saturate))))


def e4m3_decode(c: int) -> float:
    return float(_load().orc_e4m3_decode(int(c)))


def e5m2_decode(c: int) -> float:
    return float(_load().orc_e5m2_decode(int(c)))


# ---------------------------------------------------------------- attention
def _bits(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("q/k/v must be bf16 bit patterns (np.uint16)")
    return a


def _rows(rows, total):
    if rows is None:
        return np.arange(total, dtype=np.int64)
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    if rows.size and (rows.min() < 0 or rows.max() >= total):
        raise ValueError("row index out of range")
    return rows


def attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, mode=E2E_HIF8, lam=1, n_b0=1,
              literal_else=False, scale_log2=0.0, rows=None, nthreads=0, margin=False, pv_bf16=False,
              restart_rows=1, b0_last=False, visits=False, tie_even=False, acc=None, refs=False):
    """Attention rows in one of the paper's setups.

    q: [B,Hq,Sq,D], k/v: [B,Hkv,Sk,D] bf16 bit patterns.  rows: global row
    indices (b*Hq + h)*Sq + r (all rows when None).  Returns (o[n,D] fp64,
    lse[n] fp64, restarts[n] int32 -- restarted B1 blocks per row), plus the
    per-row decision margin when margin=True: how far the row's 8-bit
    decisions sit from a rounding boundary, in units of the fp32 dot-product
    accumulation error bound (>= 1: every valid high-precision S yields this
    result).  pv_bf16 (the setups of eq. (2) only): P enters the P V product
    rounded to bf16, the input precision of a matrix unit, while the
    denominator sums P as computed.  tie_even: the 8-bit casts of the
    softmax round ties to even (else away from zero).

    acc: float32 [n, >= Sk] -- the high-precision dot products q.k of each
    requested row (row i, key c at acc[i, c]; only the keys the row sees are
    read) in place of fl32 of the exact ones: the result of the setup on that
    S, e.g. a matrix unit's own sums.  refs=True also returns the reference
    of every requested row at every key block it sees ([n, ceil(Sk/block)],
    NaN elsewhere): Alg. 1's m~ (the value T = S - m~ is taken against), or
    the running maximum m after the block in the eq. (2) setups.

    restart_rows / b0_last / visits (Alg. 1 setups only) take the tile-level
    path: the restart decision is shared by restart_rows consecutive query
    positions of one head, B0 also holds each row's last key block when
    b0_last, and the counts are per tile: restarts[n] (and, with visits,
    one more array of visited B1 tile-blocks before the margin) hold the
    row's tile's restarted B1 tile-blocks.  With acc, every row of every
    tile touched must be requested.

    Extra outputs come in the order visits, margin, refs."""
    L = _load()
    q, k, v = _bits(q), _bits(k), _bits(v)
    rows = _rows(rows, B * Hq * Sq)
    n = rows.size
    o = np.zeros((n, D), dtype=np.float64)
    lse = np.zeros(n, dtype=np.float64)
    nrs = np.zeros(n, dtype=np.int32)
    mg = np.zeros(n, dtype=np.float64) if margin else None
    nblk = (Sk + block - 1) // block if block > 0 else 0
    ref = np.full((n, max(nblk, 1)), np.nan, dtype=np.float64) if refs else None
    ld_ref = ref.shape[1] if refs else 0
    if acc is not None:
        acc = np.ascontiguousarray(acc, dtype=np.float32)
        if acc.ndim != 2 or acc.shape[0] != n or acc.shape[1] < Sk:
            raise ValueError("acc must be float32 [len(rows), >= Sk]")
        ld_acc = acc.shape[1]
    else:
        ld_acc = 0
    if restart_rows != 1 or b0_last or visits:
        nvs = np.zeros(n, dtype=np.int32)
        st = L.orc_attention_tiles(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, Sq, Sk, D, int(causal), block,
                                   int(mode), int(lam), int(n_b0), int(bool(b0_last)), int(restart_rows),
                                   int(literal_else), float(scale_log2), _ptr(rows), n, _ptr(o), _ptr(lse),
                                   _ptr(nrs), _ptr(nvs), _ptr(mg), int(nthreads), int(bool(tie_even)),
                                   _ptr(acc), ld_acc, _ptr(ref), ld_ref)
        if st:
            raise ValueError("oracle rejected the attention arguments")
        return (o, lse, nrs) + ((nvs,) if visits else ()) + ((mg,) if margin else ()) + ((ref,) if refs else ())
    st = L.orc_attention_ex(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, Sq, Sk, D, int(causal), block,
                            int(mode), int(lam), int(n_b0), int(literal_else), float(scale_log2),
                            _ptr(rows), n, _ptr(o), _ptr(lse), _ptr(nrs), _ptr(mg), int(nthreads),
                            int(bool(pv_bf16)), int(bool(tie_even)), _ptr(acc), ld_acc, _ptr(ref), ld_ref)
    if st:
        raise ValueError("oracle rejected the attention arguments")
    return (o, lse, nrs) + ((mg,) if margin else ()) + ((ref,) if refs else ())


def acc_bound(q, k, B, Hq, Hkv, Sq, Sk, D, rows):
    """The accumulation error bound of each requested row's dot products,
    [n, Sk] fp64: gamma_(D-1) * sum_d |q_d k_d| with gamma_n = n u/(1 - n u),
    u = 2^-24 -- how far a sum of the D exact products formed with fp32
    round-to-nearest additions, in any order, can lie from the exact q.k."""
    def f64(bits):
        return (_bits(bits).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    rows = _rows(rows, B * Hq * Sq)
    qf = f64(q).reshape(B * Hq * Sq, D)[rows]
    kf = f64(k).reshape(B, Hkv, Sk, D)
    b = rows // (Hq * Sq)
    g = (rows // Sq) % Hq // (Hq // Hkv)
    n_, u = max(D - 1, 0), 2.0 ** -24
    gamma = n_ * u / (1 - n_ * u)
    out = np.empty((rows.size, Sk), dtype=np.float64)
    for i in range(rows.size):
        out[i] = gamma * (np.abs(kf[b[i], g[i]]) @ np.abs(qf[i]))
    return out


def e4m3_to_bf16(codes) -> np.ndarray:
    """FP8 E4M3 (OCP) codes -> bf16 bit patterns of the same values, exactly:
    every finite E4M3 value (3 mantissa bits, exponents -9 .. 8) is a bf16
    value.  NaN codes (0x7F, 0xFF) are rejected."""
    L = _load()
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    table = np.array([L.orc_e4m3_decode(i) for i in range(256)], dtype=np.float64)
    if np.isnan(table[c]).any():
        raise ValueError("NaN FP8 code in q or k")
    f32 = table.astype(np.float32)
    bits = (f32.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal((bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)[~np.isnan(table)],
                          table[~np.isnan(table)])
    return bits[c]


def fp8_scale_log2(D, q_scale, k_scale, scale_log2=0.0) -> float:
    """The score scale with FP8 Q/K: c' = c * q_scale * k_scale in double
    (the scales as fp32), rounded once to fp32 by the attention path; c is
    scale_log2 or log2(e)/sqrt(D)."""
    base = float(scale_log2) if scale_log2 else math.log2(math.e) / math.sqrt(D)
    return base * float(np.float32(q_scale)) * float(np.float32(k_scale))


def exact_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, scale_log2=0.0, rows=None, nthreads=0):
    """eq. (1) in fp64.  Returns (o[n,D], lse[n])."""
    L = _load()
    q, k, v = _bits(q), _bits(k), _bits(v)
    rows = _rows(rows, B * Hq * Sq)
    n = rows.size
    o = np.zeros((n, D), dtype=np.float64)
    lse = np.zeros(n, dtype=np.float64)
    st = L.orc_exact_attention(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, Sq, Sk, D, int(causal),
                               float(scale_log2), _ptr(rows), n, _ptr(o), _ptr(lse), int(nthreads))
    if st:
        raise ValueError("oracle rejected the attention arguments")
    return o, lse


def softmax_block(s, block, lam=1, n_b0=1, nthreads=0):
    """The vector-side steps of Alg. 1 on fp32 scores s[rows, cols] (log2
    units, -inf = masked).  Returns codes[rows,cols] (uint8), ref_shift
    [rows,nblk] (int32), m_final[rows], d_final[rows] (fp64), restarted
    [rows,nblk] (uint8)."""
    L = _load()
    s = np.ascontiguousarray(np.asarray(s, dtype=np.float32))
    rows, cols = s.shape
    nblk = (cols + block - 1) // block
    codes = np.zeros((rows, cols), dtype=np.uint8)
    refs = np.zeros((rows, nblk), dtype=np.int32)
    m = np.zeros(rows, dtype=np.float64)
    d = np.zeros(rows, dtype=np.float64)
    rs = np.zeros((rows, nblk), dtype=np.uint8)
    st = L.orc_softmax_block(_ptr(s), rows, cols, cols, block, int(lam), int(n_b0), _ptr(codes),
                             _ptr(refs), _ptr(m), _ptr(d), _ptr(rs), int(nthreads))
    if st:
        raise ValueError("oracle rejected the softmax-block arguments")
    return codes, refs, m, d, rs
