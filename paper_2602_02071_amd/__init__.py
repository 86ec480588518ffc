"""BAPS attention on MI355X: Python binding of libbaps.so.

The names match the C ABI in include/baps.h.  This module only marshals
arguments (tensor -> device pointer, stream -> handle, status -> exception);
every step of the method runs in the library's HIP kernels.  PyTorch is used
for device memory and streams only.  If the library has not been built the
calls raise: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbaps.so")

BAPS_OK = 0
BAPS_INVALID_ARGUMENT = 1
BAPS_UNSUPPORTED = 2
BAPS_HIP_ERROR = 3
BAPS_HIF8_SATURATE = 1
BAPS_HIF8_TIES_EVEN = 2
BAPS_TIES_AWAY = 0
BAPS_TIES_EVEN = 1

BAPS_SPLIT_SCRATCH_BYTES = 32 << 20

EXPORTS = ("baps_attention_fwd", "baps_attention_fwd_ex", "baps_attention_fwd_split", "baps_attention_fwd_dump",
           "baps_attention_fwd_split_noalloc",
           "hif8_encode", "hif8_decode", "baps_softmax_block", "baps_get_exp2_lut", "baps_init",
           "baps_attention_split_workspace", "baps_last_hip_error", "baps_status_string")

_lib = None


class BapsError(RuntimeError):
    def __init__(self, fn, status):
        detail = f", {load().baps_last_hip_error().decode()}" if status == 3 else ""
        super().__init__(f"{fn}: {status_string(status)} (status {status}{detail})")
        self.status = status


class baps_params_t(ctypes.Structure):
    _fields_ = [("lambda_", ctypes.c_int), ("n_b0", ctypes.c_int), ("scale_log2", ctypes.c_float),
                ("restart_counts", ctypes.c_void_p), ("mode", ctypes.c_int), ("restart_rows", ctypes.c_int),
                ("b0_last", ctypes.c_int), ("tile_counts", ctypes.c_void_p), ("qk_format", ctypes.c_int),
                ("q_scale", ctypes.c_float), ("k_scale", ctypes.c_float), ("tie_mode", ctypes.c_int),
                ("saturate", ctypes.c_int), ("out_bf16", ctypes.c_int)]


# softmax setups (include/baps.h)
BAPS_MODE_E2E_HIF8 = 0
BAPS_MODE_DEFAULT = 1
BAPS_MODE_EXP2_HIF8 = 2
# Q/K formats (include/baps.h)
BAPS_QK_BF16 = 0
BAPS_QK_FP8_E4M3 = 1


def load():
    """Load libbaps.so (raises when it is missing: build it first)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() (hipcc, gfx950) first")
    # torch ships its own HIP and HSA runtimes under the same sonames as the
    # system ones; with torch loaded first the library binds to them, so the
    # process holds one runtime (two would both claim the GPU, and the second
    # to start up finds no device).
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P, I, LL = ctypes.c_void_p, ctypes.c_int, ctypes.c_longlong
    L.baps_attention_fwd.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I, P]
    L.baps_attention_fwd_ex.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I,
                                        ctypes.POINTER(baps_params_t), P]
    L.baps_attention_fwd_split.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I,
                                           ctypes.POINTER(baps_params_t), P, LL, P]
    L.baps_attention_fwd_dump.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I,
                                          ctypes.POINTER(baps_params_t), P, P, P, P]
    L.baps_attention_fwd_split_noalloc.argtypes = [P, P, P, P, P, I, I, I, I, I, I, I, I,
                                                   ctypes.POINTER(baps_params_t), P]
    L.baps_attention_split_workspace.argtypes = [I, I, I, I, I, I, I, ctypes.POINTER(baps_params_t)]
    L.hif8_encode.argtypes = [P, P, LL, I, P]
    L.hif8_decode.argtypes = [P, P, LL, P]
    L.baps_softmax_block.argtypes = [P, LL, LL, LL, I, I, I, I, P, P, P, P, P, P]
    L.baps_get_exp2_lut.argtypes = [P]
    L.baps_init.argtypes = []
    L.baps_status_string.argtypes = [I]
    L.baps_status_string.restype = ctypes.c_char_p
    L.baps_last_hip_error.argtypes = []
    L.baps_last_hip_error.restype = ctypes.c_char_p
    for name in EXPORTS[:-2]:
        getattr(L, name).restype = I
    L.baps_attention_split_workspace.restype = LL
    _lib = L
    return L


def status_string(status: int) -> str:
    return load().baps_status_string(int(status)).decode()


def _p(x):
    """Device pointer of a tensor (or an int / None passed through)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(fn, st):
    if st != BAPS_OK:
        raise BapsError(fn, st)


def baps_attention_fwd(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, stream=None):
    _check("baps_attention_fwd", load().baps_attention_fwd(
        _p(q), _p(k), _p(v), _p(o), _p(lse), B, Hq, Hkv, Sq, Sk, D, int(causal), block, _stream(stream)))


def _params(lam=1, n_b0=1, scale_log2=0.0, restart_counts=None, mode=BAPS_MODE_E2E_HIF8, restart_rows=1,
            b0_last=False, tile_counts=None, qk_scales=None, tie_mode=BAPS_TIES_AWAY, saturate=True,
            out_bf16=False):
    fmt, qs, ks = (BAPS_QK_BF16, 1.0, 1.0) if qk_scales is None else (BAPS_QK_FP8_E4M3,) + tuple(qk_scales)
    return baps_params_t(int(lam), int(n_b0), float(scale_log2), _p(restart_counts), int(mode), int(restart_rows),
                         int(bool(b0_last)), _p(tile_counts), int(fmt), float(qs), float(ks), int(tie_mode),
                         int(bool(saturate)), int(bool(out_bf16)))


def baps_attention_fwd_ex(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, lam=1, n_b0=1,
                          scale_log2=0.0, restart_counts=None, stream=None, mode=BAPS_MODE_E2E_HIF8,
                          restart_rows=1, b0_last=False, tile_counts=None, qk_scales=None, tie_mode=BAPS_TIES_AWAY,
                          saturate=True, out_bf16=False):
    """qk_scales=(q_scale, k_scale): q and k are FP8 E4M3 codes (uint8 tensors).
    out_bf16: o is a bf16 tensor."""
    prm = _params(lam, n_b0, scale_log2, restart_counts, mode, restart_rows, b0_last, tile_counts, qk_scales,
                  tie_mode, saturate, out_bf16)
    _check("baps_attention_fwd_ex", load().baps_attention_fwd_ex(
        _p(q), _p(k), _p(v), _p(o), _p(lse), B, Hq, Hkv, Sq, Sk, D, int(causal), block,
        ctypes.byref(prm), _stream(stream)))


def baps_attention_fwd_dump(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, row_slot, acc_out, ref_out,
                            stream=None, **knobs):
    """The fused pass with a dump of the selected rows' raw dot products and
    block references (include/baps.h); knobs as baps_attention_fwd_ex."""
    prm = _params(**knobs)
    _check("baps_attention_fwd_dump", load().baps_attention_fwd_dump(
        _p(q), _p(k), _p(v), _p(o), _p(lse), B, Hq, Hkv, Sq, Sk, D, int(causal), block,
        ctypes.byref(prm), _p(row_slot), _p(acc_out), _p(ref_out), _stream(stream)))


def baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, block, lam=1, n_b0=1, scale_log2=0.0,
                                   mode=BAPS_MODE_E2E_HIF8, restart_rows=1, b0_last=False, qk_scales=None,
                                   tie_mode=BAPS_TIES_AWAY, saturate=True, out_bf16=False):
    prm = _params(lam, n_b0, scale_log2, None, mode, restart_rows, b0_last, None, qk_scales, tie_mode, saturate,
                  out_bf16)
    return int(load().baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, block, ctypes.byref(prm)))


def baps_attention_fwd_split(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, workspace, workspace_bytes,
                             lam=1, n_b0=1, scale_log2=0.0, restart_counts=None, stream=None,
                             mode=BAPS_MODE_E2E_HIF8, restart_rows=1, b0_last=False, tile_counts=None,
                             qk_scales=None, tie_mode=BAPS_TIES_AWAY, saturate=True, out_bf16=False):
    prm = _params(lam, n_b0, scale_log2, restart_counts, mode, restart_rows, b0_last, tile_counts, qk_scales,
                  tie_mode, saturate, out_bf16)
    _check("baps_attention_fwd_split", load().baps_attention_fwd_split(
        _p(q), _p(k), _p(v), _p(o), _p(lse), B, Hq, Hkv, Sq, Sk, D, int(causal), block,
        ctypes.byref(prm), _p(workspace), int(workspace_bytes), _stream(stream)))


def baps_attention_fwd_split_noalloc(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block, stream=None, **knobs):
    """The split-key path on the library's static scratch (no allocation);
    knobs as baps_attention_fwd_ex."""
    prm = _params(**knobs)
    _check("baps_attention_fwd_split_noalloc", load().baps_attention_fwd_split_noalloc(
        _p(q), _p(k), _p(v), _p(o), _p(lse), B, Hq, Hkv, Sq, Sk, D, int(causal), block,
        ctypes.byref(prm), _stream(stream)))


def hif8_encode(x, codes, n, flags=BAPS_HIF8_SATURATE, stream=None):
    _check("hif8_encode", load().hif8_encode(_p(x), _p(codes), n, flags, _stream(stream)))


def hif8_decode(codes, x, n, stream=None):
    _check("hif8_decode", load().hif8_decode(_p(codes), _p(x), n, _stream(stream)))


def baps_softmax_block(s, rows, cols, ld_s, block, lam, n_b0, flags, p_codes, ref_shift, m_final, d_final,
                       restarted=None, stream=None):
    _check("baps_softmax_block", load().baps_softmax_block(
        _p(s), rows, cols, ld_s, block, lam, n_b0, flags, _p(p_codes), _p(ref_shift), _p(m_final),
        _p(d_final), _p(restarted), _stream(stream)))


def baps_get_exp2_lut():
    buf = (ctypes.c_ubyte * 256)()
    _check("baps_get_exp2_lut", load().baps_get_exp2_lut(buf))
    return bytes(buf)


def baps_init():
    _check("baps_init", load().baps_init())


# ------------------------------------------------------------ tensor helpers
def attention(q, k, v, causal, block, lse=True, lam=None, n_b0=None, scale_log2=0.0, restart_counts=None,
              stream=None, mode=BAPS_MODE_E2E_HIF8, split=False, restart_rows=1, b0_last=False, tile_counts=None,
              qk_scales=None, tie_mode=BAPS_TIES_AWAY, saturate=True, out_bf16=False):
    """Allocate O (and lse) with torch on q's device and run the fused pass.
    q [B,Hq,Sq,D], k/v [B,Hkv,Sk,D] bf16 CUDA tensors, contiguous.  split:
    take baps_attention_fwd_split, with a workspace allocated here.
    restart_rows / b0_last / tile_counts: the tile-level restart knobs of
    baps_params_t.  qk_scales=(q_scale, k_scale): q and k are FP8 E4M3 codes
    (uint8 tensors) with those dequantisation scales.  out_bf16: O is
    returned as bf16."""
    import torch
    B, Hq, Sq, D = q.shape
    Hkv, Sk = k.shape[1], k.shape[2]
    _check_inputs(q, k, v, qk_scales)
    o = torch.empty((B, Hq, Sq, D), dtype=torch.bfloat16 if out_bf16 else torch.float32, device=q.device)
    l = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device) if lse else None
    lam_, nb_ = 1 if lam is None else lam, 1 if n_b0 is None else n_b0
    extra = dict(tie_mode=tie_mode, saturate=saturate, out_bf16=out_bf16)
    if split:
        nbytes = baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, block, lam_, nb_, scale_log2, mode,
                                                restart_rows, b0_last, qk_scales, **extra)
        ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=q.device)
        baps_attention_fwd_split(q, k, v, o, l, B, Hq, Hkv, Sq, Sk, D, causal, block, ws, nbytes, lam_, nb_,
                                 scale_log2, restart_counts, stream, mode, restart_rows, b0_last, tile_counts,
                                 qk_scales, **extra)
    elif (lam is None and n_b0 is None and not scale_log2 and restart_counts is None and mode == BAPS_MODE_E2E_HIF8
          and restart_rows == 1 and not b0_last and tile_counts is None and qk_scales is None
          and tie_mode == BAPS_TIES_AWAY and saturate and not out_bf16):
        baps_attention_fwd(q, k, v, o, l, B, Hq, Hkv, Sq, Sk, D, causal, block, stream)
    else:
        baps_attention_fwd_ex(q, k, v, o, l, B, Hq, Hkv, Sq, Sk, D, causal, block, lam_, nb_, scale_log2,
                              restart_counts, stream, mode, restart_rows, b0_last, tile_counts, qk_scales, **extra)
    return o, l


def _check_inputs(q, k, v, qk_scales):
    import torch
    qk_dtype = torch.bfloat16 if qk_scales is None else torch.uint8
    for t, dt in ((q, qk_dtype), (k, qk_dtype), (v, torch.bfloat16)):
        if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("q, k (bf16, or uint8 FP8 codes with qk_scales) and v (bf16) must be contiguous "
                             "device tensors")


def attention_dump(q, k, v, causal, block, rows, lam=1, n_b0=1, scale_log2=0.0, mode=BAPS_MODE_E2E_HIF8,
                   restart_rows=1, b0_last=False, qk_scales=None, tie_mode=BAPS_TIES_AWAY, saturate=True,
                   stream=None):
    """baps_attention_fwd_dump with buffers allocated here: the fused pass
    (o, lse as from attention()) plus, for the global query rows `rows`
    ((b*Hq + h)*Sq + r, distinct), their raw dot products acc [n, Sk] (NaN
    where the row sees no key) and block references ref [n, ceil(Sk/block)]
    (NaN where the row sees no key of the block), as device tensors."""
    import torch
    B, Hq, Sq, D = q.shape
    Hkv, Sk = k.shape[1], k.shape[2]
    _check_inputs(q, k, v, qk_scales)
    rows = torch.as_tensor(rows, dtype=torch.int64).reshape(-1)
    n = rows.numel()
    if n and (rows.min() < 0 or rows.max() >= B * Hq * Sq or rows.unique().numel() != n):
        raise ValueError("rows must be distinct query-row indices")
    slot = torch.full((B * Hq * Sq,), -1, dtype=torch.int32)
    slot[rows] = torch.arange(n, dtype=torch.int32)
    slot = slot.to(q.device)
    nblk = (Sk + block - 1) // block
    acc = torch.full((max(n, 1), max(Sk, 1)), float("nan"), dtype=torch.float32, device=q.device)
    ref = torch.full((max(n, 1), max(nblk, 1)), float("nan"), dtype=torch.float32, device=q.device)
    o = torch.empty((B, Hq, Sq, D), dtype=torch.float32, device=q.device)
    l = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
    baps_attention_fwd_dump(q, k, v, o, l, B, Hq, Hkv, Sq, Sk, D, causal, block, slot, acc, ref, stream,
                            lam=lam, n_b0=n_b0, scale_log2=scale_log2, mode=mode, restart_rows=restart_rows,
                            b0_last=b0_last, qk_scales=qk_scales, tie_mode=tie_mode, saturate=saturate)
    return o, l, acc[:n, :Sk], ref[:n, :nblk]
