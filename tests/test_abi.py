"""The C-ABI library loads, exports every symbol include/baps.h declares, and
rejects bad arguments before touching the GPU (CPU only)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2602_02071_amd as baps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "baps.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?(?:(?:unsigned|long|short)\s+)*\w+[\s*]+(\w+)\s*\(",
                                 src, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(baps.LIB_PATH):
        pytest.fail("libbaps.so is not built (run __graft_entry__.build())")
    return baps.load()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) >= {"baps_attention_fwd", "baps_attention_fwd_ex", "hif8_encode", "hif8_decode",
                          "baps_softmax_block", "baps_get_exp2_lut"}
    for n in names:
        assert hasattr(lib, n), n
    assert set(baps.EXPORTS) == set(names)


def test_exp2_lut_matches_oracle(lib):
    lut = np.frombuffer(baps.baps_get_exp2_lut(), dtype=np.uint8)
    assert np.array_equal(lut, O.exp2_table(0))


def test_status_strings(lib):
    assert baps.status_string(0) == "ok"
    assert "invalid" in baps.status_string(1)
    assert "unsupported" in baps.status_string(2)
    assert baps.status_string(99) == "unknown status"


def _attn(lib, q=16, k=16, v=16, o=16, B=1, Hq=2, Hkv=1, Sq=8, Sk=8, D=64, causal=0, block=64):
    return lib.baps_attention_fwd(q, k, v, o, None, B, Hq, Hkv, Sq, Sk, D, causal, block, None)


def test_attention_argument_checks(lib):
    assert _attn(lib, B=-1) == 1
    assert _attn(lib, Sk=-3) == 1
    assert _attn(lib, Hq=3, Hkv=2) == 1
    assert _attn(lib, Hkv=0) == 1
    assert _attn(lib, q=None) == 1
    assert _attn(lib, o=None) == 1
    assert _attn(lib, q=18) == 1                 # q not 16-byte aligned
    assert _attn(lib, D=96) == 2
    assert _attn(lib, block=48) == 2
    assert _attn(lib, B=0) == 0                  # empty work
    assert _attn(lib, Sq=0, q=None, o=None) == 0
    prm = baps.baps_params_t(1, 1, -1.0, None, 0)
    assert lib.baps_attention_fwd_ex(16, 16, 16, 16, None, 1, 1, 1, 4, 4, 64, 0, 64, ctypes.byref(prm), None) == 1
    for bad_mode in (-1, 3, 7):                  # softmax setup out of range
        prm = baps.baps_params_t(1, 1, 0.0, None, bad_mode)
        assert lib.baps_attention_fwd_ex(16, 16, 16, 16, None, 1, 1, 1, 4, 4, 64, 0, 64, ctypes.byref(prm),
                                         None) == 1
    for mode in (baps.BAPS_MODE_DEFAULT, baps.BAPS_MODE_EXP2_HIF8):   # valid, empty work
        prm = baps.baps_params_t(1, 1, 0.0, None, mode)
        assert lib.baps_attention_fwd_ex(16, 16, 16, 16, None, 0, 1, 1, 4, 4, 64, 0, 64, ctypes.byref(prm),
                                         None) == 0
    assert lib.baps_attention_fwd_ex(16, 16, 16, 16, None, 1, 1, 1, 4, 4, 64, 0, 64, None, None) == 1


def test_tile_restart_argument_checks(lib):
    """Tile-level restart needs powers of two that keep a tile inside one
    workgroup (no GPU work: the checks run before any HIP call)."""
    def ex(Hq, Hkv, Sq, R, mode=0):
        prm = baps.baps_params_t(1, 1, 0.0, None, mode, R, 0, None)
        return lib.baps_attention_fwd_ex(16, 16, 16, 16, None, 1, Hq, Hkv, Sq, 64, 64, 1, 64, ctypes.byref(prm), None)
    assert ex(8, 2, 64, -1) == 1                 # negative tile height
    assert ex(8, 2, 64, 3) == 2                  # not a power of two
    assert ex(6, 2, 64, 2) == 2                  # Hq/Hkv = 3: not a power of two
    assert ex(32, 1, 64, 16) == 2                # 16 positions x 32 heads > 256 rows
    assert ex(8, 2, 64, 2, mode=baps.BAPS_MODE_DEFAULT) == 2   # eq. (2) setups have no restarts
    assert ex(8, 2, 0, 3) == 0                   # empty work is checked first
    assert baps.baps_attention_split_workspace(1, 32, 8, 4, 32768, 128, 128, restart_rows=4) == 0
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128, restart_rows=4) > 0   # Sq = 1
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128, b0_last=True) > 0


def test_split_workspace_and_checks(lib):
    P = ctypes.POINTER(baps.baps_params_t)
    # the split path is taken for few streams and many keys only
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128) > 0
    assert baps.baps_attention_split_workspace(64, 32, 8, 1, 8192, 128, 128) == 0      # enough streams
    assert baps.baps_attention_split_workspace(1, 32, 8, 4096, 4096, 128, 128) == 0    # prefill regime
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 256, 128, 128) == 0        # 2 key blocks
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128, lam=9) == 0
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128, mode=1) == 0
    need = baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128)
    # a needed workspace that is missing, short or misaligned is an invalid argument (no GPU work)
    args = (16, 16, 16, 16, None, 1, 32, 8, 1, 32768, 128, 0, 128, None)
    assert lib.baps_attention_fwd_split(*args, None, need, None) == 1
    assert lib.baps_attention_fwd_split(*args, 4096, need - 1, None) == 1
    assert lib.baps_attention_fwd_split(*args, 4096 + 16, need, None) == 1
    assert lib.baps_attention_fwd_split(16, 16, 16, 16, None, 0, 32, 8, 1, 32768, 128, 0, 128, None, None, 0,
                                        None) == 0                                      # empty work


def test_codec_and_softmax_block_argument_checks(lib):
    assert lib.hif8_encode(16, 16, -1, 1, None) == 1
    assert lib.hif8_encode(16, 16, 10, 4, None) == 1
    assert lib.hif8_encode(None, 16, 10, 1, None) == 1
    assert lib.hif8_encode(None, None, 0, 1, None) == 0
    assert lib.hif8_decode(16, None, 10, None) == 1
    assert lib.hif8_decode(None, None, 0, None) == 0
    sb = lib.baps_softmax_block
    assert sb(16, 4, 100, 99, 64, 1, 1, 0, 16, 16, 16, 16, None, None) == 1      # ld < cols
    assert sb(16, 4, 100, 100, 96, 1, 1, 0, 16, 16, 16, 16, None, None) == 2     # block
    assert sb(16, 4, 100, 100, 64, 1, 1, 3, 16, 16, 16, 16, None, None) == 1     # flags
    assert sb(16, 4, 100, 100, 64, 1, -1, 0, 16, 16, 16, 16, None, None) == 1    # n_b0
    assert sb(None, 4, 100, 100, 64, 1, 1, 0, 16, 16, 16, 16, None, None) == 1
    assert sb(None, 0, 100, 100, 64, 1, 1, 0, None, None, None, None, None, None) == 0


def test_fp8_argument_checks(lib):
    """FP8 Q/K: scales must be finite and positive, the format known, and
    tile-level restart is not combined with it (no GPU work)."""
    def ex(fmt, qs, ks, R=1):
        prm = baps.baps_params_t(1, 1, 0.0, None, 0, R, 0, None, fmt, qs, ks)
        return lib.baps_attention_fwd_ex(16, 16, 16, 16, None, 1, 8, 2, 64, 64, 128, 1, 128, ctypes.byref(prm), None)
    assert ex(2, 1.0, 1.0) == 1                  # unknown format
    assert ex(baps.BAPS_QK_FP8_E4M3, 0.0, 1.0) == 1
    assert ex(baps.BAPS_QK_FP8_E4M3, 1.0, -2.0) == 1
    assert ex(baps.BAPS_QK_FP8_E4M3, float("inf"), 1.0) == 1
    assert ex(baps.BAPS_QK_FP8_E4M3, 1.0, 1.0, R=4) == 2
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128, qk_scales=(1.0, 1.0)) > 0


def test_cast_and_output_knob_checks(lib):
    """tie_mode, saturate and out_bf16 of baps_params_t (no GPU work: the
    checks run before any HIP call, or the work is empty)."""
    def ex(tie=0, sat=1, out_bf16=0, lam=1, mode=0, R=1, fmt=0, B=1, o=16):
        prm = baps.baps_params_t(lam, 1, 0.0, None, mode, R, 0, None, fmt, 1.0, 1.0, tie, sat, out_bf16)
        return lib.baps_attention_fwd_ex(16, 16, 16, o, None, B, 8, 2, 64, 64, 128, 1, 128, ctypes.byref(prm), None)
    assert ex(tie=2) == 1 and ex(tie=-1) == 1                       # unknown tie rule
    assert ex(tie=1, mode=baps.BAPS_MODE_DEFAULT) == 2               # ties to even: Alg. 1 only
    assert ex(tie=1, lam=9) == 2                                     # ... with the compact table
    assert ex(tie=1, R=4) == 2                                       # ... per row
    assert ex(tie=1, fmt=baps.BAPS_QK_FP8_E4M3) == 2                 # ... bf16 Q/K
    assert ex(tie=1, B=0) == 0                                       # empty work first
    assert ex(sat=0, lam=16) == 2                                    # an 8-bit P could overflow
    assert ex(sat=0, lam=15, B=0) == 0 and ex(sat=0, lam=100, mode=baps.BAPS_MODE_DEFAULT, B=0) == 0
    assert ex(out_bf16=1, o=18) == 1                                 # misaligned output
    # the split-key path keeps the canonical ties; other knobs go to the one-pass kernels
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128, tie_mode=1) == 0
    assert baps.baps_attention_split_workspace(1, 32, 8, 1, 32768, 128, 128, out_bf16=True) > 0
    assert lib.hif8_encode(16, 16, 10, baps.BAPS_HIF8_TIES_EVEN | 4, None) == 1


def test_dump_argument_checks(lib):
    d = lib.baps_attention_fwd_dump
    assert d(16, 16, 16, 16, None, 1, 2, 1, 8, 8, 64, 0, 64, None, None, 16, 16, None) == 1     # no row map
    assert d(16, 16, 16, 16, None, 1, 2, 1, 8, 8, 64, 0, 64, None, 16, None, 16, None) == 1     # no acc buffer
    assert d(16, 16, 16, 16, None, 1, 2, 1, 8, 8, 64, 0, 64, None, 16, 16, None, None) == 1     # no ref buffer
    assert d(16, 16, 16, 16, None, 1, 2, 1, 8, 8, 96, 0, 64, None, 16, 16, 16, None) == 2       # D
    assert d(16, 16, 16, 16, None, 0, 2, 1, 8, 8, 64, 0, 64, None, None, None, None, None) == 0  # empty
