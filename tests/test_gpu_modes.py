"""The two eq. (2) setups of the fused kernels against the oracle (GPU):
Default (fp32 softmax; P enters P V as bf16, the oracle's pv_bf16 reading)
and Exp2 HiF8 (the exp2 on 8-bit input, rounded to 8 bits; its 8-bit
decisions use the same margin and valid-S rule as the E2E HiF8 checks).
Same bar: O within rel-L2 2e-3 and max-abs 1e-2 of the oracle."""
import numpy as np
import pytest

import oracle as O
from helpers import check_parity, gpu_attention
from paper_2602_02071_amd.workloads import make_qkv, make_workload, sample_rows

pytestmark = pytest.mark.gpu

MODES = {"default": O.DEFAULT, "exp2_hif8": O.EXP2_HIF8}


def _check(q, k, v, shape, block, mode, rows=None, label=""):
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    o, lse = gpu_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, mode=mode)
    if rows is not None:
        o, lse = o[rows], lse[rows]
    return check_parity(q, k, v, shape, block, o, lse, rows=rows, label=label, mode=mode,
                        pv_bf16=(mode == O.DEFAULT))


SHAPES = [
    # B, Hq, Hkv, Sq, Sk, D, causal, block
    (1, 1, 1, 256, 256, 64, False, 64),
    (2, 4, 2, 300, 300, 128, True, 128),
    (1, 8, 2, 200, 333, 64, True, 64),
    (3, 2, 2, 97, 515, 128, False, 32),
    (2, 8, 2, 1, 1000, 128, False, 128),     # decode kernel
    (1, 4, 1, 5, 400, 128, True, 64),        # decode kernel, causal chunk
]


@pytest.mark.parametrize("mode", list(MODES), ids=list(MODES))
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_mode_shapes(shape, mode):
    B, Hq, Hkv, Sq, Sk, D, causal, block = shape
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=sum(shape) + 3, outliers=True)
    _check(q, k, v, shape[:7], block, MODES[mode], label=f"{mode} {shape}")


@pytest.mark.parametrize("mode", list(MODES), ids=list(MODES))
def test_mode_llama_prefill_sampled_rows(mode):
    w, q, k, v = make_workload(2)
    shape = (w.B, w.Hq, w.Hkv, w.Sq, w.Sk, w.D, w.causal)
    rows = sample_rows(w, every=512, tile=1024, heads=range(0, w.Hq, 5))
    _check(q, k, v, shape, w.block, MODES[mode], rows=rows, label=f"{mode} {w.name}")
