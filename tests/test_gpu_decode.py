"""Parity of the few-rows-per-KV-head kernel (decode, short query chunks) with
the oracle (GPU).

A KV head with at most 64 flattened (query position, query head) rows takes
the decode kernel, whose waves split every key block and exchange row maxima;
these cases cover every (D, block) pair, ragged key counts, bottom-right
causal short queries, the 64/65-row boundary to the prefill kernel, the
lambda knobs (lambda > 8 uses the full score table) and the restart
counters."""
import numpy as np
import pytest

import oracle as O
from helpers import check_parity, dev_bf16, gpu_attention
from paper_2602_02071_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu


def _check(q, k, v, shape, block, label="", **knobs):
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    o, lse = gpu_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, **knobs)
    okw = {key: knobs[key] for key in ("lam", "n_b0", "scale_log2") if key in knobs}
    return check_parity(q, k, v, shape, block, o, lse, label=label, **okw)


DECODE = [
    # B, Hq, Hkv, Sq, Sk, D, causal, block
    (3, 8, 2, 1, 777, 64, False, 64),       # ragged key count, GQA 4
    (2, 4, 4, 1, 300, 64, False, 32),       # MHA, one wave per workgroup
    (2, 8, 1, 1, 1030, 128, False, 128),    # GQA 8
    (2, 4, 1, 1, 4096 + 33, 128, False, 64),
    (1, 4, 1, 5, 400, 128, True, 128),      # causal chunk of 5 queries: 20 rows, 2 row tiles
    (1, 4, 1, 16, 640, 128, True, 64),      # 64 rows: the last shape on the decode kernel
    (1, 4, 1, 17, 640, 128, True, 64),      # 68 rows: the first on the prefill kernel
    (2, 2, 2, 3, 31, 128, True, 128),       # fewer keys than one 32-key slot
    (1, 16, 1, 4, 2000, 64, True, 128),     # GQA 16, 64 rows, D 64
    (1, 2, 1, 9, 5, 128, True, 32),         # Sq > Sk: the leading rows see no key
]


@pytest.mark.parametrize("shape", DECODE, ids=lambda s: "x".join(map(str, s)))
def test_decode_shapes(shape):
    B, Hq, Hkv, Sq, Sk, D, causal, block = shape
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=sum(shape) + 7, outliers=True, lognormal_k=True)
    _check(q, k, v, shape[:7], block, label=str(shape))


@pytest.mark.parametrize("lam,n_b0", [(0, 1), (1, 3), (100, 1), (-100, 1), (8, 1), (9, 2)])
def test_decode_knobs(lam, n_b0):
    shape = (4, 8, 2, 1, 2048 + 64, 128, False)
    q, k, v = make_qkv(*shape[:6], seed=77, outliers=True, sink=3)
    _check(q, k, v, shape, 128, label=f"decode lam={lam} n_b0={n_b0}", lam=lam, n_b0=n_b0)


@pytest.mark.parametrize("block", [32, 128])
def test_decode_restart_counts(block):
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D = 3, 8, 2, 2, 1500, 128
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=91 + block, outliers=True)
    cnt = torch.zeros((B * Hq, 2), dtype=torch.int64, device="cuda:0")
    baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), True, block, restart_counts=cnt)
    torch.cuda.synchronize()
    cnt = cnt.cpu().numpy()
    _, _, nr = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, True, block)
    want = nr.reshape(B * Hq, Sq).sum(1)
    assert np.abs(cnt[:, 0] - want).max() <= max(2, 0.01 * want.max()), (cnt[:, 0], want)
    kmax = np.minimum(Sk - 1, np.arange(Sq) + Sk - Sq)
    assert np.all(cnt[:, 1] == (kmax // block).sum())
