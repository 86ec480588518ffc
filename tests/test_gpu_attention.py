"""Parity of the fused BAPS attention kernel with the oracle (GPU).

Bar: O within relative L2 2e-3 and max abs 1e-2 of the oracle on the same
seeded bf16 inputs; lse likewise; deviation from the fp64 exact attention is
printed alongside.  Small cases cover several tiles, ragged tails, GQA,
causal with Sq < Sk and Sq > Sk, every kernel (D, block) pair and the Alg. 1
knobs; the full-size workloads are checked on a deterministic row subset
(rows are independent under the per-row restart reading, so the subset is
exact)."""
import numpy as np
import pytest

import oracle as O
from helpers import check_parity, gpu_attention
from paper_2602_02071_amd.workloads import WORKLOADS, f32_to_bf16_bits, make_qkv, make_workload, sample_rows

pytestmark = pytest.mark.gpu


def _check(q, k, v, shape, block, rows=None, label="", **knobs):
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    o, lse = gpu_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, **knobs)
    okw = {key: knobs[key] for key in ("lam", "n_b0", "scale_log2") if key in knobs}
    if rows is not None:
        o, lse = o[rows], lse[rows]
    check_parity(q, k, v, shape, block, o, lse, rows=rows, label=label, **okw)
    return o


SMALL = [
    # B, Hq, Hkv, Sq, Sk, D, causal, block
    (1, 1, 1, 256, 256, 64, False, 64),
    (2, 4, 2, 300, 300, 128, True, 128),
    (1, 8, 2, 200, 333, 64, True, 64),        # Sq < Sk causal, ragged
    (1, 2, 1, 333, 150, 128, True, 64),       # Sq > Sk: leading rows see nothing
    (3, 2, 2, 97, 515, 128, False, 32),
    (1, 4, 4, 129, 129, 64, False, 128),
    (2, 4, 1, 1, 1000, 128, False, 128),      # decode-shaped, GQA 4
    (1, 2, 2, 64, 64, 64, True, 32),
]


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_small_shapes(shape):
    B, Hq, Hkv, Sq, Sk, D, causal, block = shape
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=sum(shape), outliers=True)
    _check(q, k, v, shape[:7], block, label=str(shape))


@pytest.mark.parametrize("lam,n_b0", [(0, 1), (2, 1), (1, 0), (1, 3), (-100, 1), (100, 1)])
def test_alg1_knobs(lam, n_b0):
    shape = (1, 4, 2, 256, 512, 128, True)
    q, k, v = make_qkv(*shape[:6], seed=41, outliers=True, sink=2)
    _check(q, k, v, shape, 128, label=f"lam={lam} n_b0={n_b0}", lam=lam, n_b0=n_b0)


def test_restart_counts_match_oracle():
    import torch
    import paper_2602_02071_amd as baps
    from helpers import dev_bf16
    B, Hq, Hkv, Sq, Sk, D = 1, 4, 2, 256, 512, 128
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=42, outliers=True)
    cnt = torch.zeros((B * Hq, 2), dtype=torch.int64, device="cuda:0")
    baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), True, 64, lam=1, n_b0=1, restart_counts=cnt)
    torch.cuda.synchronize()
    cnt = cnt.cpu().numpy()
    _, _, nr = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, True, 64)
    want = nr.reshape(B * Hq, Sq).sum(1)
    # restart decisions hinge on ceil of 8-bit values: allow a handful of flips
    assert np.abs(cnt[:, 0] - want).max() <= max(2, 0.01 * want.max()), (cnt[:, 0], want)
    kmax = np.minimum(Sk - 1, np.arange(Sq) + Sk - Sq)
    visits = (kmax // 64).sum()                 # B1 blocks per head (blocks after the first)
    assert np.all(cnt[:, 1] == visits)


def test_integer_scores_exact():
    # scale 1, entries in {-1,0,1}: every score, T and P is exact, so GPU and
    # oracle agree to fp32 rounding of the accumulations
    g = np.random.default_rng(5)
    B, H, Sq, Sk, D = 1, 2, 130, 260, 64
    q = f32_to_bf16_bits(g.integers(-1, 2, (B, H, Sq, D)).astype(np.float32) * np.float32(0.25))
    k = f32_to_bf16_bits(g.integers(-1, 2, (B, H, Sk, D)).astype(np.float32))
    v = f32_to_bf16_bits(g.standard_normal((B, H, Sk, D)).astype(np.float32))
    o = _check(q, k, v, (B, H, H, Sq, Sk, D, True), 64, label="integer scores", scale_log2=1.0)
    ref, _, _ = O.attention(q, k, v, B, H, H, Sq, Sk, D, True, 64, scale_log2=1.0)
    assert np.abs(o - ref).max() < 1e-5


def test_zero_keys():
    import torch
    import paper_2602_02071_amd as baps
    from helpers import dev_bf16
    q, _, _ = make_qkv(1, 2, 1, 5, 1, 64, seed=1)
    k = np.zeros((1, 1, 0, 64), np.uint16)
    o, lse = baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(k), False, 64)
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.all(torch.isneginf(lse))


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workload_sampled_rows(cfg):
    # the full-size workloads in the benchmark's launch configuration: every
    # row of workloads 1 and 3, and every 64th query row of every head plus
    # the last row of each 128-row query tile of workloads 2, 4 and 5
    # (3072, 12288 and 24576 rows)
    w, q, k, v = make_workload(cfg)
    shape = (w.B, w.Hq, w.Hkv, w.Sq, w.Sk, w.D, w.causal)
    if cfg == 1:
        rows = None
    elif cfg == 3:
        rows = sample_rows(w, every=1, tile=1)            # every decode row
    else:
        rows = sample_rows(w, every=64, tile=128)
    _check(q, k, v, shape, w.block, rows=rows, label=w.name)
