"""Tile-level restart (the paper's granularity) on the GPU against the oracle.

The restart decision is shared by the rows of one head at restart_rows
consecutive query positions (Sec. 3.2); B0 can also hold each row's last
visible block (b0_last).  Cases cover tiles inside one wave of the prefill
kernel (restart_rows * G <= 32), tiles spanning several waves, tiles inside
the decode kernel's 16 rows, a tile too tall for it (the prefill kernel takes
the call), the full score table (lambda > 8) and the per-tile counters
behind Table 4's restart rates."""
import numpy as np
import pytest

import oracle as O
from helpers import check_parity, dev_bf16, gpu_attention
from paper_2602_02071_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu


def _check(shape, block, R, b0_last=False, seed=0, **knobs):
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=seed, outliers=True, lognormal_k=True)
    o, lse = gpu_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, restart_rows=R, b0_last=b0_last,
                           **knobs)
    return check_parity(q, k, v, shape, block, o, lse, label=f"{shape} R={R} b0_last={b0_last} {knobs}",
                        restart_rows=R, b0_last=b0_last, **knobs)


PREFILL = [
    # B, Hq, Hkv, Sq, Sk, D, causal, block, R
    ((1, 8, 2, 256, 256, 64, True), 64, 2),         # G 4: 8 rows per tile, one wave
    ((1, 8, 2, 256, 256, 64, True), 64, 8),         # 32 rows: a whole wave
    ((1, 8, 2, 256, 256, 64, True), 64, 16),        # 64 rows: two waves
    ((1, 8, 2, 200, 256, 128, True), 128, 64),      # 256 rows: the whole workgroup, ragged Sq
    ((1, 4, 4, 300, 300, 128, True), 128, 32),      # MHA: 32 rows
    ((1, 4, 4, 300, 333, 128, True), 128, 128),     # MHA: 4 waves, ragged
    ((2, 16, 2, 70, 150, 128, False), 32, 4),       # G 8: 32 rows
    ((2, 16, 2, 70, 150, 128, False), 32, 32),      # G 8: 256 rows
]


@pytest.mark.parametrize("case", PREFILL, ids=lambda c: "x".join(map(str, c[0])) + f"-b{c[1]}-R{c[2]}")
@pytest.mark.parametrize("b0_last", [False, True])
def test_prefill_tiles(case, b0_last):
    shape, block, R = case
    _check(shape, block, R, b0_last, seed=sum(shape) + R)


@pytest.mark.parametrize("lam,n_b0", [(0, 1), (2, 2), (9, 1)])
def test_prefill_tiles_knobs(lam, n_b0):
    _check((1, 8, 2, 128, 384, 128, True), 128, 16, True, seed=lam + 40, lam=lam, n_b0=n_b0)


DECODE = [
    ((2, 8, 2, 4, 1000, 128, True), 128, 4),        # 16 rows: the decode kernel's tile
    ((2, 8, 2, 4, 1000, 128, True), 64, 2),         # 8 rows
    ((1, 4, 1, 16, 640, 64, True), 64, 4),          # 64 flattened rows, 4 decode tiles
    ((1, 4, 1, 16, 640, 128, True), 64, 8),         # 32 rows per tile: taken by the prefill kernel
    ((3, 8, 2, 1, 777, 64, False), 64, 16),         # Sq = 1: a tile is one row
]


@pytest.mark.parametrize("case", DECODE, ids=lambda c: "x".join(map(str, c[0])) + f"-b{c[1]}-R{c[2]}")
@pytest.mark.parametrize("b0_last", [False, True])
def test_decode_tiles(case, b0_last):
    shape, block, R = case
    _check(shape, block, R, b0_last, seed=sum(shape) + 3 * R)


@pytest.mark.parametrize("shape,block,R", [((1, 8, 2, 256, 512, 128, True), 128, 16),
                                           ((2, 8, 2, 4, 2000, 128, True), 128, 4),
                                           ((1, 8, 2, 64, 700, 64, True), 64, 1),
                                           # ragged causal offsets: a block boundary falls
                                           # inside a tile that spans two waves, so the
                                           # tile's first wave sees nothing of a block its
                                           # second wave sees
                                           ((1, 8, 2, 250, 512, 128, True), 128, 16),
                                           ((1, 4, 4, 300, 301, 128, True), 128, 64)])
def test_tile_counters(shape, block, R):
    """Per-tile restarted / visited B1 blocks against the oracle: equal on
    every tile whose decisions are clear of a rounding boundary."""
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=R + 70, outliers=True)
    ntq = (Sq + R - 1) // R
    tc = torch.zeros((B * Hq * ntq, 2), dtype=torch.int64, device="cuda:0")
    hc = torch.zeros((B * Hq, 2), dtype=torch.int64, device="cuda:0")
    baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, block, restart_rows=R, b0_last=True,
                   tile_counts=tc, restart_counts=hc)
    torch.cuda.synchronize()
    tc, hc = tc.cpu().numpy(), hc.cpu().numpy()
    _, _, nr, nv, mg = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, restart_rows=R, b0_last=True,
                                   visits=True, margin=True)
    first = np.arange(B * Hq * Sq).reshape(B * Hq, Sq)[:, ::R].reshape(-1)   # one row per tile
    want = np.stack([nr[first], nv[first]], 1)
    clear = mg[first] >= 1.0
    assert np.array_equal(tc[:, 1], want[:, 1])                               # visits never depend on rounding
    assert np.array_equal(tc[clear, 0], want[clear, 0]), (tc[clear][:8], want[clear][:8])
    assert np.abs(tc[:, 0] - want[:, 0]).max() <= 2
    assert np.array_equal(hc, tc.reshape(B * Hq, ntq, 2).sum(1))


def test_split_path_with_diagonal_b0():
    """The split-key path replays B0 = {first, last} per row (Sq = 1)."""
    import torch
    import paper_2602_02071_amd as baps
    shape = (1, 32, 8, 1, 20000, 128, False)
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    assert baps.baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, 128, b0_last=True) > 0
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=99, outliers=True, lognormal_k=True)
    c1 = torch.zeros((B * Hq, 2), dtype=torch.int64, device="cuda:0")
    c2 = torch.zeros_like(c1)
    o, lse = baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, 128, split=True, b0_last=True,
                            tile_counts=c1)
    o1, _ = baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, 128, b0_last=True, tile_counts=c2)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)
    assert float((o - o1).abs().max()) <= 2e-5 * max(1.0, float(o1.abs().max()))
    check_parity(q, k, v, shape, 128, o.cpu().numpy().reshape(-1, D).astype(np.float64),
                 lse.cpu().numpy().reshape(-1).astype(np.float64), label="split b0_last", b0_last=True,
                 same_kernels=False)
