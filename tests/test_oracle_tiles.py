"""Pins of the oracle's tile-level restart path (CPU only).

The paper takes the restart decision per tile of query rows (Sec. 3.2, Alg.
1) and counts restarts per tile (Sec. 4.3, Table 4); the canonical path of
this repository decides per row.  What fixes the tile path, other than its
own code:
- restart_rows = 1 reduces it exactly to the pinned per-row path;
- with the 8-bit casts removed it reduces to eq. (1) for every tile height,
  B0 choice and lambda (any restart pattern is exact without the casts);
- integer scores make every T and P exact, so the result is the base-2
  softmax attention whatever the tiles decide;
- where no B1 block can restart (lambda huge) or every one must (lambda very
  negative), tiles and rows agree;
- a hand-derived two-row case fixes which blocks restart and what is
  counted, with and without the last block in B0.
"""
import numpy as np
import pytest

import oracle as O
from paper_2602_02071_amd.workloads import bf16_bits_to_f32, f32_to_bf16_bits, make_qkv


def _args(B, Hq, Hkv, Sq, Sk, D, causal, seed=0, **kw):
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=seed, **kw)
    return (q, k, v, B, Hq, Hkv, Sq, Sk, D, causal)


@pytest.mark.parametrize("shape", [(2, 4, 2, 37, 300, 64, True, 64), (1, 2, 1, 50, 50, 16, False, 8),
                                   (1, 2, 2, 70, 33, 8, True, 16)])
@pytest.mark.parametrize("lam,n_b0", [(0, 1), (1, 1), (2, 2), (1, 0)])
def test_one_row_tiles_are_the_row_path(shape, lam, n_b0):
    B, Hq, Hkv, Sq, Sk, D, causal, block = shape
    args = _args(B, Hq, Hkv, Sq, Sk, D, causal, seed=5, outliers=True)
    o1, l1, n1, m1 = O.attention(*args, block, lam=lam, n_b0=n_b0, margin=True)
    o2, l2, n2, v2, m2 = O.attention(*args, block, lam=lam, n_b0=n_b0, margin=True, visits=True)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2) and np.array_equal(n1, n2)
    assert np.array_equal(m1, m2)
    assert np.all(n2 <= v2)


@pytest.mark.parametrize("R", [1, 2, 5, 16, 64])
@pytest.mark.parametrize("b0_last", [False, True])
@pytest.mark.parametrize("lam,n_b0", [(0, 1), (1, 1), (2, 0), (-3, 1)])
def test_tiles_quantizer_off_reduce_to_exact_attention(R, b0_last, lam, n_b0):
    args = _args(1, 2, 1, 45, 130, 16, True, seed=8, outliers=True)
    oe, le = O.exact_attention(*args)
    o, l, _ = O.attention(*args, 16, mode=O.E2E_EXACT, lam=lam, n_b0=n_b0, restart_rows=R, b0_last=b0_last)
    assert np.abs(o - oe).max() < 1e-12
    assert np.abs(l - le).max() < 1e-10


@pytest.mark.parametrize("R", [2, 8, 40])
@pytest.mark.parametrize("causal", [False, True])
def test_tiles_integer_scores_are_exact(R, causal):
    g = np.random.default_rng(21)
    B, H, Sq, Sk, D, block = 1, 2, 40, 57, 4, 8
    q = f32_to_bf16_bits(g.integers(-1, 2, (B, H, Sq, D)).astype(np.float32))
    k = f32_to_bf16_bits(g.integers(-1, 2, (B, H, Sk, D)).astype(np.float32))
    v = f32_to_bf16_bits(g.standard_normal((B, H, Sk, D)).astype(np.float32))
    o, l, _ = O.attention(q, k, v, B, H, H, Sq, Sk, D, causal, block, scale_log2=1.0, restart_rows=R, b0_last=True)
    qf, kf, vf = (bf16_bits_to_f32(x).astype(np.float64) for x in (q, k, v))
    s = np.einsum("bhqd,bhkd->bhqk", qf, kf)
    if causal:
        s = np.where(np.arange(Sk)[None, :] > (np.arange(Sq)[:, None] + Sk - Sq), -np.inf, s)
    w = np.exp2(s)
    want = (np.einsum("bhqk,bhkd->bhqd", w, vf) / w.sum(-1, keepdims=True)).reshape(-1, D)
    assert np.abs(o - want).max() < 1e-13
    assert np.abs(l - np.log(w.sum(-1)).reshape(-1)).max() < 1e-12


@pytest.mark.parametrize("lam", [1000, -1000])
def test_tiles_agree_with_rows_when_the_decision_is_fixed(lam):
    # lambda 1000: only forced blocks restart (block 0 for every row: causal
    # with Sq <= Sk); lambda -1000: every block restarts in both paths
    args = _args(1, 2, 1, 48, 200, 16, True, seed=9, outliers=True)
    o1, l1, _ = O.attention(*args, 16, lam=lam)
    o2, l2, _ = O.attention(*args, 16, lam=lam, restart_rows=16)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def _two_rows():
    """Two query rows, one head, D = 2, scale 1, blocks of 2 keys, not causal.
    q_A = (1, 0) and q_B = (0, 1), so row A's log2 scores are the first
    components of the keys and row B's the second:
        block 0: A (0, 0)  B (0, 0)   B0: both restart, m_A = m_B = 0
        block 1: A (0, 1)  B (5, 0)   A: T max 1, ceil 1 <= lambda 1, no restart, m_A = 1
                                      B: T max 5 > 1, restart, m_B = 5
        block 2: A (1, 0)  B (0, 0)   A: T max 0; B: T max -5: no restart
    Every score is an integer, so every P is exact."""
    one = lambda a: f32_to_bf16_bits(np.asarray(a, np.float32))
    q = one([[1, 0], [0, 1]]).reshape(1, 1, 2, 2)
    k = one([[0, 0], [0, 0], [0, 5], [1, 0], [1, 0], [0, 0]]).reshape(1, 1, 6, 2)
    v = one(np.arange(12).reshape(6, 2) - 5.0).reshape(1, 1, 6, 2)
    return q, k, v, 1, 1, 1, 2, 6, 2, False


def test_two_row_tile_hand_derived():
    args = _two_rows()
    # per row: A restarts in no B1 block (of 2), B in one (block 1)
    _, _, nr, nv = O.attention(*args, 2, scale_log2=1.0, visits=True)
    assert nr.tolist() == [0, 1] and nv.tolist() == [2, 2]
    # one tile of both rows: block 1 restarts for the tile (B's T exceeds lambda)
    o, _, nr, nv = O.attention(*args, 2, scale_log2=1.0, restart_rows=2, visits=True)
    assert nr.tolist() == [1, 1] and nv.tolist() == [2, 2]
    # with each row's last block in B0 as well, block 2 is forced: one B1 block left
    _, _, nr, nv = O.attention(*args, 2, scale_log2=1.0, restart_rows=2, b0_last=True, visits=True)
    assert nr.tolist() == [1, 1] and nv.tolist() == [1, 1]
    # every P is exact: the result is the base-2 softmax attention
    q, k, v = (bf16_bits_to_f32(x).astype(np.float64).reshape(-1, 2) for x in args[:3])
    w = np.exp2(q @ k.T)
    assert np.abs(o - (w @ v) / w.sum(1, keepdims=True)).max() < 1e-14


def test_tile_margin_is_shared_by_the_tile():
    args = _args(1, 2, 1, 40, 260, 64, True, seed=12, outliers=True)
    _, _, _, m1 = O.attention(*args, 64, margin=True)
    _, _, _, mt = O.attention(*args, 64, margin=True, restart_rows=8)
    mt = mt.reshape(2, 5, 8)
    assert np.all(mt == mt[:, :, :1])                  # one margin per tile
    assert np.all(np.isfinite(mt)) and np.all(mt >= 0)
    assert np.all(np.isfinite(m1)) and np.all(m1 >= 0)


def test_restart_rate_grows_with_tile_height():
    # a tile restarts when any of its rows would: over peaked inputs the
    # fraction of restarted B1 tile-blocks does not fall as tiles grow
    args = _args(1, 4, 1, 256, 1024, 64, True, seed=13, outliers=True)
    rates = []
    for R in (1, 4, 16, 64):
        _, _, nr, nv = O.attention(*args, 64, lam=1, restart_rows=R, visits=True)
        ntile = (256 + R - 1) // R
        nr_t, nv_t = nr.reshape(4, ntile, -1)[:, :, 0], nv.reshape(4, ntile, -1)[:, :, 0]
        rates.append(nr_t.sum() / nv_t.sum())
    assert all(b >= a - 0.02 for a, b in zip(rates, rates[1:])), rates
