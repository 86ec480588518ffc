"""The cast and output knobs of baps_params_t on the GPU (tie_mode,
saturate, out_bf16) and the verification entry point itself.

- Ties to even (App. A: HiF8 rounding; the canonical rule is ties away):
  integer scores put T exactly on HiF8 midpoints (|T| = 10, 20, ... in the
  one-bit binades), so the two rules give different O; both kernels must
  match the oracle run with the same rule, on the prefill and decode paths.
- bf16 O: each element is the round-to-nearest-even bf16 of the fp32 result
  of the same kernel, bit for bit, on every path (prefill, decode, split).
- saturate = 0 gives the same result as saturate = 1 wherever the library
  accepts it (no 8-bit P can exceed 2^15 below lambda 16).
"""
import numpy as np
import pytest

import oracle as O
from helpers import check_parity, dev_bf16
from paper_2602_02071_amd.workloads import f32_to_bf16_bits, make_qkv

pytestmark = pytest.mark.gpu


def _int_qkv(B, Hq, Hkv, Sq, Sk, D, seed):
    g = np.random.default_rng(seed)
    q = f32_to_bf16_bits(g.integers(-1, 2, (B, Hq, Sq, D)).astype(np.float32))
    k = f32_to_bf16_bits(g.integers(-1, 2, (B, Hkv, Sk, D)).astype(np.float32))
    v = f32_to_bf16_bits(g.standard_normal((B, Hkv, Sk, D)).astype(np.float32))
    return q, k, v


@pytest.mark.parametrize("shape,block", [((1, 4, 2, 200, 300, 64, True), 64), ((2, 8, 2, 1, 900, 128, False), 128),
                                         ((1, 4, 1, 130, 257, 128, False), 32)])
def test_ties_to_even(shape, block):
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    q, k, v = _int_qkv(B, Hq, Hkv, Sq, Sk, D, seed=Sk)
    args = (dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, block)
    oe, le = baps.attention(*args, scale_log2=1.0, tie_mode=baps.BAPS_TIES_EVEN)
    oa, _ = baps.attention(*args, scale_log2=1.0)
    torch.cuda.synchronize()
    assert float((oe - oa).abs().max()) > 1e-4            # the ties are really there
    oe = oe.cpu().numpy().reshape(-1, D).astype(np.float64)
    le = le.cpu().numpy().reshape(-1).astype(np.float64)
    check_parity(q, k, v, shape, block, oe, le, label=f"ties even, integer scores {shape}", scale_log2=1.0,
                 tie_even=True)
    # on ordinary scores ties are rare; the even kernels still meet the bar
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=Sk + 1, outliers=True)
    o, l = baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, block, tie_mode=baps.BAPS_TIES_EVEN)
    torch.cuda.synchronize()
    check_parity(q, k, v, shape, block, o.cpu().numpy().reshape(-1, D).astype(np.float64),
                 l.cpu().numpy().reshape(-1).astype(np.float64), label=f"ties even {shape}", tie_even=True)


@pytest.mark.parametrize("shape,block,split", [((1, 8, 2, 300, 333, 128, True), 128, False),
                                               ((2, 4, 4, 257, 257, 64, False), 64, False),
                                               ((3, 8, 2, 1, 1500, 128, False), 64, False),
                                               ((1, 32, 8, 1, 20000, 128, False), 128, True)])
def test_bf16_output_is_the_rounded_fp32_output(shape, block, split):
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=7 * Sk, outliers=True)
    args = (dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, block)
    o32, l32 = baps.attention(*args, split=split)
    o16, l16 = baps.attention(*args, split=split, out_bf16=True)
    torch.cuda.synchronize()
    assert o16.dtype == torch.bfloat16
    assert torch.equal(o16.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
    assert torch.equal(l16, l32)
    # and against the oracle, with bf16's rounding on top of the bar
    rows = np.arange(0, B * Hq * Sq, 7)
    o = o16.float().cpu().numpy().reshape(-1, D).astype(np.float64)[rows]
    ref, _, _ = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, rows=rows)
    assert np.linalg.norm(o - ref) / np.linalg.norm(ref) <= 2e-3 + 2.0 ** -8


def test_saturate_off_is_the_same_below_lambda_16():
    import torch
    import paper_2602_02071_amd as baps
    shape = (1, 8, 2, 256, 400, 128, True)
    q, k, v = make_qkv(*shape[:6], seed=3, outliers=True, sink=2)
    args = (dev_bf16(q), dev_bf16(k), dev_bf16(v), True, 128)
    for lam in (1, 8, 15):
        a, la = baps.attention(*args, lam=lam, saturate=True)
        b, lb = baps.attention(*args, lam=lam, saturate=False)
        torch.cuda.synchronize()
        assert torch.equal(a, b) and torch.equal(la, lb)
    with pytest.raises(baps.BapsError):
        baps.attention(*args, lam=16, saturate=False)


def test_dump_leaves_unseen_entries_and_matches_exact_scores():
    """The dump writes exactly the keys and blocks each selected row sees,
    and its sums lie within the fp32 summation bound of the exact q.k."""
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, block = 1, 4, 2, 70, 200, 64, 64
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=5, outliers=True)
    rows = np.array([0, 1, 69, 70 + 33, 3 * 70 + 69])
    o, lse, acc, ref = baps.attention_dump(dev_bf16(q), dev_bf16(k), dev_bf16(v), True, block, rows)
    torch.cuda.synchronize()
    acc, ref = acc.cpu().numpy(), ref.cpu().numpy()
    r = rows % Sq
    kmax = r + Sk - Sq
    for i in range(rows.size):
        assert np.all(np.isfinite(acc[i, :kmax[i] + 1])) and np.all(np.isnan(acc[i, kmax[i] + 1:]))
        nb = kmax[i] // block + 1
        assert np.all(np.isfinite(ref[i, :nb])) and np.all(np.isnan(ref[i, nb:]))
        assert np.all(ref[i, :nb] == np.round(ref[i, :nb]))         # integer references (Sec. 3.3)
        assert np.all(np.diff(ref[i, :nb]) >= 0)                     # never decrease
    bound = O.acc_bound(q, k, B, Hq, Hkv, Sq, Sk, D, rows)
    qf = (q.astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1, D)[rows]
    kf = (k.astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(Hkv, Sk, D)
    for i in range(rows.size):
        ex = kf[(rows[i] // Sq) // (Hq // Hkv)] @ qf[i]
        seen = slice(0, kmax[i] + 1)
        assert np.all(np.abs(acc[i, seen] - ex[seen]) <= bound[i, seen])
    o1, l1 = baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), True, block)
    torch.cuda.synchronize()
    assert torch.equal(o, o1) and torch.equal(lse, l1)


def test_workload2_full_size_ties_even_and_bf16_o():
    """Ties to even and bf16 O on the full Llama-3-8B-shaped prefill in the
    benchmark's launch configuration (the persistent grid): parity of the
    ties-to-even kernel on the sampled rows (every 64th query row of every
    head and the last row of each 128-row tile), and bf16 O equal, bit for
    bit, to the round-to-nearest-even of the fp32 O."""
    import torch
    import paper_2602_02071_amd as baps
    from paper_2602_02071_amd.workloads import make_workload, sample_rows
    w, q, k, v = make_workload(2)
    shape = (w.B, w.Hq, w.Hkv, w.Sq, w.Sk, w.D, w.causal)
    args = (dev_bf16(q), dev_bf16(k), dev_bf16(v), w.causal, w.block)
    oe, le = baps.attention(*args, tie_mode=baps.BAPS_TIES_EVEN)
    o32, l32 = baps.attention(*args)
    o16, l16 = baps.attention(*args, out_bf16=True)
    torch.cuda.synchronize()
    assert torch.equal(o16.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
    assert torch.equal(l16, l32)
    rows = sample_rows(w, every=64, tile=128)
    oe = oe.cpu().numpy().reshape(-1, w.D)[rows].astype(np.float64)
    le = le.cpu().numpy().reshape(-1)[rows].astype(np.float64)
    check_parity(q, k, v, shape, w.block, oe, le, rows=rows, label=f"ties even {w.name}", tie_even=True)
