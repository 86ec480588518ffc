"""Pins of the oracle's attention and softmax-block steps (CPU only).

What fixes the oracle here, other than its own code:
- quantizer-off reduction: with the 8-bit casts removed, Alg. 1 under the
  consistent else-branch reading reduces exactly to eq. (1) for every
  lambda, B0 size and block size (and the literal reading does not);
- integer scores: every T and P is exact in HiF8, so the result equals the
  base-2 softmax attention computed with numpy;
- a hand-derived walk through Alg. 1 (tests/golden);
- integer-shift invariance, normalisation, row independence;
- a second, separately written closed-form evaluation on tiny shapes
  (consistency, not a pin);
- the paper's qualitative orderings (Table 1: Naive E2E far worse; Table 4:
  fewer restarts as lambda grows).
"""
import json
import os

import numpy as np
import pytest

import oracle as O
from paper_2602_02071_amd.workloads import bf16_bits_to_f32, f32_to_bf16_bits, make_qkv, random_scores

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _args(B, Hq, Hkv, Sq, Sk, D, causal, seed=0, **kw):
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=seed, **kw)
    return (q, k, v, B, Hq, Hkv, Sq, Sk, D, causal)


@pytest.mark.parametrize("shape", [
    (1, 2, 1, 70, 70, 16, True, 16),
    (2, 2, 2, 33, 100, 8, False, 32),
    (1, 4, 2, 100, 37, 8, True, 8),      # Sq > Sk: leading rows fully masked
    (1, 1, 1, 1, 300, 32, False, 64),
])
@pytest.mark.parametrize("lam,n_b0", [(0, 1), (1, 1), (2, 0), (1, 3), (-5, 1), (1000, 1)])
def test_quantizer_off_reduces_to_exact_attention(shape, lam, n_b0):
    B, Hq, Hkv, Sq, Sk, D, causal, block = shape
    args = _args(B, Hq, Hkv, Sq, Sk, D, causal, seed=3, outliers=True)
    oe, le = O.exact_attention(*args)
    o, l, _ = O.attention(*args, block, mode=O.E2E_EXACT, lam=lam, n_b0=n_b0)
    fin = np.isfinite(le)
    assert np.array_equal(fin, np.isfinite(l))
    assert np.abs(o - oe).max() < 1e-12
    assert np.abs(l[fin] - le[fin]).max() < 1e-10
    assert np.all(o[~fin] == 0) and np.all(l[~fin] == -np.inf)


def test_literal_else_branch_breaks_the_reduction():
    # the else-branch taken literally leaves the new block 2^delta too heavy
    args = _args(1, 2, 1, 64, 256, 16, False, seed=4)
    oe, _ = O.exact_attention(*args)
    o, _, _ = O.attention(*args, 16, mode=O.E2E_EXACT, lam=1, n_b0=1, literal_else=True)
    assert np.abs(o - oe).max() > 1e-3


def test_two_block_else_branch_closed_form():
    # two one-key blocks with log2 scores 0 and 0.875 (exact in bf16): the
    # second block takes the else-branch (ceil(0.875) = 1 <= lambda) and
    # raises m to 1; the softmax weights are 1/(1+2^0.875), 2^0.875/(1+2^0.875)
    one = int(f32_to_bf16_bits(np.array([1.0], np.float32))[0])
    q = np.array([one], np.uint16).reshape(1, 1, 1, 1)
    k = f32_to_bf16_bits(np.array([0.0, 0.875], np.float32)).reshape(1, 1, 2, 1)
    v = f32_to_bf16_bits(np.array([0.0, 1.0], np.float32)).reshape(1, 1, 2, 1)
    args = (q, k, v, 1, 1, 1, 1, 2, 1, False)
    w1 = 2 ** 0.875 / (1 + 2 ** 0.875)
    o, _, nr = O.attention(*args, 1, mode=O.E2E_EXACT, lam=1, n_b0=1, scale_log2=1.0)
    assert nr[0] == 0 and abs(o[0, 0] - w1) < 1e-15
    o, _, _ = O.attention(*args, 1, mode=O.E2E_EXACT, lam=1, n_b0=1, scale_log2=1.0, literal_else=True)
    w1_lit = 2 ** 0.875 / (0.5 + 2 ** 0.875)
    assert abs(o[0, 0] - w1_lit) < 1e-15 and abs(w1_lit - w1) > 0.1


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("lam,n_b0,block", [(1, 1, 8), (0, 1, 4), (2, 2, 16), (1, 0, 8)])
def test_integer_scores_are_exact(causal, lam, n_b0, block):
    # entries in {-1,0,1}, D = 4, scale 1: S = q.k is an integer in [-4, 4], so
    # T = S - ref is an integer >= -13, exact in HiF8, and 2^T is exact
    g = np.random.default_rng(11)
    B, H, Sq, Sk, D = 1, 3, 40, 57, 4
    q = f32_to_bf16_bits(g.integers(-1, 2, (B, H, Sq, D)).astype(np.float32))
    k = f32_to_bf16_bits(g.integers(-1, 2, (B, H, Sk, D)).astype(np.float32))
    v = f32_to_bf16_bits(g.standard_normal((B, H, Sk, D)).astype(np.float32))
    o, l, _ = O.attention(q, k, v, B, H, H, Sq, Sk, D, causal, block, lam=lam, n_b0=n_b0, scale_log2=1.0)
    qf, kf, vf = (bf16_bits_to_f32(x).astype(np.float64) for x in (q, k, v))
    s = np.einsum("bhqd,bhkd->bhqk", qf, kf)
    if causal:
        mask = np.arange(Sk)[None, :] > (np.arange(Sq)[:, None] + Sk - Sq)
        s = np.where(mask, -np.inf, s)
    w = np.exp2(s)
    want = (np.einsum("bhqk,bhkd->bhqd", w, vf) / w.sum(-1, keepdims=True)).reshape(-1, D)
    lse = (np.log(w.sum(-1))).reshape(-1)
    assert np.abs(o - want).max() < 1e-13
    assert np.abs(l - lse).max() < 1e-12


def test_golden_walkthrough():
    g = json.load(open(os.path.join(GOLDEN, "softmax_block_walkthrough.json")))
    s = np.array([g["scores"]], np.float32)
    for c in g["cases"]:
        codes, refs, m, d, rs = O.softmax_block(s, g["block"], c["lambda"], g["n_b0"])
        assert O.hif8_decode(codes[0]).tolist() == c["p_values"]
        assert refs[0].tolist() == c["ref_shift"]
        assert rs[0].tolist() == c["restarted"]
        assert m[0] == c["m_final"] and d[0] == c["d_final"]


def _phat(codes, refs, d, block):
    p = O.hif8_decode(codes)
    cols = codes.shape[1]
    sh = np.repeat(refs, block, axis=1)[:, :cols].astype(np.float64)
    sh = np.where(refs.repeat(block, axis=1)[:, :cols] == np.iinfo(np.int32).min, -np.inf, sh)
    with np.errstate(invalid="ignore", divide="ignore"):
        return p * np.exp2(sh) / d[:, None]


def test_softmax_block_normalised_and_shift_invariant():
    s = random_scores(64, 333, seed=1, std=6.0, masked_frac=0.05)
    s = (np.round(s * 64) / 64).astype(np.float32)          # dyadic: S + k stays exact
    codes, refs, m, d, rs = O.softmax_block(s, 32, 1, 1)
    ph = _phat(codes, refs, d, 32)
    assert np.abs(ph.sum(1) - 1).max() < 1e-13
    assert np.all(ph[np.isinf(s)] == 0)
    for k in (1, 7, -13):
        c2, r2, m2, d2, rs2 = O.softmax_block(s + np.float32(k), 32, 1, 1)
        assert np.array_equal(c2, codes) and np.array_equal(r2, refs) and np.array_equal(rs2, rs)
        assert np.array_equal(m2, m + k) and np.array_equal(d2, d)


def test_softmax_block_degenerate_rows():
    s = np.full((3, 10), -np.inf, np.float32)
    s[1, 7] = 2.5                       # first finite score in block 1 (n_b0 = 1)
    s[2, :] = 0.0
    codes, refs, m, d, rs = O.softmax_block(s, 4, 1, 1)
    assert m[0] == -np.inf and d[0] == 0 and np.all(codes[0] == 0)
    assert np.all(refs[0] == np.iinfo(np.int32).min)
    # row 1: block 0 has nothing; block 1 restarts from m = -inf
    assert rs[1].tolist() == [1, 1, 0] and m[1] == 3.0
    assert O.hif8_decode(codes[1, 7]) == O.hif8_decode(O.exp2_table(0)[O.hif8_encode_scalar(-0.5)])
    assert refs[1].tolist()[1:] == [0, 0]
    ph = _phat(codes, refs, d, 4)
    assert abs(ph[1].sum() - 1) < 1e-15 and abs(ph[2].sum() - 1) < 1e-15


def test_rows_independent_and_subset_exact():
    args = _args(1, 4, 2, 96, 96, 32, True, seed=5, outliers=True)
    o, l, nr = O.attention(*args, 32)
    rows = np.array([5, 95, 96 + 17, 3 * 96 + 40], np.int64)
    o2, l2, nr2 = O.attention(*args, 32, rows=rows)
    assert np.array_equal(o[rows], o2) and np.array_equal(l[rows], l2) and np.array_equal(nr[rows], nr2)
    o1, _, _ = O.attention(*args, 32, nthreads=1)
    assert np.array_equal(o1, o)


# --- a second evaluation, written separately, for tiny shapes --------------------------
def _closed_form_row(qr, K, V, c32, block, lam, n_b0, kmax):
    vals = O.hif8_decode(np.arange(256))
    fin = np.sort(vals[np.isfinite(vals)])

    def q8(x):
        if x == -np.inf:
            return -np.inf
        if x == np.inf:
            return np.inf
        a = abs(x)
        if a >= fin[-1]:
            return np.copysign(fin[-1], x)
        i = np.searchsorted(fin, a, side="right") - 1
        lo, hi = fin[i], fin[i + 1]
        r = hi if a >= (lo + hi) / 2 else lo
        return np.copysign(r, x) if r != 0 else 0.0

    def e8(t):
        return 0.0 if t == -np.inf else q8(2.0 ** t)

    acc = np.array([np.float32(np.dot(qr, K[c])) for c in range(kmax + 1)], np.float32)
    m = -np.inf
    refs = []
    for j in range(kmax // block + 1):
        a = acc[j * block: min((j + 1) * block, kmax + 1)]
        amax = np.max(a)
        M = float(np.float32(amax) * np.float32(c32))
        if j >= n_b0 and m != -np.inf:
            tq = q8(float(np.float32(np.float64(amax) * c32 - m)))
            if np.ceil(tq) <= lam:
                refs.append(m)
                m = m + max(0.0, np.ceil(tq))
                continue
        m = max(m, np.ceil(M))
        refs.append(m)
    w = np.array([2.0 ** (refs[c // block] - m) * e8(q8(float(np.float32(
        np.float64(acc[c]) * np.float64(np.float32(c32)) - refs[c // block]))))
        for c in range(kmax + 1)])
    return (w[:, None] * V[: kmax + 1]).sum(0) / w.sum()


def test_tiny_shapes_closed_form():
    rng = np.random.default_rng(12)
    for trial in range(25):
        Sq, Sk, D = int(rng.integers(1, 9)), int(rng.integers(1, 9)), int(rng.integers(1, 5))
        block = int(rng.integers(1, 4))
        lam, n_b0 = int(rng.integers(-1, 3)), int(rng.integers(0, 3))
        causal = bool(rng.integers(0, 2))
        q, k, v = make_qkv(1, 1, 1, Sq, Sk, D, seed=100 + trial, q_scale=3.0, k_scale=3.0)
        o, _, _ = O.attention(q, k, v, 1, 1, 1, Sq, Sk, D, causal, block, lam=lam, n_b0=n_b0)
        qf, kf, vf = (bf16_bits_to_f32(x)[0, 0].astype(np.float64) for x in (q, k, v))
        c32 = float(np.float32(np.log2(np.e) / np.sqrt(D)))
        for r in range(Sq):
            kmax = min(Sk - 1, r + Sk - Sq) if causal else Sk - 1
            if kmax < 0:
                assert np.all(o[r] == 0)
                continue
            want = _closed_form_row(qf[r], kf, vf, c32, block, lam, n_b0, kmax)
            assert np.abs(o[r] - want).max() < 1e-12, (trial, r)


# --- the paper's qualitative results on synthetic data -----------------------------
@pytest.fixture(scope="module")
def peaked():
    args = _args(1, 4, 1, 512, 512, 128, True, seed=7, outliers=True)
    oe, _ = O.exact_attention(*args)
    return args, oe


def _rel(o, oe):
    return np.linalg.norm(o - oe) / np.linalg.norm(oe)


def test_naive_e2e_much_worse(peaked):
    # Table 1 / Fig. 3: casting the scores to 8 bits before the max subtraction
    # degrades far more than E2E HiF8 or Exp2 HiF8
    args, oe = peaked
    e2e = _rel(O.attention(*args, 128, mode=O.E2E_HIF8)[0], oe)
    exp2 = _rel(O.attention(*args, 128, mode=O.EXP2_HIF8)[0], oe)
    naive = _rel(O.attention(*args, 128, mode=O.NAIVE_E2E)[0], oe)
    dflt = _rel(O.attention(*args, 128, mode=O.DEFAULT)[0], oe)
    assert dflt < 1e-5
    assert naive > 10 * e2e and naive > 10 * exp2
    assert e2e < 3 * exp2


def test_restarts_fall_as_lambda_grows(peaked):
    # Table 4: raising the restart threshold lowers the restart rate
    args, _ = peaked
    counts = [O.attention(*args, 128, lam=lam)[2].sum() for lam in (0, 1, 2, 4)]
    assert all(a >= b for a, b in zip(counts, counts[1:])) and counts[0] > counts[-1]


def _exact_acc(q, k, B, Hq, Hkv, Sq, Sk, D, rows=None):
    """fl32 of the exact dot products q.k of every requested row, [n, Sk]."""
    rows = np.arange(B * Hq * Sq) if rows is None else np.asarray(rows)
    qf = bf16_bits_to_f32(q).astype(np.float64).reshape(B * Hq * Sq, D)[rows]
    kf = bf16_bits_to_f32(k).astype(np.float64).reshape(B, Hkv, Sk, D)
    b, g = rows // (Hq * Sq), (rows // Sq) % Hq // (Hq // Hkv)
    return np.stack([kf[b[i], g[i]] @ qf[i] for i in range(rows.size)])


def _valid_acc(q, k, shape, t, seed):
    """Another valid high-precision S: every dot product moved by t (|t| < 1)
    times its accumulation error bound, with random signs for seed > 0."""
    B, Hq, Hkv, Sq, Sk, D = shape
    ex = _exact_acc(q, k, B, Hq, Hkv, Sq, Sk, D)
    bound = O.acc_bound(q, k, B, Hq, Hkv, Sq, Sk, D, np.arange(B * Hq * Sq))
    sgn = np.random.default_rng(seed).choice([-1.0, 1.0], ex.shape) if seed else 1.0
    return (ex + t * sgn * bound).astype(np.float32)


def test_acc_bound_is_the_summation_bound():
    # gamma_(D-1) * sum |q_d k_d|: at D = 1 a single exact product (zero), and
    # fp32 sums of the exact products in two orders stay within it
    q, k, _, *shape = _args(1, 2, 1, 16, 40, 64, False, seed=21, outliers=True)
    B, Hq, Hkv, Sq, Sk, D, _ = shape
    bound = O.acc_bound(q, k, B, Hq, Hkv, Sq, Sk, D, np.arange(B * Hq * Sq))
    ex = _exact_acc(q, k, B, Hq, Hkv, Sq, Sk, D)
    qf = bf16_bits_to_f32(q).reshape(Hq * Sq, D)
    kf = bf16_bits_to_f32(k).reshape(Sk, D)
    prods = (qf[:, None, :] * kf[None, :, :]).astype(np.float32)          # exact in fp32
    fwd = np.zeros(prods.shape[:2], np.float32)
    for d in range(D):
        fwd += prods[:, :, d]
    pair = prods
    while pair.shape[2] > 1:
        pair = (pair[:, :, 0::2] + pair[:, :, 1::2]).astype(np.float32)
    for s in (fwd, pair[:, :, 0]):
        assert np.all(np.abs(s.astype(np.float64) - ex) <= bound)
    q1, k1, _, *sh1 = _args(1, 1, 1, 4, 5, 1, False, seed=2)
    assert np.all(O.acc_bound(q1, k1, 1, 1, 1, 4, 5, 1, np.arange(4)) == 0.0)


def test_given_scores_reproduce_the_oracle():
    # feeding fl32 of the exact dot products back in is the canonical result,
    # bit for bit, in every setup and on the tile path
    args = _args(1, 4, 2, 50, 130, 32, True, seed=5, outliers=True)
    q, k, v, B, Hq, Hkv, Sq, Sk, D, causal = args
    acc = _exact_acc(q, k, B, Hq, Hkv, Sq, Sk, D).astype(np.float32)
    for kw in (dict(), dict(mode=O.EXP2_HIF8), dict(mode=O.DEFAULT, pv_bf16=True), dict(lam=0, n_b0=2),
               dict(restart_rows=8, b0_last=True), dict(tie_even=True)):
        o0, l0, r0 = O.attention(*args, 32, **kw)[:3]
        o1, l1, r1 = O.attention(*args, 32, acc=acc, **kw)[:3]
        assert np.array_equal(o0, o1) and np.array_equal(l0, l1) and np.array_equal(r0, r1), kw
    # a tile needs every one of its rows
    with pytest.raises(ValueError):
        O.attention(*args, 32, rows=np.arange(3), acc=acc[:3], restart_rows=8)


def test_given_scores_are_used():
    # doubling one row's scores (scale 1, integer scores) is the row with
    # doubled scores
    g = np.random.default_rng(4)
    q = f32_to_bf16_bits(g.integers(-1, 2, (1, 1, 3, 4)).astype(np.float32))
    k = f32_to_bf16_bits(g.integers(-1, 2, (1, 1, 20, 4)).astype(np.float32))
    v = f32_to_bf16_bits(g.standard_normal((1, 1, 20, 4)).astype(np.float32))
    q2 = f32_to_bf16_bits(2 * bf16_bits_to_f32(q))
    acc2 = _exact_acc(q2, k, 1, 1, 1, 3, 20, 4).astype(np.float32)
    want, _, _ = O.attention(q2, k, v, 1, 1, 1, 3, 20, 4, False, 8, scale_log2=1.0)
    got, _, _ = O.attention(q, k, v, 1, 1, 1, 3, 20, 4, False, 8, scale_log2=1.0, acc=acc2)
    assert np.array_equal(got, want)


def test_refs_are_the_softmax_block_references():
    # on integer scores (S exact in fp32) the per-block references of the
    # fused row equal those of the standalone vector-side step
    # (ref_shift + m_final), which the hand-derived walkthrough pins
    g = np.random.default_rng(6)
    Sq, Sk, D, blk = 6, 200, 4, 16
    q = f32_to_bf16_bits(g.integers(-3, 4, (1, 1, Sq, D)).astype(np.float32))
    k = f32_to_bf16_bits(g.integers(-3, 4, (1, 1, Sk, D)).astype(np.float32))
    v = f32_to_bf16_bits(g.standard_normal((1, 1, Sk, D)).astype(np.float32))
    for lam in (0, 1, 2):
        _, _, _, refs = O.attention(q, k, v, 1, 1, 1, Sq, Sk, D, False, blk, lam=lam, scale_log2=1.0,
                                    refs=True)
        s = _exact_acc(q, k, 1, 1, 1, Sq, Sk, D).astype(np.float32)
        _, shift, m, _, _ = O.softmax_block(s, blk, lam=lam)
        assert np.array_equal(refs, shift + m[:, None])
    # causal: blocks a row does not see stay NaN
    _, _, _, refs = O.attention(q, k, v, 1, 1, 1, Sq, Sk, D, True, blk, scale_log2=1.0, refs=True)
    for r in range(Sq):
        nb = (r + Sk - Sq) // blk + 1
        assert np.all(np.isfinite(refs[r, :nb])) and np.all(np.isnan(refs[r, nb:]))
    # eq. (2) setups: the running maximum after each block, non-decreasing
    _, _, _, mref = O.attention(q, k, v, 1, 1, 1, Sq, Sk, D, False, blk, mode=O.DEFAULT, scale_log2=1.0,
                                refs=True)
    s64 = s.astype(np.float64)
    for j in range(mref.shape[1]):
        assert np.array_equal(mref[:, j], s64[:, :(j + 1) * blk].max(axis=1))


def test_margin_marks_rows_stable_under_valid_scores():
    # a row whose decisions all clear their rounding boundaries by the
    # accumulation error bound keeps its result for every valid
    # high-precision S; ambiguous rows exist and may move
    args = _args(1, 4, 2, 200, 400, 128, True, seed=13, outliers=True)
    q, k = args[0], args[1]
    o, _, _, mg = O.attention(*args, 32, margin=True)
    det = mg >= 1
    assert det.sum() > 0.7 * det.size
    moved_amb = 0
    for t, seed in ((0.99, 0), (-0.99, 0), (0.7, 3), (0.99, 9)):
        oj, _, _ = O.attention(*args, 32, acc=_valid_acc(q, k, (1, 4, 2, 200, 400, 128), t, seed))
        diff = np.abs(oj - o).max(axis=1)
        # (a T of weight below 2^-12 of the row maximum may still round the
        # other way: the margin leaves those out, they move O by < 1e-3)
        assert diff[det].max() <= 1e-3
        moved_amb += int((diff[~det] > 1e-3).sum())
    assert moved_amb > 0


def test_exp2_hif8_margin_marks_rows_stable_under_valid_scores():
    # Exp2 HiF8 (eq. 2 with the exp2 in 8 bits): rows whose HiF8 roundings
    # all clear their boundaries by the accumulation error bound give the
    # same 8-bit P and alpha, hence the same O, for every valid high-precision S
    args = _args(1, 4, 2, 160, 300, 128, True, seed=17, outliers=True)
    q, k = args[0], args[1]
    shape = (1, 4, 2, 160, 300, 128)
    o, _, _, mg = O.attention(*args, 64, mode=O.EXP2_HIF8, margin=True)
    det = mg >= 1
    assert det.sum() > 0.5 * det.size
    moved_amb = 0
    for t, seed in ((0.99, 0), (-0.99, 0), (0.7, 3), (0.99, 9)):
        oj, _, _ = O.attention(*args, 64, mode=O.EXP2_HIF8, acc=_valid_acc(q, k, shape, t, seed))
        diff = np.abs(oj - o).max(axis=1)
        assert diff[det].max() <= 1e-5
        moved_amb += int((diff[~det] > 1e-5).sum())
    assert moved_amb > 0
    # the Default setup has no 8-bit decision: every row is determined,
    # unless P is rounded to bf16 for the P V product, whose roundings are
    # decisions as well (and the same rule holds for them)
    _, _, _, mgd = O.attention(*args, 64, mode=O.DEFAULT, margin=True)
    assert np.all(np.isinf(mgd))
    od, _, _, mgb = O.attention(*args, 64, mode=O.DEFAULT, margin=True, pv_bf16=True)
    detb = mgb >= 1
    assert 0.2 * detb.size < detb.sum() < detb.size
    for t, seed in ((0.99, 0), (-0.99, 0), (0.99, 9)):
        oj, _, _ = O.attention(*args, 64, mode=O.DEFAULT, pv_bf16=True, acc=_valid_acc(q, k, shape, t, seed))
        # a moved score moves P continuously (here up to ~3e-3 relative: the
        # outlier channels make the accumulation bound large); a bf16 flip of
        # a dominant P would move O by ~2^-8 |v| more
        assert np.abs(oj - od).max(axis=1)[detb].max() <= 4e-3


def test_pv_bf16_rounding_bound():
    # pv_bf16 rounds each P to bf16 (relative error <= 2^-9) only inside the
    # P V product: O moves by at most 2^-9 * sum_c p_c |v_c| / d, and not at
    # all when every P is a power of two (integer scores)
    q, k, v, *shape = _args(1, 2, 1, 40, 90, 32, True, seed=23)
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    o32, _, _ = O.attention(q, k, v, *shape, 32, mode=O.DEFAULT)
    o16, _, _ = O.attention(q, k, v, *shape, 32, mode=O.DEFAULT, pv_bf16=True)
    vmax = np.abs(bf16_bits_to_f32(v)).max()
    assert 0 < np.abs(o16 - o32).max() <= 2.0 ** -9 * vmax * 1.01
    g = np.random.default_rng(3)
    qi = f32_to_bf16_bits(g.integers(-1, 2, (1, 2, 40, 32)).astype(np.float32))
    ki = f32_to_bf16_bits(g.integers(-1, 2, (1, 1, 90, 32)).astype(np.float32))
    a32, _, _ = O.attention(qi, ki, v, *shape, 32, mode=O.DEFAULT, scale_log2=1.0)
    a16, _, _ = O.attention(qi, ki, v, *shape, 32, mode=O.DEFAULT, scale_log2=1.0, pv_bf16=True)
    assert np.array_equal(a32, a16)
