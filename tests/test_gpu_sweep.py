"""Seeded random shapes through the library's own dispatch (GPU): batch, head
counts and grouping, query and key lengths (ragged against every tile and
block size), head dimension, causal or not, block size, the Alg. 1 knobs and
the input recipe are drawn per case, and every output row is judged by the
two-stage parity check of helpers.check_parity.  A second set draws
single-sequence and small-batch decode shapes that take the split-key path,
which must also agree with the one-pass kernels.  A third set draws one
setup per case on top of a random shape: the Default and Exp2 HiF8 softmax
setups, ties to even, tile-level restart, the diagonal B0 block, FP8 Q/K
(inputs without outlier channels) and bf16 O.  A fourth set draws group
sizes (query heads per key/value head) of 3 to 32, most not powers of two."""
import numpy as np
import pytest

import oracle as O
from helpers import check_parity, dev_bf16, lse_agree
from paper_2602_02071_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu

N_CASES = 24
N_SPLIT = 8
MAX_SCORES = 6_000_000          # B * Hq * Sq * Sk per case: the oracle finishes in about a second


def _draw(i):
    g = np.random.Generator(np.random.PCG64(9000 + i))
    while True:
        D = int(g.choice([64, 128]))
        block = int(g.choice([32, 64, 128]))
        Hkv = int(g.choice([1, 2, 4]))
        G = int(g.choice([1, 2, 4, 8]))
        B = int(g.integers(1, 4))
        decode_like = g.random() < 0.3
        Sq = int(g.integers(1, 17)) if decode_like else int(g.integers(1, 700))
        Sk = int(g.integers(1, 2500))
        causal = bool(g.random() < 0.5)
        if B * Hkv * G * Sq * Sk <= MAX_SCORES:
            break
    knobs = {}
    if g.random() < 0.3:
        knobs = dict(lam=int(g.choice([-1, 0, 2, 5])), n_b0=int(g.choice([0, 1, 2])))
    recipe = dict(outliers=bool(g.random() < 0.5), lognormal_k=bool(g.random() < 0.3),
                  sink=int(g.choice([0, 0, 4])))
    return (B, Hkv * G, Hkv, Sq, Sk, D, causal), block, knobs, recipe


def _run(q, k, v, shape, block, split=False, **knobs):
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    o, lse = baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, block, split=split, **knobs)
    torch.cuda.synchronize()
    return o.cpu().numpy().reshape(-1, D).astype(np.float64), lse.cpu().numpy().reshape(-1).astype(np.float64)


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape(i):
    shape, block, knobs, recipe = _draw(i)
    label = f"case {i}: shape {shape} block {block} knobs {knobs} inputs {recipe}"
    print(label, flush=True)
    q, k, v = make_qkv(*shape[:6], seed=700 + i, **recipe)
    o, lse = _run(q, k, v, shape, block, **knobs)
    check_parity(q, k, v, shape, block, o, lse, label=label, **knobs)


def _draw_split(i):
    import paper_2602_02071_amd as baps
    g = np.random.Generator(np.random.PCG64(9500 + i))
    while True:
        D = int(g.choice([64, 128]))
        block = int(g.choice([32, 64, 128]))
        Hkv = int(g.choice([1, 2, 4, 8]))
        G = int(g.choice([1, 2, 4, 8]))
        B = int(g.integers(1, 3))
        Sq = int(g.integers(1, max(2, 64 // G) + 1))
        Sk = int(g.integers(4 * block, 24000))
        causal = bool(g.random() < 0.5)
        shape = (B, Hkv * G, Hkv, Sq, Sk, D, causal)
        if (B * Hkv * G * Sq * Sk <= MAX_SCORES
                and baps.baps_attention_split_workspace(B, Hkv * G, Hkv, Sq, Sk, D, block) > 0):
            return shape, block


@pytest.mark.parametrize("i", range(N_SPLIT))
def test_random_split_shape(i):
    shape, block = _draw_split(i)
    label = f"split case {i}: shape {shape} block {block}"
    print(label, flush=True)
    q, k, v = make_qkv(*shape[:6], seed=800 + i, outliers=True, lognormal_k=bool(i % 2))
    o, lse = _run(q, k, v, shape, block, split=True)
    o1, lse1 = _run(q, k, v, shape, block)
    fin = np.isfinite(lse1)
    assert np.array_equal(fin, np.isfinite(lse))
    assert np.abs(o - o1).max() <= 2e-5 * max(1.0, np.abs(o1).max())
    assert lse_agree(lse, lse1)
    check_parity(q, k, v, shape, block, o, lse, label=label, same_kernels=False)


N_SETUP = 24
SETUPS = ("default", "exp2_hif8", "ties_even", "tiles", "b0_last", "fp8", "fp8_default", "out_bf16")


def _draw_setup(i):
    g = np.random.Generator(np.random.PCG64(9800 + i))
    setup = SETUPS[i % len(SETUPS)]
    shape, block, knobs, recipe = _draw(1000 + i)
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    G = Hq // Hkv
    if setup in ("ties_even", "fp8", "fp8_default") or "lam" in knobs and knobs["lam"] > 8:
        knobs = {}
    if setup == "tiles":
        R = int(g.choice([r for r in (2, 4, 8, 16, 32, 64) if r * G <= 256]))
        knobs = dict(knobs, restart_rows=R, b0_last=bool(g.random() < 0.5))
    elif setup == "b0_last":
        knobs = dict(knobs, b0_last=True)
    if setup.startswith("fp8"):
        recipe = dict(recipe, outliers=False)
    return setup, shape, block, knobs, recipe


@pytest.mark.parametrize("i", range(N_SETUP))
def test_random_setup(i):
    import torch
    import paper_2602_02071_amd as baps
    from paper_2602_02071_amd.workloads import make_qk_fp8
    setup, shape, block, knobs, recipe = _draw_setup(i)
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    label = f"setup case {i}: {setup} shape {shape} block {block} knobs {knobs} inputs {recipe}"
    print(label, flush=True)
    q, k, v = make_qkv(*shape[:6], seed=900 + i, **recipe)
    mode = {"default": O.DEFAULT, "exp2_hif8": O.EXP2_HIF8, "fp8_default": O.DEFAULT}.get(setup, O.E2E_HIF8)
    gkw = dict(knobs, mode=mode)
    okw = dict(knobs, mode=mode, pv_bf16=(mode == O.DEFAULT))
    if setup == "ties_even":
        gkw["tie_mode"] = baps.BAPS_TIES_EVEN
        okw["tie_even"] = True
    fp8 = None
    if setup.startswith("fp8"):
        q8, k8, qs, ks = make_qk_fp8(q, k)
        fp8 = (q8, k8, qs, ks)
        qt = torch.from_numpy(np.ascontiguousarray(q8)).to("cuda:0")
        kt = torch.from_numpy(np.ascontiguousarray(k8)).to("cuda:0")
        gkw["qk_scales"] = (qs, ks)
        q, k = O.e4m3_to_bf16(q8), O.e4m3_to_bf16(k8)
        okw["scale_log2"] = O.fp8_scale_log2(D, qs, ks)
    else:
        qt, kt = dev_bf16(q), dev_bf16(k)
    o, lse = baps.attention(qt, kt, dev_bf16(v), causal, block, out_bf16=(setup == "out_bf16"), **gkw)
    torch.cuda.synchronize()
    if setup == "out_bf16":
        o32, lse32 = baps.attention(qt, kt, dev_bf16(v), causal, block, **gkw)
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16))
        assert torch.equal(lse, lse32)
        o = o32
    o = o.float().cpu().numpy().reshape(-1, D).astype(np.float64)
    lse = lse.cpu().numpy().reshape(-1).astype(np.float64)
    check_parity(q, k, v, shape, block, o, lse, label=label, fp8=fp8, **okw)


N_GROUP = 12


def _draw_group(i):
    g = np.random.Generator(np.random.PCG64(9900 + i))
    while True:
        G = int(g.choice([3, 5, 6, 7, 12, 16, 32]))
        Hkv = int(g.choice([1, 2, 3]))
        B = int(g.integers(1, 3))
        Sq = int(g.choice([1, 2, 3, int(g.integers(4, 65)), int(g.integers(65, 400))]))
        Sk = int(g.integers(1, 3000))
        D = int(g.choice([64, 128]))
        block = int(g.choice([32, 64, 128]))
        causal = bool(g.random() < 0.5)
        if B * Hkv * G * Sq * Sk <= MAX_SCORES:
            return (B, Hkv * G, Hkv, Sq, Sk, D, causal), block


@pytest.mark.parametrize("i", range(N_GROUP))
def test_random_group_size(i):
    # query heads per key/value head that are not powers of two, and large
    # groups whose rows fill a tile from few query positions
    shape, block = _draw_group(i)
    label = f"group case {i}: shape {shape} block {block}"
    print(label, flush=True)
    q, k, v = make_qkv(*shape[:6], seed=1000 + i, outliers=bool(i % 2), lognormal_k=bool(i % 3 == 0))
    o, lse = _run(q, k, v, shape, block)
    check_parity(q, k, v, shape, block, o, lse, label=label)
