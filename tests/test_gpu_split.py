"""The split-key path (few streams, many keys) against the oracle and against
the one-pass kernels (GPU).

The split passes replay Alg. 1's per-block decisions from the block maxima,
so every T, P and reference equals the one-pass kernels': O and lse must
agree with them to fp32 summation order, and with the oracle to the usual
bar (rel-L2 2e-3, max-abs 1e-2, determined rows 2e-3)."""
import numpy as np
import pytest

import oracle as O
from helpers import check_parity, lse_agree, dev_bf16
from paper_2602_02071_amd.workloads import f32_to_bf16_bits, make_qkv

pytestmark = pytest.mark.gpu

SPLIT = [
    # B, Hq, Hkv, Sq, Sk, D, causal, block
    (1, 32, 8, 1, 32768, 128, False, 128),      # one long sequence: 8 streams, 256 blocks
    (1, 8, 2, 1, 5000 + 77, 64, False, 64),     # ragged key count
    (1, 4, 1, 8, 3000, 128, True, 128),         # causal chunk of 8 queries
    (2, 16, 2, 1, 2000, 128, False, 32),        # one wave per workgroup
    (1, 16, 1, 4, 4096, 64, True, 128),         # 64 rows, D 64
]


def _run(q, k, v, shape, block, split, **knobs):
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    o, lse = baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), causal, block, split=split, **knobs)
    torch.cuda.synchronize()
    return o.cpu().numpy().reshape(-1, D).astype(np.float64), lse.cpu().numpy().reshape(-1).astype(np.float64)


@pytest.mark.parametrize("shape", SPLIT, ids=lambda s: "x".join(map(str, s)))
def test_split_matches_oracle_and_one_pass(shape):
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal, block = shape
    assert baps.baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, block) > 0   # the split path is taken
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=sum(shape) + 11, outliers=True, lognormal_k=True)
    o, lse = _run(q, k, v, shape[:7], block, True)
    o1, lse1 = _run(q, k, v, shape[:7], block, False)
    fin = np.isfinite(lse1)
    assert np.array_equal(fin, np.isfinite(lse))
    assert np.abs(o - o1).max() <= 2e-5 * max(1.0, np.abs(o1).max())
    assert lse_agree(lse, lse1)
    check_parity(q, k, v, shape[:7], block, o, lse, label=f"split {shape}", same_kernels=False)


@pytest.mark.parametrize("lam,n_b0", [(0, 1), (8, 1), (-3, 2), (1, 7)])
def test_split_knobs(lam, n_b0):
    shape = (1, 8, 2, 1, 6000, 128, False)
    q, k, v = make_qkv(*shape[:6], seed=5 + lam, outliers=True, sink=2)
    o, lse = _run(q, k, v, shape, 128, True, lam=lam, n_b0=n_b0)
    o1, _ = _run(q, k, v, shape, 128, False, lam=lam, n_b0=n_b0)
    assert np.abs(o - o1).max() <= 2e-5 * max(1.0, np.abs(o1).max())
    check_parity(q, k, v, shape, 128, o, lse, label=f"split lam={lam} n_b0={n_b0}", lam=lam, n_b0=n_b0,
                 same_kernels=False)


def test_split_restart_counts():
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D = 1, 8, 2, 2, 9000, 128
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=61, outliers=True)
    cnt = torch.zeros((B * Hq, 2), dtype=torch.int64, device="cuda:0")
    cnt1 = torch.zeros_like(cnt)
    baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), True, 128, restart_counts=cnt, split=True)
    baps.attention(dev_bf16(q), dev_bf16(k), dev_bf16(v), True, 128, restart_counts=cnt1)
    torch.cuda.synchronize()
    assert torch.equal(cnt, cnt1)
    _, _, nr = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, True, 128)
    want = nr.reshape(B * Hq, Sq).sum(1)
    got = cnt.cpu().numpy()[:, 0]
    assert np.abs(got - want).max() <= max(2, 0.01 * want.max())


def _ramp_qkv(B, Hq, Hkv, Sq, Sk, D, seed):
    """Scores that climb along the keys: the running maximum of Alg. 1 moves
    at almost every block, so the replay takes its serial step nearly always."""
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((B, Hq, Sq, D)) * 0.3 + 1.0).astype(np.float32)
    k = rng.standard_normal((B, Hkv, Sk, D)).astype(np.float32) * 0.3
    k += (np.linspace(0.0, 3.0, Sk, dtype=np.float32)[None, None, :, None])
    v = rng.standard_normal((B, Hkv, Sk, D)).astype(np.float32)
    return f32_to_bf16_bits(q), f32_to_bf16_bits(k), f32_to_bf16_bits(v)


@pytest.mark.parametrize("block", [32, 64, 128])
def test_split_climbing_scores(block):
    shape = (1, 8, 2, 2, 9000, 128, True)
    q, k, v = _ramp_qkv(*shape[:6], seed=block)
    o, lse = _run(q, k, v, shape, block, True)
    o1, lse1 = _run(q, k, v, shape, block, False)
    assert np.abs(o - o1).max() <= 2e-5 * max(1.0, np.abs(o1).max())
    assert lse_agree(lse, lse1)
    check_parity(q, k, v, shape, block, o, lse, label=f"split climbing block={block}", same_kernels=False)


def test_split_long_context_many_windows():
    """More than 16384 key blocks: the splits are capped at 32 blocks each and
    the replay of the last split walks 1000+ LDS windows (against the one-pass
    kernel; the oracle samples a few rows)."""
    import paper_2602_02071_amd as baps
    shape = (1, 2, 1, 1, 600000, 64, False)
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    assert baps.baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, 32) > 0
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=3, outliers=True)
    o, lse = _run(q, k, v, shape, 32, True)
    o1, lse1 = _run(q, k, v, shape, 32, False)
    assert np.abs(o - o1).max() <= 2e-5 * max(1.0, np.abs(o1).max())
    assert lse_agree(lse, lse1)


def test_split_reused_dirty_workspace():
    """A workspace holding garbage (all bits set) and reused back to back
    gives the same bits every time."""
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, block = 1, 16, 4, 1, 20000, 128, 128
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=19, outliers=True)
    qd, kd, vd = dev_bf16(q), dev_bf16(k), dev_bf16(v)
    need = baps.baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, block)
    assert need > 0
    ws = torch.full((need,), 255, dtype=torch.uint8, device="cuda:0")
    outs = []
    for _ in range(3):
        o = torch.empty((B, Hq, Sq, D), dtype=torch.float32, device="cuda:0")
        lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device="cuda:0")
        baps.baps_attention_fwd_split(qd, kd, vd, o, lse, B, Hq, Hkv, Sq, Sk, D, False, block, ws, need)
        outs.append((o, lse))
    torch.cuda.synchronize()
    for o, lse in outs[1:]:
        assert torch.equal(o, outs[0][0]) and torch.equal(lse, outs[0][1])
    o1, lse1 = _run(q, k, v, (B, Hq, Hkv, Sq, Sk, D, False), block, False)
    assert np.abs(outs[0][0].cpu().numpy().reshape(-1, D) - o1).max() <= 2e-5 * max(1.0, np.abs(o1).max())


def test_library_loaded_before_the_gpu_is_initialised():
    """In a fresh process, load the library before torch touches the GPU, then
    call it: the runtime's start-up leaves an error behind that the library
    must not report as its own launch failure."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = (
        "import numpy as np, torch\n"
        "import paper_2602_02071_amd as baps\n"
        "baps.load()\n"
        "from paper_2602_02071_amd.workloads import make_qkv\n"
        "q, k, v = make_qkv(1, 8, 2, 1, 4096, 128, seed=1)\n"
        "dev = lambda x: torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to('cuda:0')\n"
        "o, lse = baps.attention(dev(q), dev(k), dev(v), False, 128, split=True)\n"
        "o1, lse1 = baps.attention(dev(q), dev(k), dev(v), False, 128)\n"
        "torch.cuda.synchronize()\n"
        "assert torch.allclose(o, o1, rtol=0, atol=2e-5), float((o - o1).abs().max())\n"
        "print('ok', flush=True)\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=180)
    assert r.returncode == 0 and "ok" in r.stdout, (r.stdout[-2000:], r.stderr[-2000:])
