"""The no-allocation split-key entry point (GPU): the same kernels as
baps_attention_fwd_split on the library's static scratch.  Two calls in a
row, the second on a smaller input, each against the caller-workspace entry
point bit for bit and against the oracle; a shape whose workspace exceeds the
scratch is refused before any GPU work; a shape for the one-pass kernels
runs them."""
import numpy as np
import pytest

from helpers import check_parity, dev_bf16
from paper_2602_02071_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu


def _both(shape, block, seed, **knobs):
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=seed, outliers=True, lognormal_k=True)
    qt, kt, vt = dev_bf16(q), dev_bf16(k), dev_bf16(v)
    nbytes = baps.baps_attention_split_workspace(B, Hq, Hkv, Sq, Sk, D, block, **knobs)
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda:0")
    o1 = torch.full((B, Hq, Sq, D), float("nan"), device="cuda:0")
    l1 = torch.full((B, Hq, Sq), float("nan"), device="cuda:0")
    o2, l2 = torch.full_like(o1, float("nan")), torch.full_like(l1, float("nan"))
    baps.baps_attention_fwd_split(qt, kt, vt, o1, l1, B, Hq, Hkv, Sq, Sk, D, causal, block, ws, nbytes, **knobs)
    baps.baps_attention_fwd_split_noalloc(qt, kt, vt, o2, l2, B, Hq, Hkv, Sq, Sk, D, causal, block, **knobs)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    return (q, k, v), o2.cpu().numpy().reshape(-1, D).astype(np.float64), l2.cpu().numpy().reshape(-1).astype(np.float64)


def test_noalloc_twice_then_smaller():
    import paper_2602_02071_amd as baps
    big = (1, 32, 8, 1, 32768, 128, False)
    small = (1, 8, 2, 1, 6000, 128, False)
    assert 0 < baps.baps_attention_split_workspace(*big[:6], 128) <= baps.BAPS_SPLIT_SCRATCH_BYTES
    assert 0 < baps.baps_attention_split_workspace(*small[:6], 128)
    (q, k, v), o, lse = _both(big, 128, seed=31)
    rows = np.arange(0, 32, 3)
    check_parity(q, k, v, big, 128, o[rows], lse[rows], rows=rows, label="noalloc sk32768", same_kernels=False)
    (q, k, v), o, lse = _both(small, 128, seed=32)
    check_parity(q, k, v, small, 128, o, lse, label="noalloc sk6000", same_kernels=False)
    # knobs pass through (diagonal B0, lambda 0)
    (q, k, v), o, lse = _both(small, 64, seed=33, lam=0, b0_last=True)
    check_parity(q, k, v, small, 64, o, lse, label="noalloc sk6000 lam0 b0_last", lam=0, b0_last=True,
                 same_kernels=False)


def test_noalloc_one_pass_shapes_and_limit():
    import paper_2602_02071_amd as baps
    shape = (64, 32, 8, 1, 2048, 128, False)      # enough streams: the one-pass decode kernel
    assert baps.baps_attention_split_workspace(*shape[:6], 128) == 0
    (q, k, v), o, lse = _both(shape, 128, seed=34)
    rows = np.arange(0, 64 * 32, 17)
    check_parity(q, k, v, shape, 128, o[rows], lse[rows], rows=rows, label="noalloc one-pass", same_kernels=False)
    # a workspace beyond the scratch: refused before any GPU work
    big = (1, 2, 1, 1, 5_000_000, 64, False)
    assert baps.baps_attention_split_workspace(*big[:6], 32) > baps.BAPS_SPLIT_SCRATCH_BYTES
    with pytest.raises(baps.BapsError) as e:
        baps.baps_attention_fwd_split_noalloc(16, 16, 16, 16, None, *big, 32)
    assert e.value.status == baps.BAPS_UNSUPPORTED
