"""The prefill kernel's work schedule (GPU).

With D = 128 the kernel runs a persistent grid: at most one workgroup per
resident slot, each taking a sequence of (query tile, key/value head, batch)
items.  These shapes have more items than the GPU holds at once, (batch, key/
value head) counts that are and are not multiples of 8, and ragged last
tiles.  O and lse start as NaN, so an item that is skipped (or a row written
by no item) shows; sampled rows, including the last row of every ragged
tile, are compared with the oracle to the usual bar."""
import numpy as np
import pytest

from helpers import check_parity, dev_bf16
from paper_2602_02071_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu

SHAPES = [
    # B, Hq, Hkv, Sq, Sk, D, causal, block: items = ceil(Sq*G/256) * B*Hkv
    (3, 6, 3, 5000, 5000, 128, True, 128),     # 9 heads, 40 tiles each (last one 16 rows): 360 items
    (2, 8, 4, 4500, 2100, 128, False, 64),     # 8 heads, 36 tiles each (last one 40 rows): 288 items
    (1, 40, 8, 3000, 3000, 128, True, 32),     # 8 heads, G = 5 (a tile splits query positions): 472 items
    (1, 32, 8, 4096, 4096, 128, True, 128),    # the Llama-3-8B prefill: 512 items, two per workgroup
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_persistent_schedule(shape):
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal, block = shape
    G = Hq // Hkv
    q, k, v = make_qkv(B, Hq, Hkv, Sq, Sk, D, seed=sum(shape), outliers=True)
    o = torch.full((B, Hq, Sq, D), float("nan"), dtype=torch.float32, device="cuda:0")
    lse = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device="cuda:0")
    cnt = torch.zeros((B * Hq, 2), dtype=torch.int64, device="cuda:0")
    print(f"persistent schedule {shape}: {-(-Sq * G // 256) * B * Hkv} items", flush=True)
    baps.baps_attention_fwd_ex(dev_bf16(q), dev_bf16(k), dev_bf16(v), o, lse, B, Hq, Hkv, Sq, Sk, D, causal, block,
                               restart_counts=cnt)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any(), "rows never written"
    assert not torch.isnan(lse).any(), "lse never written"
    # every (row, key block after the first) that a row sees is visited once:
    # an item run twice (or skipped) moves its heads' totals
    r = np.arange(Sq)
    kmax = np.minimum(Sk - 1, r + Sk - Sq) if causal else np.full(Sq, Sk - 1)
    want = int((np.clip(kmax, 0, None) // block).sum())
    assert np.all(cnt[:, 1].cpu().numpy() == want), (cnt[:, 1].cpu().numpy(), want)
    o = o.cpu().numpy().reshape(-1, D).astype(np.float64)
    lse = lse.cpu().numpy().reshape(-1).astype(np.float64)
    # per (batch, head): a few positions, plus the positions of the last
    # flattened row of every 256-row tile and the last query position
    last_of_tile = {min(Sq - 1, (t * 256 + 255) // G) for t in range(-(-Sq * G // 256))}
    pos = np.array(sorted(set(range(0, Sq, 997)) | last_of_tile | {Sq - 1}), np.int64)
    heads = range(0, Hq, max(1, Hq // 5))
    rows = np.concatenate([(b * Hq + h) * Sq + pos for b in range(B) for h in heads])
    check_parity(q, k, v, (B, Hq, Hkv, Sq, Sk, D, causal), block, o[rows], lse[rows], rows=rows,
                 label=f"persistent {shape}")
