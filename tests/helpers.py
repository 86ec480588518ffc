"""Shared helpers of the GPU tests: move seeded inputs to the device, run the
library, compare with the oracle."""
import numpy as np

REL_L2_TOL = 2e-3     # O within relative L2 2e-3 of the oracle
MAX_ABS_TOL = 1e-2    # and max abs error 1e-2


def dev_bf16(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to("cuda:0")


def gpu_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, **knobs):
    """Run the fused pass on cuda:0; returns (o [B*Hq*Sq, D] fp64, lse fp64)."""
    import torch
    import paper_2602_02071_amd as baps
    qt, kt, vt = dev_bf16(q), dev_bf16(k), dev_bf16(v)
    o, lse = baps.attention(qt, kt, vt, causal, block, **knobs)
    torch.cuda.synchronize()
    return (o.cpu().numpy().reshape(-1, D).astype(np.float64), lse.cpu().numpy().reshape(-1).astype(np.float64))


def errors(o, ref):
    rel = float(np.linalg.norm(o - ref) / max(np.linalg.norm(ref), 1e-300))
    mx = float(np.abs(o - ref).max()) if o.size else 0.0
    return rel, mx
