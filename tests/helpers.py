"""Shared helpers of the GPU tests: move seeded inputs to the device, run the
library, compare with the oracle."""
import numpy as np

import oracle as O

REL_L2_TOL = 2e-3        # O within relative L2 2e-3 of the oracle
MAX_ABS_TOL = 1e-2       # and max abs error 1e-2
DETERMINED_TOL = 2e-3    # rows whose every 8-bit decision is clear of its rounding boundary
LSE_TOL = 1e-3

# other valid high-precision S for rows whose decisions sit within the
# accumulation error bound of a rounding boundary: every dot product moved by
# a fraction of its bound, the same way or with random signs
JITTERS = [(1.0, 0), (-1.0, 0), (0.5, 0), (-0.5, 0), (1.0, 1), (1.0, 2), (1.0, 3), (1.0, 4), (0.5, 5), (0.5, 6)]


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


def check_parity(q, k, v, shape, block, o, lse, rows=None, label="", **okw):
    """Compare GPU rows (already restricted to `rows`) with the oracle.

    Every row must be within MAX_ABS_TOL of the oracle, and rows whose 8-bit
    decisions are all clear of their rounding boundaries (margin >= 1) within
    DETERMINED_TOL.  A row beyond MAX_ABS_TOL passes only if its margin is
    below 1 -- the scores' fp32 accumulation error can legitimately move one of
    its decisions -- and the oracle, run on another valid high-precision S
    (JITTERS), lands within MAX_ABS_TOL of it.  Returns a summary dict."""
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    rows_arr = np.arange(B * Hq * Sq) if rows is None else np.asarray(rows)
    ref, ref_lse, _, mg = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, rows=rows_arr,
                                      margin=True, **okw)
    rel, mx = errors(o, ref)
    fin = np.isfinite(ref_lse)
    assert np.array_equal(fin, np.isfinite(lse)), f"{label}: lse finiteness differs"
    assert np.all(o[~fin] == 0), label
    row_err = np.abs(o - ref).max(axis=1) if o.size else np.zeros(0)
    lse_err = np.where(fin, np.abs(np.where(fin, lse, 0) - np.where(fin, ref_lse, 0)), 0.0)
    determined = mg >= 1.0
    bad = np.where(row_err > MAX_ABS_TOL)[0]
    rescued = 0
    for i in bad:
        assert not determined[i], (f"{label}: row {rows_arr[i]} is determined (margin {mg[i]:.2f}) "
                                   f"but differs by {row_err[i]:.3e}")
        ok = False
        for scale, seed in JITTERS:
            alt, _, _ = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, rows=rows_arr[i:i + 1],
                                    jitter=scale, jitter_seed=seed, **okw)
            if np.abs(o[i] - alt[0]).max() <= MAX_ABS_TOL:
                ok = True
                break
        assert ok, f"{label}: row {rows_arr[i]} (margin {mg[i]:.2f}) differs by {row_err[i]:.3e} from every valid S"
        rescued += 1
    det_err = float(row_err[determined].max()) if determined.any() else 0.0
    det_lse = float(lse_err[determined].max()) if determined.any() else 0.0
    ex, _ = O.exact_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, rows=rows_arr,
                              scale_log2=okw.get("scale_log2", 0.0))
    rel_ex, _ = errors(o, ex)
    rel_or, _ = errors(ref, ex)
    summary = dict(rows=len(rows_arr), rel_l2=rel, max_abs=mx, determined=int(determined.sum()),
                   determined_max_abs=det_err, determined_lse=det_lse, ambiguous=int((~determined).sum()),
                   rescued=rescued, gpu_vs_exact=rel_ex, oracle_vs_exact=rel_or)
    print(f"{label}: " + " ".join(f"{k_}={v_:.3g}" if isinstance(v_, float) else f"{k_}={v_}"
                                  for k_, v_ in summary.items()), flush=True)
    assert rel <= REL_L2_TOL, f"{label}: rel-L2 {rel:.3e}"
    assert det_err <= DETERMINED_TOL, f"{label}: determined rows differ by {det_err:.3e}"
    assert det_lse <= LSE_TOL, f"{label}: lse of determined rows differs by {det_lse:.3e}"
    return summary
