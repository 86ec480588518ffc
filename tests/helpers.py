"""Shared helpers of the GPU tests: move seeded inputs to the device, run the
library, compare with the oracle.

Parity of the fused kernels is judged twice (check_parity):

1. Against the oracle run on the kernel's own high-precision scores.  Alg. 1
   forms T from S "in high precision"; the matrix unit's fp32 sums q.k are
   such an S, but not the only one (any S within the fp32 summation bound of
   the exact q.k is), so the verification entry point baps_attention_fwd_dump
   hands the kernel's own sums and block references to the oracle.  On that S
   every decision is fixed: the references must match bit for bit and O to
   the order of fp32 additions (ARB_TOL).  This holds for every sampled row.
2. Against the canonical oracle (dot products in fp64, rounded once): O
   within relative L2 2e-3 and max abs 1e-2.  A row past 1e-2 is a row where
   the kernel's S and the fp64 S round one decision differently; it must
   satisfy 1. and their number is capped (RESCUE_CAP).  Rows whose decisions
   all clear their rounding boundaries by the summation bound (margin >= 1)
   must match the canonical oracle within 2e-3.
"""
import json
import os

import numpy as np

import oracle as O

REL_L2_TOL = 2e-3        # O within relative L2 2e-3 of the oracle
MAX_ABS_TOL = 1e-2       # and max abs error 1e-2
DETERMINED_TOL = 2e-3    # rows whose every 8-bit decision is clear of its rounding boundary
LSE_TOL = 1e-3          # lse of those rows (plus two fp32 ulps of lse, which grows with m)
# O against the oracle run on the kernel's own S: the same decisions and 8-bit
# values, fp32 sums in another order.  The rounding error of an fp32 sum of n
# terms grows like sqrt(n) 2^-24 relative to the sum of magnitudes
# (sqrt(32768) * 2^-24 = 1.1e-5 at 32K keys; |v| is a few units): 1e-4 leaves
# a margin of about ten.
ARB_TOL = 1e-4
# lse = ln2 (m + log2 d) moves by the relative error of the denominator d, an
# fp32 sum of the n positive P of the row, plus the error of its own fp32
# evaluation.  The kernel sums P with v_dot2_f32_bf16, whose rounding is not
# documented as round-to-nearest: each addition is only taken to be faithful
# (error below one ulp, 2^-23 relative), so d is within n 2^-23 relative.
# The evaluation: the kernel's d carries a factor 2^-104, so log2 d runs at
# magnitudes near 2^7, where an ulp is 2^-17 (a few of them: 5e-5); the sum
# m + log2 d and the product by ln2 are each rounded to fp32 at the magnitude
# of lse itself, which grows with m (outlier channels and sink keys put it in
# the thousands): two ulps of lse on top (lse_arb_tol).
ARB_LSE_TOL = 5e-5
# rows past MAX_ABS_TOL of the canonical oracle (each one explained by the
# kernel's own S) may be at most this fraction of the sampled rows
RESCUE_FRAC = 0.005
# the Default setup's fp32 exp2 (v_exp_f32) is within a few ulps, not
# correctly rounded: a P that close to a bf16 midpoint may enter P V rounded
# either way, which moves O by at most 2^-8 of that key's weighted |v|
DEFAULT_FLIP_TOL = 2e-3

# the GPU tests append one JSON record per parity check here
PARITY_LOG = os.environ.get("BAPS_PARITY_LOG",
                            os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                                         "test_records", "parity_records.jsonl"))


def dev_bf16(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to("cuda:0")


def dev_u8(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def gpu_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, **knobs):
    """Run the fused pass on cuda:0; returns (o [B*Hq*Sq, D] fp64, lse fp64)."""
    import torch
    import paper_2602_02071_amd as baps
    qt, kt, vt = dev_bf16(q), dev_bf16(k), dev_bf16(v)
    o, lse = baps.attention(qt, kt, vt, causal, block, **knobs)
    torch.cuda.synchronize()
    return (o.cpu().numpy().reshape(-1, D).astype(np.float64), lse.cpu().numpy().reshape(-1).astype(np.float64))


# oracle keyword -> library keyword of the same knob
_GPU_KNOB = {"lam": "lam", "n_b0": "n_b0", "scale_log2": "scale_log2", "mode": "mode",
             "restart_rows": "restart_rows", "b0_last": "b0_last"}


def gpu_dump(q, k, v, shape, block, rows, fp8=None, **okw):
    """The verification entry point on the same inputs and knobs: (o, lse,
    acc [n, Sk] float32, ref [n, nblk] float64) for the given rows.  fp8 =
    (q8, k8, q_scale, k_scale): the kernels take those FP8 codes."""
    import torch
    import paper_2602_02071_amd as baps
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    knobs = {_GPU_KNOB[key]: val for key, val in okw.items() if key in _GPU_KNOB}
    if okw.get("tie_even"):
        knobs["tie_mode"] = baps.BAPS_TIES_EVEN
    if fp8 is not None:
        q8, k8, qs, ks = fp8
        qt, kt = dev_u8(q8), dev_u8(k8)
        knobs["qk_scales"] = (qs, ks)
        knobs.pop("scale_log2", None)       # the oracle's scale already holds the FP8 scales
    else:
        qt, kt = dev_bf16(q), dev_bf16(k)
    o, lse, acc, ref = baps.attention_dump(qt, kt, dev_bf16(v), causal, block, rows, **knobs)
    torch.cuda.synchronize()
    rows_t = torch.as_tensor(rows, dtype=torch.int64, device=o.device)
    o = o.reshape(-1, D)[rows_t].cpu().numpy().astype(np.float64)
    lse = lse.reshape(-1)[rows_t].cpu().numpy().astype(np.float64)
    return o, lse, acc.cpu().numpy(), ref.cpu().numpy().astype(np.float64)


def lse_arb_tol(lse_ref, n_keys):
    """Per-row bound on |lse - lse of the oracle on the kernel's own S|: the
    denominator's n 2^-23, the log2 evaluation (ARB_LSE_TOL) and two fp32
    ulps at the magnitude of lse."""
    mag = np.where(np.isfinite(lse_ref), np.abs(lse_ref), 0.0).astype(np.float32)
    return ARB_LSE_TOL + np.asarray(n_keys) * 2.0 ** -23 + 2.0 * np.spacing(mag).astype(np.float64)


def lse_agree(lse, lse_ref, tol=1e-5):
    """lse of two kernel paths whose sums differ only in order: within tol
    plus two fp32 ulps at the magnitude of lse (its last roundings happen
    there).  -inf must match -inf."""
    lse, lse_ref = np.asarray(lse, np.float64), np.asarray(lse_ref, np.float64)
    fin = np.isfinite(lse_ref)
    if not np.array_equal(fin, np.isfinite(lse)):
        return False
    if not fin.any():
        return True
    bound = tol + 2.0 * np.spacing(np.abs(lse_ref[fin]).astype(np.float32)).astype(np.float64)
    return bool(np.all(np.abs(lse[fin] - lse_ref[fin]) <= bound))


def errors(o, ref):
    rel = float(np.linalg.norm(o - ref) / max(np.linalg.norm(ref), 1e-300))
    mx = float(np.abs(o - ref).max()) if o.size else 0.0
    return rel, mx


def _acc_bound_ratio(q, k, shape, rows, acc, limit=512):
    """Largest |acc - q.k| / (summation bound) over the first `limit` rows:
    <= 1 when the matrix unit's sums obey the fp32 summation bound."""
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    sel = np.arange(min(limit, len(rows)))
    r = np.asarray(rows)[sel]
    bound = O.acc_bound(q, k, B, Hq, Hkv, Sq, Sk, D, r)
    qf = (np.ascontiguousarray(q).astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(-1, D)[r]
    kf = (np.ascontiguousarray(k).astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(B, Hkv, Sk, D)
    b, g = r // (Hq * Sq), (r // Sq) % Hq // (Hq // Hkv)
    worst = 0.0
    for i in range(sel.size):
        ex = kf[b[i], g[i]] @ qf[i]
        seen = np.isfinite(acc[sel[i]])
        if not seen.any():
            continue
        d = np.abs(acc[sel[i]][seen].astype(np.float64) - ex[seen])
        bd = bound[i][seen]
        worst = max(worst, float(np.max(np.where(bd > 0, d / np.where(bd > 0, bd, 1.0), np.where(d > 0, np.inf, 0.0)))))
    return worst


def _record(summary):
    try:
        os.makedirs(os.path.dirname(PARITY_LOG), exist_ok=True)
        with open(PARITY_LOG, "a") as f:
            f.write(json.dumps(summary) + "\n")
    except OSError:
        pass


def check_parity(q, k, v, shape, block, o, lse, rows=None, label="", fp8=None, same_kernels=True, **okw):
    """Compare GPU rows (already restricted to `rows`) with the oracle, as the
    module docstring states.  q, k, v: the oracle's inputs (bf16 patterns;
    FP8 inputs as the bf16 patterns of their values, with fp8 = the codes and
    scales the kernels took).  same_kernels: o and lse come from the one-pass
    kernels the dump runs (then they must equal the dump's bit for bit);
    False for the split-key path, whose sums run in another order.  okw: the
    oracle's knobs (mode, lam, n_b0, scale_log2, restart_rows, b0_last,
    pv_bf16, tie_even).  Returns a summary dict."""
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    rows_arr = np.arange(B * Hq * Sq) if rows is None else np.asarray(rows, dtype=np.int64)
    mode = okw.get("mode", O.E2E_HIF8)
    okw_dump = {key: val for key, val in okw.items() if key != "pv_bf16"}

    # 1. the oracle on the kernel's own scores
    od, ld, acc, gref = gpu_dump(q, k, v, shape, block, rows_arr, fp8=fp8, **okw_dump)
    if same_kernels:
        assert np.array_equal(od, o) and np.array_equal(ld, lse, equal_nan=True), \
            f"{label}: the dump kernels do not reproduce the output"
    res = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, rows=rows_arr,
                      acc=np.where(np.isfinite(acc), acc, 0).astype(np.float32), margin=(mode == O.DEFAULT),
                      refs=True, **okw)
    arb, arb_lse, aref = res[0], res[1], res[-1]
    arb_mg = res[3] if mode == O.DEFAULT else None
    assert np.array_equal(np.isnan(aref), np.isnan(gref)), f"{label}: blocks seen differ"
    ref_ok = np.array_equal(aref, gref, equal_nan=True)
    bad_ref = np.where(~((aref == gref) | (np.isnan(aref) & np.isnan(gref))).all(axis=1))[0]
    assert ref_ok, (f"{label}: block references differ from Alg. 1 on the kernel's own S in rows "
                    f"{rows_arr[bad_ref[:5]]}")
    arb_err = np.abs(o - arb).max(axis=1) if o.size else np.zeros(0)
    arb_tol = np.full(arb_err.shape, ARB_TOL)
    if mode == O.DEFAULT:
        arb_tol = np.where(arb_mg >= 1, ARB_TOL, DEFAULT_FLIP_TOL)
    worst = int(np.argmax(arb_err - arb_tol)) if arb_err.size else 0
    assert np.all(arb_err <= arb_tol), (f"{label}: row {rows_arr[worst]} differs by {arb_err[worst]:.3e} from "
                                        "Alg. 1 on the kernel's own S")
    fin = np.isfinite(arb_lse)
    assert np.array_equal(fin, np.isfinite(lse)), f"{label}: lse finiteness differs"
    lse_tol = lse_arb_tol(arb_lse, np.isfinite(acc).sum(axis=1))
    lse_gap = np.where(fin, np.abs(np.where(fin, lse, 0) - np.where(fin, arb_lse, 0)), 0.0)
    arb_lse_err = float(lse_gap.max()) if fin.any() else 0.0
    worst = int(np.argmax(lse_gap - lse_tol)) if fin.any() else 0
    assert np.all(lse_gap <= lse_tol), (f"{label}: row {rows_arr[worst]} lse differs by {lse_gap[worst]:.3e} "
                                        f"(bound {lse_tol[worst]:.2e}) on the kernel's own S")
    acc_ratio = _acc_bound_ratio(q, k, shape, rows_arr, acc) if fp8 is None else None
    if acc_ratio is not None:
        assert acc_ratio <= 1.0, f"{label}: a matrix-unit sum lies {acc_ratio:.2f}x past the fp32 summation bound"

    # 2. the canonical oracle
    margins = fp8 is None
    res = O.attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, block, rows=rows_arr, margin=margins, **okw)
    ref, ref_lse = res[0], res[1]
    rel, mx = errors(o, ref)
    assert np.array_equal(fin, np.isfinite(ref_lse)), f"{label}: lse finiteness differs from the oracle"
    assert np.all(o[~fin] == 0), label
    row_err = np.abs(o - ref).max(axis=1) if o.size else np.zeros(0)
    rescued = int((row_err > MAX_ABS_TOL).sum())
    cap = max(2, int(RESCUE_FRAC * len(rows_arr)))
    summary = dict(label=label, rows=len(rows_arr), rel_l2=rel, max_abs=mx, rescued=rescued, rescue_cap=cap,
                   arbiter_max_abs=float(arb_err.max()) if arb_err.size else 0.0, arbiter_lse=arb_lse_err,
                   refs_bit_exact=bool(ref_ok), acc_bound_ratio=acc_ratio,
                   max_abs_unrescued=float(row_err[row_err <= MAX_ABS_TOL].max()) if (row_err <= MAX_ABS_TOL).any()
                   else 0.0)
    if margins:
        mg = res[3]
        determined = mg >= 1.0
        lse_err = np.where(fin, np.abs(np.where(fin, lse, 0) - np.where(fin, ref_lse, 0)), 0.0)
        summary.update(determined=int(determined.sum()),
                       determined_max_abs=float(row_err[determined].max()) if determined.any() else 0.0,
                       determined_lse=float(lse_err[determined].max()) if determined.any() else 0.0)
    ex, _ = O.exact_attention(q, k, v, B, Hq, Hkv, Sq, Sk, D, causal, rows=rows_arr,
                              scale_log2=okw.get("scale_log2", 0.0))
    summary["gpu_vs_exact"] = errors(o, ex)[0]
    summary["oracle_vs_exact"] = errors(ref, ex)[0]
    print(f"{label}: " + " ".join(f"{k_}={v_:.3g}" if isinstance(v_, float) else f"{k_}={v_}"
                                  for k_, v_ in summary.items() if k_ != "label"), flush=True)
    _record(summary)
    assert rel <= REL_L2_TOL, f"{label}: rel-L2 {rel:.3e}"
    assert rescued <= cap, f"{label}: {rescued} rows past max-abs {MAX_ABS_TOL} (cap {cap})"
    if margins:
        assert summary["determined_max_abs"] <= DETERMINED_TOL, \
            f"{label}: determined rows differ by {summary['determined_max_abs']:.3e}"
        lse_ok = lse_err <= LSE_TOL + 2.0 * np.spacing(np.where(fin, np.abs(ref_lse), 0.0).astype(np.float32))
        assert np.all(lse_ok[determined]), \
            f"{label}: lse of determined rows differs by {summary['determined_lse']:.3e}"
    return summary
