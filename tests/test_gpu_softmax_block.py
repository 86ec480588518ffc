"""The standalone softmax-block kernel against the oracle (GPU): identical
fp32 scores in, so codes, reference shifts, final maxima and restart flags
are bit-exact and the denominator agrees to fp32 summation order."""
import json
import os

import numpy as np
import pytest

import oracle as O
from paper_2602_02071_amd.workloads import random_scores

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def gpu_softmax_block(s, block, lam=1, n_b0=1, ld=None):
    import torch
    import paper_2602_02071_amd as baps
    rows, cols = s.shape
    ld = cols if ld is None else ld
    buf = np.full((rows, ld), np.nan, np.float32)
    buf[:, :cols] = s
    st = torch.from_numpy(buf).to("cuda:0")
    nblk = (cols + block - 1) // block
    codes = torch.empty((rows, cols), dtype=torch.uint8, device="cuda:0")
    refs = torch.empty((rows, nblk), dtype=torch.int32, device="cuda:0")
    m = torch.empty(rows, dtype=torch.float32, device="cuda:0")
    d = torch.empty(rows, dtype=torch.float32, device="cuda:0")
    rs = torch.empty((rows, nblk), dtype=torch.uint8, device="cuda:0")
    baps.baps_softmax_block(st, rows, cols, ld, block, lam, n_b0, 0, codes, refs, m, d, rs)
    torch.cuda.synchronize()
    return (codes.cpu().numpy(), refs.cpu().numpy(), m.cpu().numpy().astype(np.float64),
            d.cpu().numpy().astype(np.float64), rs.cpu().numpy())


def _compare(s, block, lam=1, n_b0=1, ld=None):
    got = gpu_softmax_block(s, block, lam, n_b0, ld)
    want = O.softmax_block(s, block, lam, n_b0)
    names = ("codes", "ref_shift", "m_final", "d_final", "restarted")
    for name, g, w in zip(names, got, want):
        if name == "d_final":
            ok = np.isfinite(w) & (w > 0)
            assert np.array_equal(g[~ok], w[~ok])
            assert np.all(np.abs(g[ok] - w[ok]) <= 1e-5 * w[ok]), name
        else:
            assert np.array_equal(g, w), (name, np.argwhere(g != w)[:5])


@pytest.mark.parametrize("block", [64, 128, 256, 512, 1024])
@pytest.mark.parametrize("std", [1.5, 8.0])
def test_random_scores(block, std):
    s = random_scores(37, 3000 + block // 64, seed=block, std=std, masked_frac=0.03)
    _compare(s, block)


@pytest.mark.parametrize("lam,n_b0", [(0, 1), (2, 1), (1, 0), (1, 5), (-3, 1), (50, 2)])
def test_knobs(lam, n_b0):
    s = random_scores(16, 2000, seed=9, std=5.0)
    s[:, 1200:1300] += np.float32(7.0)          # late maxima force restarts
    _compare(s, 128, lam, n_b0)


def test_many_blocks_and_stride():
    s = random_scores(9, 64 * 70 + 17, seed=4, std=6.0, masked_frac=0.01)   # > 64 blocks per row
    _compare(s, 64, ld=s.shape[1] + 5)


def test_degenerate_rows():
    s = np.full((4, 300), -np.inf, np.float32)
    s[1, 250] = 3.25
    s[2, :] = 0.0
    s[3, ::2] = np.arange(150, dtype=np.float32)       # integer scores, steep growth
    _compare(s, 64)


def test_golden_walkthrough_on_gpu():
    # the hand-derived walk through Alg. 1, at block 64 (each 2-key block of
    # the fixture padded with masked scores)
    g = json.load(open(os.path.join(GOLDEN, "softmax_block_walkthrough.json")))
    sc = np.array(g["scores"], np.float32).reshape(-1, 2)
    s = np.full((1, 64 * sc.shape[0]), -np.inf, np.float32)
    for j, pair in enumerate(sc):
        s[0, 64 * j: 64 * j + 2] = pair
    for c in g["cases"]:
        codes, refs, m, d, rs = gpu_softmax_block(s, 64, c["lambda"], g["n_b0"])
        vals = O.hif8_decode(codes[0].reshape(-1, 64)[:, :2].reshape(-1))
        assert vals.tolist() == c["p_values"]
        assert refs[0].tolist() == c["ref_shift"]
        assert rs[0].tolist() == c["restarted"]
        assert m[0] == c["m_final"] and d[0] == c["d_final"]


@pytest.mark.parametrize("block,cols", [(64, 2560), (128, 2560), (256, 4096 + 256), (128, 132)])
def test_row_group_path_many_blocks(block, cols):
    # 16-byte aligned rows with a multiple-of-4 length take the 4-rows-per-wave
    # kernel; > 16 blocks per row exercises its reference parking
    s = random_scores(37, cols, seed=cols + block, std=6.0, masked_frac=0.02)
    s[5, :] = -np.inf
    s[6, : block] = -np.inf
    _compare(s, block)


@pytest.mark.parametrize("block", [64, 128])
def test_row_group_path_wide_launch(block):
    # enough rows to give every CU a 64-row workgroup: the 1024-thread form of
    # the row-group kernel, with a ragged last workgroup
    s = random_scores(16384 + 37, 4 * block + 4, seed=block + 11, std=6.0, masked_frac=0.02)
    s[-1, :] = -np.inf
    _compare(s, block)


def test_row_group_path_wide_launch_long_rows():
    # rows of at least 4096 columns at the 1024-thread launch: 512 columns per
    # step, with a ragged last step and a ragged last workgroup
    s = random_scores(16384 + 37, 4096 + 132, seed=23, std=6.0, masked_frac=0.02)
    s[-1, :] = -np.inf
    s[3, 4000:] += np.float32(9.0)              # a late maximum forces restarts
    _compare(s, 128)


@pytest.mark.parametrize("rows", [12288 + 5, 4096 + 3])
def test_row_group_path_step_widths(rows):
    # fewer rows than one 64-row workgroup per CU: more than two 256-thread
    # workgroups per CU step 256 columns at a time, at most two step 1024
    s = random_scores(rows, 2048 + 516, seed=rows, std=6.0, masked_frac=0.02)
    s[1, :] = -np.inf
    _compare(s, 128)
