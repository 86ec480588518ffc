"""HiF8 codec kernels against the oracle (GPU): bit-exact codes over every
fp32 bit pattern, decode over all 256 codes."""
import os

import numpy as np
import pytest

import oracle as O

pytestmark = pytest.mark.gpu


def _encode_patterns(start, n, saturate, even=False):
    import torch
    import paper_2602_02071_amd as baps
    bits = torch.arange(start, start + n, dtype=torch.int64, device="cuda:0")
    bits = torch.where(bits >= 2 ** 31, bits - 2 ** 32, bits)         # same 32 bits as int32
    x = bits.to(torch.int32).view(torch.float32)                        # fp32 pattern start + i
    del bits
    codes = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    flags = (baps.BAPS_HIF8_SATURATE if saturate else 0) | (baps.BAPS_HIF8_TIES_EVEN if even else 0)
    baps.hif8_encode(x, codes, n, flags)
    torch.cuda.synchronize()
    return codes.cpu().numpy()


@pytest.mark.parametrize("saturate,even", [(True, False), (False, False), (True, True), (False, True)])
def test_encode_every_fp32_pattern(saturate, even):
    chunk = 1 << 28
    total = 1 << 32
    # the non-saturating mode differs only near and beyond 2^15: a stride of chunks suffices there
    starts = range(0, total, chunk) if saturate else range(0, total, 4 * chunk)
    for start in starts:
        codes = _encode_patterns(start, chunk, saturate, even)
        bad, first = O.check_patterns(start, codes, saturate, ties_even=even)
        assert bad == 0, f"{bad} mismatches from pattern {start:#x}, first at {start + first:#x}"
    print(f"encode saturate={saturate} even={even}: {len(starts) * chunk} patterns bit-exact", flush=True)


def test_encode_ragged_unaligned():
    import torch
    import paper_2602_02071_amd as baps
    g = np.random.default_rng(3)
    x = (g.standard_normal(100003) * 30).astype(np.float32)
    x[::7] *= np.float32(1e-6)
    want = O.hif8_encode(x)
    xt = torch.from_numpy(x).to("cuda:0")
    buf = torch.zeros(100003 + 16, dtype=torch.uint8, device="cuda:0")
    for off_x, off_c in ((0, 0), (1, 3), (0, 5)):
        n = x.size - off_x
        baps.hif8_encode(xt.data_ptr() + 4 * off_x, buf.data_ptr() + off_c, n)
        torch.cuda.synchronize()
        got = buf[off_c:off_c + n].cpu().numpy()
        assert np.array_equal(got, want[off_x:])
    # ties to even on the unaligned (scalar) kernel, with ties present
    xt2 = torch.from_numpy(np.concatenate([x, np.float32([1.0625, 22.0, 2.0 ** -23, -10.0])])).to("cuda:0")
    want2 = O.hif8_encode(xt2.cpu().numpy(), ties_even=True)
    baps.hif8_encode(xt2.data_ptr() + 4, buf.data_ptr() + 1, xt2.numel() - 1,
                     baps.BAPS_HIF8_SATURATE | baps.BAPS_HIF8_TIES_EVEN)
    torch.cuda.synchronize()
    assert np.array_equal(buf[1:xt2.numel()].cpu().numpy(), want2[1:])


def test_decode_all_codes_and_lut():
    import torch
    import paper_2602_02071_amd as baps
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8).repeat(1000).to("cuda:0")
    out = torch.empty(codes.numel(), dtype=torch.float32, device="cuda:0")
    baps.hif8_decode(codes, out, codes.numel())
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(1000, 256).astype(np.float64)
    want = O.hif8_decode(np.arange(256))
    for row in (got[0], got[-1]):
        assert np.array_equal(row, want, equal_nan=True)
    lut = np.frombuffer(baps.baps_get_exp2_lut(), dtype=np.uint8)
    assert np.array_equal(lut, O.exp2_table(0))
    # ragged, unaligned decode
    baps.hif8_decode(codes.data_ptr() + 1, out.data_ptr() + 4, 999)
    torch.cuda.synchronize()
    assert np.array_equal(out[1:1000].cpu().numpy().astype(np.float64), O.hif8_decode(np.arange(1, 1000) % 256),
                          equal_nan=True)
