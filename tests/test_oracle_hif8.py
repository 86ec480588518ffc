"""Pins of the oracle's HiF8 codec and 8-bit exp2 table (CPU only).

Each check ties the oracle to something other than its own code: the value
set the HiF8 format defines (binade counts and mantissa widths), library
conversions (numpy float16, torch float8 e4m3fn / e5m2, torch bfloat16) in
the binades where those formats have the same mantissa width, explicit
rounding thresholds, and closed forms of exp2 on integers.
"""
import numpy as np
import pytest
import torch

import oracle as O

CODES = np.arange(256)


@pytest.fixture(scope="module")
def values():
    return O.hif8_decode(CODES)


def test_value_set_counts(values):
    fin = values[np.isfinite(values)]
    assert fin.size == 253                      # 2 x 126 nonzero values + zero
    pos = np.sort(fin[fin > 0])
    assert pos.size == 126
    assert pos[0] == 2.0 ** -22 and pos[-1] == 2.0 ** 15
    assert np.isnan(values[0x80]) and values[0x00] == 0.0
    assert values[0x6F] == np.inf and values[0xEF] == -np.inf
    # per binade: 7 denormal powers of two 2^-22..2^-16, then mantissa widths
    # 1 bit for |e| in 8..15, 2 bits for |e| in 4..7, 3 bits for |e| <= 3
    e = np.floor(np.log2(pos)).astype(int)
    for ex in range(-22, 16):
        n = int((e == ex).sum())
        if ex <= -16:
            want = 1
        elif abs(ex) >= 8:
            want = 2
        elif abs(ex) >= 4:
            want = 4
        else:
            want = 8
        if ex == 15:
            want = 1                            # 1.5 * 2^15 is the Inf code
        assert n == want, (ex, n, want)
        # the values of a binade are evenly spaced (no missing mantissas)
        vals = pos[e == ex]
        if want > 1:
            assert np.allclose(np.diff(vals), 2.0 ** ex / want)
    # odd symmetry of the code space: code | 0x80 is the negative value
    for c in range(1, 128):
        if np.isfinite(values[c]):
            assert values[c | 0x80] == -values[c]


def test_subset_of_fp16_and_bf16(values):
    fin = values[np.isfinite(values)]
    assert np.array_equal(fin.astype(np.float16).astype(np.float64), fin)
    t = torch.tensor(fin, dtype=torch.float64)
    assert torch.equal(t.to(torch.bfloat16).to(torch.float64), t)


def test_round_trip(values):
    for c in range(256):
        v = values[c]
        if np.isnan(v):
            assert O.hif8_encode_scalar(float("nan")) == 0x80
            continue
        assert O.hif8_encode_scalar(v, saturate=False) == c
        if np.isfinite(v):
            assert O.hif8_encode_scalar(v, saturate=True) == c


def _rand_in(lo_exp, hi_exp, n, seed):
    g = np.random.default_rng(seed)
    e = g.integers(lo_exp, hi_exp, n)
    m = g.random(n, dtype=np.float64)
    x = (np.ldexp(1.0 + m, e)).astype(np.float32)
    sgn = np.where(g.random(n) < 0.5, -1.0, 1.0).astype(np.float32)
    return x * sgn


def _is_tie(x, step_exp_fn):
    """True where |x| lies exactly on a midpoint of the format's grid."""
    a = np.abs(x.astype(np.float64))
    e = np.floor(np.log2(a)).astype(int)
    step = np.ldexp(1.0, step_exp_fn(e))
    r = a / step
    return r - np.floor(r) == 0.5


def test_matches_e4m3_where_three_mantissa_bits():
    # |x| in [2^-3, 2^4): HiF8 keeps 3 mantissa bits, as does float8_e4m3fn
    x = _rand_in(-3, 4, 200000, 1)
    tie = _is_tie(x, lambda e: e - 3)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = O.hif8_round(x)
    assert np.array_equal(got[~tie], ref[~tie])


def test_matches_e5m2_where_two_mantissa_bits():
    # |x| in [2^-7, 2^-3) and [2^4, 2^8): 2 mantissa bits, as float8_e5m2
    x = np.concatenate([_rand_in(-7, -3, 100000, 2), _rand_in(4, 8, 100000, 3)])
    tie = _is_tie(x, lambda e: e - 2)
    ref = torch.from_numpy(x).to(torch.float8_e5m2).to(torch.float64).numpy()
    got = O.hif8_round(x)
    assert np.array_equal(got[~tie], ref[~tie])


def test_one_mantissa_bit_thresholds():
    # |x| in [2^e, 2^(e+1)) for |e| in 8..15 (e < 15): grid {1, 1.5, 2} * 2^e,
    # nearest with midpoints 1.25 and 1.75, ties away from zero
    x = np.concatenate([_rand_in(8, 15, 50000, 4), _rand_in(-15, -7, 50000, 5)])
    a = np.abs(x.astype(np.float64))
    e = np.floor(np.log2(a))
    f = a / np.exp2(e)
    want = np.where(f < 1.25, 1.0, np.where(f < 1.75, 1.5, 2.0)) * np.exp2(e)
    want = np.copysign(want, x)
    assert np.array_equal(O.hif8_round(x), want)


def test_denormal_region_thresholds():
    # below 2^-15 only powers of two remain: nearest power, midpoint 1.5 * 2^k;
    # below 2^-22: 2^-22 from 2^-23 up, zero under it
    x = np.concatenate([_rand_in(-23, -15, 50000, 6), _rand_in(-30, -23, 2000, 7)])
    a = np.abs(x.astype(np.float64))
    e = np.floor(np.log2(a))
    f = a / np.exp2(e)
    want = np.where(f < 1.5, 1.0, 2.0) * np.exp2(e)
    want = np.where(e < -23, 0.0, np.where(e == -23, 2.0 ** -22, want))
    got = O.hif8_round(x)
    assert np.array_equal(np.abs(got), want)


def test_ties_away_from_zero():
    cases = {1.0625: 1.125, -1.0625: -1.125, 1.1875: 1.25, 2.125: 2.25, 0.15625 + 0.0078125: 0.171875,
             20.0 + 2.0: 24.0, 1.25 * 256: 1.5 * 256, 1.5 * 2.0 ** -20: 2.0 ** -19,
             2.0 ** -23: 2.0 ** -22, -(2.0 ** -23): -(2.0 ** -22)}
    for x, want in cases.items():
        assert O.hif8_round(np.array([x], np.float32))[0] == want, x


def test_saturation_and_specials():
    x = np.array([32768.0, 40000.0, 1.25 * 32768, 3.0e38, np.inf, -np.inf, -5e4, np.nan, -0.0, 1e-30],
                 np.float32)
    c = O.hif8_encode(x, saturate=True)
    assert list(c) == [0x6E, 0x6E, 0x6E, 0x6E, 0x6F, 0xEF, 0xEE, 0x80, 0x00, 0x00]
    c = O.hif8_encode(x, saturate=False)
    assert list(c[:6]) == [0x6E, 0x6E, 0x6F, 0x6F, 0x6F, 0xEF]   # 1.25*2^15 is the midpoint to Inf


def test_monotone_idempotent_symmetric():
    g = np.random.default_rng(8)
    x = np.sort(np.concatenate([
        g.standard_normal(100000).astype(np.float32) * np.float32(10.0),
        (g.standard_normal(100000) * 1e-5).astype(np.float32),
        _rand_in(-25, 16, 100000, 9)]))
    r = O.hif8_round(x)
    assert np.all(np.diff(r) >= 0)
    assert np.array_equal(O.hif8_round(r.astype(np.float32)), r)
    assert np.array_equal(O.hif8_round(-x), -r)


def test_codes_not_value_ordered(values):
    # integer code order is not value order: never take a max over raw codes
    pos = [c for c in range(1, 128) if np.isfinite(values[c])]
    assert any(values[a] > values[b] for a, b in zip(pos, pos[1:]))


def test_fp16_rounding_matches_numpy():
    g = np.random.default_rng(10)
    y = np.concatenate([np.exp2(g.uniform(-26, 17, 20000)), g.standard_normal(2000)])
    with np.errstate(over="ignore"):
        want = y.astype(np.float16).astype(np.float64)
    got = np.array([O.round_fp16(float(t)) for t in y])
    assert np.array_equal(got, want)


def test_exp2_table_closed_forms(values):
    t = O.exp2_table(0)
    tv = values[t]
    for c in range(256):
        x = values[c]
        if np.isnan(x):
            assert t[c] == 0x80
            continue
        if x == -np.inf:
            assert tv[c] == 0.0
            continue
        if x == np.inf or x >= 15:
            assert tv[c] in (np.inf, 2.0 ** 15)
            continue
        if x == int(x) and -22 <= x <= 15:
            assert tv[c] == 2.0 ** x, x                     # integer powers are exact
        if x <= -24:
            assert tv[c] == 0.0
        # HiF8(2^x) is a nearest HiF8 value to 2^x: no finite value is closer
        y = 2.0 ** x
        fin = values[np.isfinite(values)]
        assert abs(y - tv[c]) <= np.min(np.abs(fin - y)) * (1 + 1e-15)
    assert tv[0] == 1.0
    # non-decreasing in the input value
    order = np.argsort([values[c] if np.isfinite(values[c]) else np.nan for c in range(256)])
    fin_codes = [c for c in order if np.isfinite(values[c])]
    seq = tv[fin_codes]
    assert np.all(np.diff(seq) >= 0)


def test_exp2_table_fp16_carrier_agrees_below_overflow(values):
    # Alg. 2 evaluates exp2 in FP16; it can differ from the fp64 evaluation only
    # where 2^x exceeds FP16's range (x >= 16), far outside the scores' domain
    t0, t1 = O.exp2_table(0), O.exp2_table(1)
    diff = [c for c in range(256) if t0[c] != t1[c]]
    assert all(values[c] >= 16 for c in diff), diff


def test_fp8_value_sets():
    e4 = np.array([O.e4m3_decode(c) for c in range(256)])
    e5 = np.array([O.e5m2_decode(c) for c in range(256)])
    ref4 = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ref5 = torch.arange(256, dtype=torch.uint8).view(torch.float8_e5m2).to(torch.float64).numpy()
    assert np.array_equal(e4, ref4, equal_nan=True)
    assert np.array_equal(e5, ref5, equal_nan=True)
