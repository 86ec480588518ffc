"""Pins of the FP8 Q/K inputs of the oracle (CPU only).

With FP8 Q/K the attention path takes OCP FP8 E4M3 codes and per-tensor
dequantisation scales; the oracle carries every code as the bf16 pattern of
the same value (every finite E4M3 value is a bf16 value) and folds the
scales into the score scale.  What fixes that here:
- values of the OCP E4M3 encoding at its landmarks (one, the largest normal,
  the smallest normal and subnormal, signed zero, NaN);
- integer-valued FP8 inputs with unit scales give exact base-2 attention;
- the input quantiser (test infrastructure) rounds to the nearest E4M3
  value with ties to even, against a brute-force search.
"""
import math

import numpy as np
import pytest

import oracle as O
from paper_2602_02071_amd.workloads import bf16_bits_to_f32, f32_to_bf16_bits, quantize_e4m3


def _val(code):
    return float(bf16_bits_to_f32(O.e4m3_to_bf16(np.array([code], np.uint8)))[0])


def test_e4m3_landmarks():
    assert _val(0x38) == 1.0
    assert _val(0x7E) == 448.0                  # largest finite value
    assert _val(0xFE) == -448.0
    assert _val(0x08) == 2.0 ** -6              # smallest normal
    assert _val(0x01) == 2.0 ** -9              # smallest subnormal
    assert _val(0x07) == 7 * 2.0 ** -9
    assert _val(0x3C) == 1.5 and _val(0x44) == 3.0
    z = _val(0x80)
    assert z == 0.0 and math.copysign(1.0, z) < 0
    for nan in (0x7F, 0xFF):
        with pytest.raises(ValueError):
            O.e4m3_to_bf16(np.array([nan], np.uint8))


def test_e4m3_values_are_monotone_and_exact_in_bf16():
    codes = np.array([c for c in range(0x7F)], np.uint8)      # 0 .. 126: the non-negative finite codes
    v = bf16_bits_to_f32(O.e4m3_to_bf16(codes)).astype(np.float64)
    assert np.all(np.diff(v) > 0)
    assert v.size == 127


def test_quantizer_is_nearest_ties_to_even():
    codes = np.arange(0x7F, dtype=np.uint8)
    vals = bf16_bits_to_f32(O.e4m3_to_bf16(codes)).astype(np.float64)
    g = np.random.default_rng(5)
    x = np.concatenate([g.standard_normal(3000) * 50, g.standard_normal(1000) * 0.01,
                        (vals[1:] + vals[:-1]) / 2, -vals, [500.0, -1e4]])
    got = bf16_bits_to_f32(O.e4m3_to_bf16(quantize_e4m3(x, 1.0))).astype(np.float64)
    a = np.minimum(np.abs(x), 448.0)
    d = np.abs(a[:, None] - vals[None, :])
    best = d.min(1, keepdims=True)
    cand = np.where(d == best, codes[None, :], 255)
    # ties go to the even code (its mantissa's last bit is 0)
    even = np.where((d == best) & (codes[None, :] % 2 == 0), codes[None, :], 255).min(1)
    pick = np.where(even < 255, even, cand.min(1))
    want = np.copysign(vals[pick], x)
    assert np.array_equal(np.abs(got), np.abs(want))
    assert np.all((got == 0) | (np.sign(got) == np.sign(x)))


@pytest.mark.parametrize("causal", [False, True])
def test_fp8_integer_inputs_are_exact(causal):
    # codes of -1, 0, 1 with unit scales and scale 1: integer scores in
    # [-4, 4], so every T >= -8 is exact in HiF8 and every P = 2^T exact
    g = np.random.default_rng(3)
    B, H, Sq, Sk, D = 1, 2, 30, 45, 4
    lut = np.array([0xB8, 0x00, 0x38], np.uint8)
    q8 = lut[g.integers(0, 3, (B, H, Sq, D))]
    k8 = lut[g.integers(0, 3, (B, H, Sk, D))]
    v = f32_to_bf16_bits(g.standard_normal((B, H, Sk, D)).astype(np.float32))
    qb, kb = O.e4m3_to_bf16(q8), O.e4m3_to_bf16(k8)
    c = O.fp8_scale_log2(D, 1.0, 1.0, scale_log2=1.0)
    assert c == 1.0
    o, l, _ = O.attention(qb, kb, v, B, H, H, Sq, Sk, D, causal, 8, scale_log2=c)
    qf, kf, vf = (bf16_bits_to_f32(x).astype(np.float64) for x in (qb, kb, v))
    s = np.einsum("bhqd,bhkd->bhqk", qf, kf)
    if causal:
        s = np.where(np.arange(Sk)[None, :] > (np.arange(Sq)[:, None] + Sk - Sq), -np.inf, s)
    w = np.exp2(s)
    want = (np.einsum("bhqk,bhkd->bhqd", w, vf) / w.sum(-1, keepdims=True)).reshape(-1, D)
    assert np.abs(o - want).max() < 1e-13


def test_fp8_scale_folds_into_the_score_scale():
    # c' = c * q_scale * k_scale in double: powers of two move between the
    # scales without changing it
    assert O.fp8_scale_log2(128, 0.25, 4.0) == O.fp8_scale_log2(128, 1.0, 1.0) == math.log2(math.e) / math.sqrt(128)
    assert O.fp8_scale_log2(64, 0.5, 0.5, scale_log2=2.0) == 0.5
