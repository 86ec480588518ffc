"""Pins of the oracle's rescale-product experiment (CPU only).

Sec. 3.3 and Fig. 2 of the paper: the rescale factors of the online softmax
multiply up over the key blocks.  Raised to integer exponents they are exact
powers of two and the running product carries no error at any length;
evaluated at 8 bits from arbitrary exponents (E8[Q8(x)]) every factor is off
by up to a few percent and the product drifts.  What fixes the experiment,
other than its own code:
- integer exponents give exactly zero error, for any real inputs;
- 8-bit factors of integer exponents are exact powers of two (zero error);
- a constant exponent -1/2 has a closed form: HiF8 keeps three mantissa
  bits at binary exponent -1, so 2^(-1/2) = 1.0110101..._2 * 2^-1 rounds to
  1.011_2 * 2^-1 = 0.6875, and after n steps the log2 error is
  n * log2(0.6875 * sqrt(2));
- with random exponents the drift of the 8-bit product grows with length.
"""
import numpy as np

import oracle as O


def test_integer_exponents_are_exact_at_any_length():
    rng = np.random.default_rng(1)
    for scale in (1.0, 5.0, 40.0):
        x = -rng.random(5000) * scale
        assert np.all(O.power_product(x, True) == 0.0)


def test_eight_bit_factors_of_integer_exponents_are_exact():
    x = np.tile([-1.0, -2.0, -3.0, -4.0, -6.0, -8.0, 0.0], 300)
    assert np.all(O.power_product(x, False) == 0.0)


def test_constant_half_exponent_closed_form():
    n = np.arange(1, 2001)
    got = O.power_product(np.full(n.size, -0.5), False)
    want = n * np.log2(0.6875 * np.sqrt(2.0))
    assert np.abs(got - want).max() < 1e-10             # fp64 summation over 2000 terms


def test_direct_exponents_drift_with_length():
    rng = np.random.default_rng(2)
    drift = np.array([np.abs(O.power_product(-rng.random(4096), False)[[63, 4095]]) for _ in range(8)])
    assert drift[:, 1].mean() > 4 * drift[:, 0].mean()
    assert drift[:, 1].mean() > 1.0           # more than a factor 2 off after 4096 blocks


def test_integer_and_direct_agree_where_the_exponents_are_integers():
    # the integer path rounds up; on integer inputs both paths are the exact
    # running product, so a sign or rounding mistake in either shows here
    x = -np.arange(0, 50, dtype=np.float64) % 7
    assert np.array_equal(O.power_product(x, True), O.power_product(x, False))
