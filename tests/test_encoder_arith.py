"""CPU checks of the arithmetic the device encoder's step relies on.

The chunk encoder (csrc/wc_encode.hip, encode_kernel) computes the rANS
encoder's quotient floor(x / f) as trunc(x * r) in double precision, with r
the double nearest above 1/f (1/f correctly rounded, raised by one unit in
the last place when below 1/f), and derives the rest of the step from that
quotient Q:
  * the lane emits its low 16 bits exactly when x >= f * 2^20, i.e. Q >= 2^20;
  * an emitting lane codes from x >> 16, whose quotient is Q >> 16;
  * the new state is v + cum + q * (2^12 - f) for the value v coded from and
    its quotient q, the same as floor(v / f) * 2^12 + v mod f + cum.
The argument is in the kernel's comment; these tests check it with IEEE
double arithmetic (numpy's, the same rounding the kernel's v_mul_f64 uses)
for every f in [1, 2^12] and x across [0, 2^32): every remainder class
boundary (x = q f, q f + 1, q f + f - 1), random quotients and the extremes.
The rANS step itself is the oracle's; nothing here is taken from the kernel.
"""
from fractions import Fraction

import numpy as np

TABLE = 1 << 12


def reciprocal_up(f):
    r = np.float64(1.0) / np.float64(f)
    if Fraction(float(r)) * f < 1:
        r = np.nextafter(r, np.float64(2.0))
    return r


def sample_states(f, rng, n=1500):
    top = (2 ** 32 - 1) // f
    q = np.concatenate([rng.integers(0, top + 1, n, dtype=np.uint64),
                        np.array([0, 1, top - 1, top, (1 << 20) - 1, 1 << 20, (1 << 20) + 1],
                                 dtype=np.uint64)])
    q = q[q <= top]
    xs = [q * np.uint64(f) + np.uint64(d) for d in {0, 1, f - 1}]
    x = np.concatenate(xs)
    return x[(x >= 1) & (x < 2 ** 32)]


def test_reciprocal_is_the_double_just_above_one_over_f():
    for f in range(1, TABLE + 1):
        r = reciprocal_up(f)
        assert Fraction(float(r)) >= Fraction(1, f)
        below = np.nextafter(r, np.float64(0.0))
        assert Fraction(float(below)) < Fraction(1, f)


def test_truncated_product_is_the_exact_quotient():
    rng = np.random.default_rng(20261202)
    for f in range(1, TABLE + 1):
        x = sample_states(f, rng)
        got = np.floor(x.astype(np.float64) * reciprocal_up(f)).astype(np.uint64)
        np.testing.assert_array_equal(got, x // np.uint64(f), err_msg=f"f = {f}")


def test_step_from_the_quotient_equals_the_textbook_step():
    rng = np.random.default_rng(7)
    for f in list(range(1, 65)) + list(range(TABLE - 64, TABLE + 1)) + \
            [int(v) for v in rng.integers(65, TABLE - 64, 200)]:
        cum = int(rng.integers(0, TABLE - f + 1))
        x = sample_states(f, rng, n=300)
        x = x[x >= (1 << 16)]  # encoder states before a step
        Q = np.floor(x.astype(np.float64) * reciprocal_up(f)).astype(np.uint64)
        emit = Q >= (1 << 20)
        np.testing.assert_array_equal(emit, x >= np.uint64(f) << np.uint64(20))
        v = np.where(emit, x >> np.uint64(16), x)
        q = np.where(emit, Q >> np.uint64(16), Q)
        new = v + np.uint64(cum) + q * np.uint64(TABLE - f)
        ref = (v // np.uint64(f)) * np.uint64(TABLE) + v % np.uint64(f) + np.uint64(cum)
        np.testing.assert_array_equal(new, ref, err_msg=f"f = {f}")
        assert int(new.max(initial=0)) < 2 ** 32
