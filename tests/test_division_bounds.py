"""The error bounds behind the option terms' divisions, checked on the CPU by emulating the
device arithmetic exactly (rational arithmetic, each double operation rounded once; fused
multiply-adds rounded once).

The kernels divide by a reciprocal biased low (recip_low in csrc/alp_device.h): the
single-precision hardware reciprocal, which is within 1 ulp, refined by Newton steps whose last
one subtracts 2^-B.  The quotient estimate is then below the true quotient by less than 1, so
its integer part is the quotient or one less, and one remainder comparison (udiv_low) makes it
exact.  Here the hardware seed is taken at the correctly rounded value and one ulp to either
side, over random divisors and dividends and over the ends of their ranges.
"""
from __future__ import annotations

import struct
from fractions import Fraction

import numpy as np
import pytest


def _f64(q: Fraction) -> float:
    return q.numerator / q.denominator          # int / int: correctly rounded


def _f32(v: float) -> float:
    return struct.unpack("f", struct.pack("f", v))[0]


def _f32_step(v: float, k: int) -> float:
    bits = struct.unpack("I", struct.pack("f", v))[0] + k
    return struct.unpack("f", struct.pack("I", bits))[0]


def _fma(a: float, b: float, c: float) -> float:
    return _f64(Fraction(a) * Fraction(b) + Fraction(c))


def recip_low(d: int, steps: int, bias: int, ulp: int) -> float:
    D = float(d)
    y = _f32_step(_f32(1.0 / _f32(float(d))), ulp)      # the hardware seed, +-1 ulp
    for _ in range(steps - 1):
        y = _fma(y, _fma(-D, y, 1.0), y)
    one_low = 1.0 - 2.0 ** -bias
    return _fma(y, _fma(-D, y, one_low), y)


def udiv_low(x: int, d: int, inv: float) -> int:
    est = _f64(Fraction(_f64(Fraction(x))) * Fraction(inv))    # (double)x * inv
    q = int(min(est, 4294967295.0))
    r = (x - q * d) % (1 << 32)
    return q + (1 if r >= d else 0)


def _cases(rng, n, qmax):
    """(x, d) with 1 <= d < 2^31 and x / d < qmax, x < 2^63: random, and the range ends."""
    out = []
    for _ in range(n):
        d = int(np.exp(rng.uniform(0, np.log(2.0**31 - 1)))) or 1
        q = int(np.exp(rng.uniform(0, np.log(qmax - 1.0))))
        r = int(rng.integers(0, d))
        x = q * d + r
        if x < 1 << 63:
            out.append((x, d))
    for d in (1, 2, 3, 1000, 16000, 2**31 - 1, 2**31 - 2, 2**30 + 1):
        for q in (0, 1, qmax - 2, qmax // 2, qmax // 3):
            for r in (0, d - 1):
                x = q * d + r
                if x < 1 << 63:
                    out.append((x, d))
    return out


@pytest.mark.parametrize("ulp", [-1, 0, 1])
def test_quotients_below_2_32_are_exact(ulp):
    rng = np.random.default_rng([2604, 15186, 90, ulp + 1])
    for x, d in _cases(rng, 4000, 2**32 - 1):
        assert udiv_low(x, d, recip_low(d, 1, 40, ulp)) == x // d, (x, d)


@pytest.mark.parametrize("ulp", [-1, 0, 1])
def test_saturating_quotients_below_2_45(ulp):
    """tau = floor(1000 d T / n), saturated at 2^32 - 1, with the <2, 50> reciprocal of n."""
    rng = np.random.default_rng([2604, 15186, 91, ulp + 1])
    for x, n in _cases(rng, 4000, 2**45):
        if x >= 2**45:
            continue
        inv = recip_low(n, 2, 50, ulp)
        est = _f64(Fraction(float(x)) * Fraction(inv))
        tq = int(min(est, 4294967295.0))
        up = (x - tq * n) % (1 << 32) >= n and tq != 0xFFFFFFFF
        tau = 0xFFFFFFFF if est >= 4294967296.0 else tq + (1 if up else 0)
        assert tau == min(x // n, 0xFFFFFFFF), (x, n)


def test_reciprocals_are_biased_low_within_bounds():
    rng = np.random.default_rng([2604, 15186, 92])
    ds = [1, 2, 3, 7, 1000, 16000, 2**31 - 1] + [int(v) for v in rng.integers(1, 2**31, 300)]
    for d in ds:
        for ulp in (-1, 0, 1):
            for steps, bias in ((1, 40), (2, 50)):
                e = 1 - Fraction(recip_low(d, steps, bias, ulp)) * d
                assert Fraction(85, 100) / 2**bias < e < Fraction(115, 100) / 2**bias
