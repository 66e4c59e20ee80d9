"""Pins of the oracle's IEEE conversions (and the generator's encoder).

References independent of both C implementations: numpy's binary16 cast,
bit reinterpretation for bfloat16 / binary32 decoding, and an exact
rational-arithmetic rounding written here from the definition of
round-to-nearest-even.
"""
from fractions import Fraction
import math

import numpy as np
import pytest

# (significand bits incl. hidden, min normal exponent, max exponent)
FORMATS = {"f16": (11, -14, 15), "bf16": (8, -126, 127), "f32": (24, -126, 127)}


def exact_rne(v: float, fmt: str) -> float:
    """Round a double to `fmt` with exact rational arithmetic, ties to even."""
    p, emin, emax = FORMATS[fmt]
    if v == 0 or math.isinf(v) or math.isnan(v):
        return v
    a = Fraction(abs(v))
    e = math.floor(math.log2(abs(v)))
    # fix floating error of log2 with exact comparisons
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, emin)
    quantum = Fraction(2) ** (e - (p - 1))
    q = a / quantum
    lo = q.numerator // q.denominator
    rem = q - lo
    r = lo + 1 if (rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1)) else lo
    out = r * quantum
    maxfin = (2 - Fraction(2) ** (1 - p)) * Fraction(2) ** emax
    res = math.inf if out > maxfin else float(out)
    return -res if v < 0 else res


def edge_values():
    vals = [0.0, -0.0, 1.0, -1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -11, 1 + 3 * 2 ** -11,
            65504.0, 65519.99, 65520.0, 2 ** -24, 2 ** -25, 3 * 2 ** -26, 2 ** -14,
            2 ** -14 - 2 ** -25, 1 / 3, -2 / 3, 3.3895e38, 3.3962e38, 3.4e38, 1e-40, 2 ** -133,
            2 ** -134, 3 * 2 ** -135, 1e300, -1e300, 5e-324]
    rng = np.random.default_rng(1)
    vals += list(rng.normal(0, 1, 300)) + list(rng.normal(0, 1e-6, 100)) + \
        list(rng.normal(0, 1e4, 100)) + list(rng.normal(0, 1e-39, 50))
    return np.array(vals, dtype=np.float64)


@pytest.mark.parametrize("fmt", ["f16", "bf16", "f32"])
def test_oracle_encode_matches_exact_rounding(orc, fmt):
    v = edge_values()
    bits = orc.encode(fmt, v)
    back = orc.decode(fmt, bits)
    ref = np.array([exact_rne(float(x), fmt) for x in v])
    same = (back == ref) | (np.isnan(back) & np.isnan(ref))
    assert same.all(), list(zip(v[~same], back[~same], ref[~same]))
    # the sign of zero survives
    assert np.all(np.signbit(back[v == 0]) == np.signbit(v[v == 0]))


def test_f16_encode_matches_numpy(orc, wl):
    rng = np.random.default_rng(2)
    v = np.concatenate([rng.normal(0, 1, 200000), rng.normal(0, 1e-5, 50000),
                        rng.normal(0, 2e4, 20000), edge_values()])
    with np.errstate(over="ignore"):
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(orc.encode("f16", v), ref)
    assert np.array_equal(wl.encode("f16", v), ref)


def test_generator_bf16_matches_exact_rounding(wl, orc):
    v = edge_values()
    got = orc.decode("bf16", wl.encode("bf16", v))
    ref = np.array([exact_rne(float(x), "bf16") for x in v])
    assert np.array_equal(got, ref)


def test_decode_all_f16_patterns(orc):
    bits = np.arange(65536, dtype=np.uint16)
    got = orc.decode("f16", bits)
    ref = bits.view(np.float16).astype(np.float64)
    assert np.all((got == ref) | (np.isnan(got) & np.isnan(ref)))


def test_decode_all_bf16_patterns(orc):
    bits = np.arange(65536, dtype=np.uint32)
    got = orc.decode("bf16", bits.astype(np.uint16))
    ref = (bits << 16).astype(np.uint32).view(np.float32).astype(np.float64)
    assert np.all((got == ref) | (np.isnan(got) & np.isnan(ref)))


def test_decode_f32_patterns(orc):
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 2 ** 32, 200000, dtype=np.uint64).astype(np.uint32)
    bits[:4] = [0x00000001, 0x007FFFFF, 0x7F7FFFFF, 0x80000000]
    got = orc.decode("f32", bits)
    ref = bits.view(np.float32).astype(np.float64)
    assert np.all((got == ref) | (np.isnan(got) & np.isnan(ref)))


def test_bf16_hand_table(orc):
    # hand-checked bfloat16 encodings (top 16 bits of binary32, RNE)
    table = {1.0: 0x3F80, 1 + 2 ** -8: 0x3F80, 1 + 3 * 2 ** -8: 0x3F82, -2.0: 0xC000,
             3.0: 0x4040, 1 / 3: 0x3EAB, 65536.0: 0x4780, 2 ** -133: 0x0001,
             3.4e38: 0x7F80, -0.0: 0x8000}
    vals = np.array(list(table.keys()))
    got = orc.encode("bf16", vals)
    assert [int(b) for b in got] == list(table.values())
