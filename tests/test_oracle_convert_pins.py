"""Pins for the oracle's float -> code converter and fixed-point rounding.

Each check compares the oracle with something other than itself:

* DeepShift-Q (Section 3, Eqs. 4-5): numpy's float64 ``log2`` and ``round``
  on the same weights. For a float32 w the distance of log2|w| from a rounding
  boundary p + 1/2 is at least about 1e-7, far above float64 log2 error, so
  the library route is exact here; values one ulp either side of every
  boundary 2^(p + 1/2) are included;
* the defining property of the nearest power of two in the log domain:
  the decoded weight 2^p lies within a factor sqrt(2) of |w| (checked in exact
  rational arithmetic on squares) unless p was clipped;
* DeepShift-PS (Section 3): the threshold form of the ternary sign against
  the other form the paper gives, sign(round(S)), with ``decimal`` rounding
  halves away from zero; round(P) against ``decimal`` as well;
* fixed point (Section 4): exact rational rounding with ``fractions`` and
  Python integers, including exact ties and saturation;
* hand-derived examples in ``tests/golden/quantize_examples.txt``.
"""
import math
import os
from decimal import ROUND_HALF_UP, Decimal
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "quantize_examples.txt")
F32 = np.float32


def decode(code):
    """(sign, p) of a code; sign 0 for the zero weight."""
    code = int(code)
    if code & 15 == 15:
        return 0, None
    return (-1 if code & 16 else 1), -(code & 15)


def log_spread_weights(rng, n):
    """Float32 weights with magnitudes spread over 2^-20 .. 2^3, both signs."""
    mag = np.exp2(rng.uniform(-20, 3, n)).astype(F32)
    return np.where(rng.random(n) < 0.5, -mag, mag).astype(F32)


def boundary_neighbours(pmin=-18, pmax=3):
    """Float32 values one ulp below and above (and nearest to) 2^(p + 1/2)."""
    out = []
    for p in range(pmin, pmax):
        b = F32(2.0 ** (p + 0.5))
        out += [np.nextafter(b, F32(0)), b, np.nextafter(b, F32(np.inf))]
    out = np.array(out, F32)
    return np.concatenate([out, -out])


def library_q(w, max_shift):
    """Expected (sign, p) from numpy: sign(w) and round(log2|w|) in float64, clipped."""
    w64 = w.astype(np.float64)
    s = np.sign(w64)
    with np.errstate(divide="ignore", invalid="ignore"):
        p = np.round(np.log2(np.abs(w64)))
    p = np.clip(np.nan_to_num(p, nan=0.0, posinf=0.0, neginf=-max_shift), -max_shift, 0)
    return s, p


@pytest.mark.parametrize("max_shift", [14, 7, 3, 0])
def test_q_matches_library_log2_round(max_shift):
    rng = np.random.default_rng(100 + max_shift)
    kaiming = (rng.standard_normal(4000) * math.sqrt(2 / 576)).astype(F32)
    w = np.concatenate([log_spread_weights(rng, 20000), kaiming, boundary_neighbours()])
    codes = oracle.quantize_q(w, max_shift)
    s, p = library_q(w, max_shift)
    for i in range(w.size):
        sign, power = decode(codes[i])
        assert sign == s[i], (w[i], codes[i])
        if sign:
            assert power == p[i], (float(w[i]), int(codes[i]), p[i])


def test_q_boundary_neighbours_round_up_and_down():
    """Just below 2^(p+1/2) rounds to p, just above rounds to p + 1."""
    for p in range(-14, 0):
        b = F32(2.0 ** (p + 0.5))
        lo, hi = np.nextafter(b, F32(0)), np.nextafter(b, F32(np.inf))
        got = oracle.quantize_q(np.array([lo, hi, -lo, -hi], F32))
        assert [decode(c)[1] for c in got] == [p, p + 1, p, p + 1]
        assert [decode(c)[0] for c in got] == [1, 1, -1, -1]


def test_q_nearest_power_property_exact():
    """Unclipped: |w| / 2^p lies in [2^-1/2, 2^1/2], checked on exact squares."""
    rng = np.random.default_rng(7)
    w = np.concatenate([log_spread_weights(rng, 3000), boundary_neighbours(-14, 0)])
    for v, c in zip(w, oracle.quantize_q(w)):
        sign, p = decode(c)
        assert sign == (1 if v > 0 else -1)
        r2 = (Fraction(float(v)) / Fraction(2) ** p) ** 2   # (|w| / 2^p)^2
        if -14 < p < 0:
            assert Fraction(1, 2) <= r2 <= 2, (float(v), p)
        elif p == 0:
            assert r2 >= Fraction(1, 2)                        # clipped from above
        else:
            assert r2 <= 2                                     # clipped from below


def test_q_special_values():
    w = np.array([0.0, -0.0, np.nan, np.inf, -np.inf, 1e-45, -1e-45, 1.1754942e-38,
                  3.4028235e38, -3.4028235e38, 1.0, -1.0, 2.0 ** -14, 2.0 ** -15], F32)
    got = [decode(c) for c in oracle.quantize_q(w)]
    assert got[:3] == [(0, None)] * 3
    assert got[3:5] == [(1, 0), (-1, 0)]
    assert got[5:8] == [(1, -14), (-1, -14), (1, -14)]
    assert got[8:10] == [(1, 0), (-1, 0)]
    assert got[10:12] == [(1, 0), (-1, 0)]
    assert got[12] == (1, -14) and got[13] == (1, -14)
    assert oracle.quantize_q(w, 0).tolist()[3] == 0


def round_half_away(v) -> int:
    return int(Decimal(float(v)).quantize(Decimal(1), rounding=ROUND_HALF_UP))


def test_ps_sign_threshold_equals_sign_of_round():
    """The ternary thresholds (Section 3) agree with sign(round(S))."""
    rng = np.random.default_rng(11)
    s = np.concatenate([rng.uniform(-2, 2, 4000),
                        [0.5, -0.5, 1.5, -1.5, 0.0, -0.0],
                        [np.nextafter(F32(0.5), F32(0)), np.nextafter(F32(-0.5), F32(0))]]).astype(F32)
    p = np.full(s.shape, -3.0, F32)
    for sv, c in zip(s, oracle.quantize_ps(p, s)):
        expect = int(np.sign(round_half_away(sv)))
        sign, power = decode(c)
        assert sign == expect, (float(sv), int(c))
        if sign:
            assert power == -3


def test_ps_round_p_halves_away_and_clips():
    rng = np.random.default_rng(12)
    halves = np.arange(-17, 3) + 0.5
    p = np.concatenate([rng.uniform(-17, 2, 4000), halves, np.arange(-17, 3)]).astype(F32)
    s = np.where(rng.random(p.size) < 0.5, -1.0, 1.0).astype(F32)
    for max_shift in (14, 5):
        codes = oracle.quantize_ps(p, s, max_shift)
        for pv, sv, c in zip(p, s, codes):
            expect = min(0, max(-max_shift, round_half_away(pv)))
            sign, power = decode(c)
            assert sign == (1 if sv > 0 else -1)
            assert power == expect, (float(pv), int(c))


def test_ps_nan_gives_zero_weight():
    p = np.array([np.nan, -2.0, np.inf, -np.inf], F32)
    s = np.array([1.0, np.nan, -1.0, 1.0], F32)
    assert [decode(c) for c in oracle.quantize_ps(p, s)] == [(0, None), (0, None), (-1, 0), (1, -14)]


def exact_fixed(v, f):
    """round(v * 2^f) halves away from zero in exact arithmetic, saturated."""
    if math.isnan(v):
        return 0
    if math.isinf(v):
        return 2 ** 31 - 1 if v > 0 else -(2 ** 31)
    t = Fraction(v) * 2 ** f
    n = math.floor(abs(t) + Fraction(1, 2))
    n = n if t >= 0 else -n
    return max(-(2 ** 31), min(2 ** 31 - 1, n))


@pytest.mark.parametrize("frac_bits", [16, 0, 8, 31])
def test_fixed_matches_exact_rounding(frac_bits):
    rng = np.random.default_rng(200 + frac_bits)
    ties = (np.arange(-40, 40) + 0.5) / 2.0 ** frac_bits
    x = np.concatenate([rng.standard_normal(3000) * 4, rng.uniform(-40000, 40000, 500),
                        np.exp2(rng.uniform(-30, 40, 500)) * np.sign(rng.standard_normal(500)),
                        ties, [np.nan, np.inf, -np.inf, 0.0, -0.0, 32767.99, -32768.0]]).astype(F32)
    got = oracle.to_fixed(x, frac_bits)
    for v, g in zip(x, got):
        assert int(g) == exact_fixed(float(v), frac_bits), (float(v), int(g))


def test_golden_examples():
    """Hand-derived cases (each line of the fixture gives its derivation)."""
    rows = []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if line:
            rows.append(line.split())
    assert len(rows) >= 20
    for kind, *vals in rows:
        if kind == "Q":
            w, ms, code = float(vals[0]), int(vals[1]), int(vals[2])
            assert int(oracle.quantize_q(np.array([w], F32), ms)[0]) == code, vals
        elif kind == "PS":
            p, s, ms, code = float(vals[0]), float(vals[1]), int(vals[2]), int(vals[3])
            assert int(oracle.quantize_ps(np.array([p], F32), np.array([s], F32), ms)[0]) == code, vals
        elif kind == "FX":
            x, f, y = float(vals[0]), int(vals[1]), int(vals[2])
            assert int(oracle.to_fixed(np.array([x], F32), f)[0]) == y, vals
        else:
            raise AssertionError(kind)
