"""Host checks of the two tables behind the device's Box-Muller transform.

The header cpes_bm_tables.hpp must be what gen_bm_tables.py writes.  Log
table: every table point must sit in its mantissa interval, and the
table-driven formula, evaluated here with exactly rounded fma (rational
arithmetic), must match -2 ln U to 2^-45 relative on the edge cases and a
spread of inputs, with U = 1 giving 2^-400 (a zero normal).  Angle table:
every entry must be cos and sin of its angle correctly rounded, the
quarter turns exact, and the device's rotation (again with exactly rounded
fma) must match the exact quadrant reduction of the oracle: 2^-48 relative
on edge cases and a spread of inputs, exact zeros and ones with the same
signs of zero.  pi, ln, sin and cos come from 60-digit decimal arithmetic
written here (Machin's formula, Taylor series), not from the generator."""
import importlib.util
import math
import os
from decimal import Decimal, getcontext
from fractions import Fraction

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_02391_amd", "csrc")


@pytest.fixture(scope="module")
def gen():
    spec = importlib.util.spec_from_file_location("gen_bm_tables", os.path.join(CSRC, "gen_bm_tables.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _pi():
    getcontext().prec = 60

    def atan_inv(k):                                   # Gregory series of atan(1/k)
        x, total, n, sign = Decimal(1) / k, Decimal(0), 1, 1
        term = x
        while term > Decimal(10) ** -64:
            total += sign * term / n
            term *= x * x
            n += 2
            sign = -sign
        return total
    return 16 * atan_inv(5) - 4 * atan_inv(239)


PI = _pi()


def _sin_cos(t):
    """Decimal sin and cos of a Decimal t, |t| <= 4, by their Taylor series."""
    getcontext().prec = 60
    s, c, term, n = Decimal(0), Decimal(0), Decimal(1), 0
    while n < 12 or abs(term) > Decimal(10) ** -64:
        if n % 4 == 0:
            c += term
        elif n % 4 == 1:
            s += term
        elif n % 4 == 2:
            c -= term
        else:
            s -= term
        n += 1
        term = term * t / n
    return s, c


def test_header_is_generated(gen):
    assert open(os.path.join(CSRC, "cpes_bm_tables.hpp")).read() == gen.render()


# ----------------------------------------------------------------- radius --

def test_log_table_points_lie_in_their_intervals(gen):
    t = gen.entries()
    assert len(t) == gen.N == 256
    assert t[0] == (2.0 ** -31, 2.0 ** -400)              # c_0 = 1, B_0 = 0 stored as 2^-400
    assert t[-1] == (2.0 ** -32, -gen.two_ln2())          # c_255 = 2: no cancellation next to U = 1
    for i, (inv, b) in enumerate(t):
        c = 1 / (Fraction(inv) * 2 ** 31)
        assert Fraction(256 + i, 256) <= c <= Fraction(256 + i + 1, 256), i
        if i:
            assert abs(b + 2 * math.log(float(c))) <= 1e-15 * max(1.0, abs(b))


def _fma(a, b, c):
    """a * b + c with one rounding, like v_fma_f64, including the sign of a zero result."""
    exact = Fraction(a) * Fraction(b) + Fraction(c)
    if exact != 0:
        return float(exact)
    prod_neg = (math.copysign(1, a) * math.copysign(1, b)) < 0
    if a * b == 0 and c == 0:                                 # -0 only for -0 + -0
        return -0.0 if prod_neg and math.copysign(1, c) < 0 else 0.0
    return 0.0                                                # exact cancellation: +0


def _device_L(m, table, two_ln2):
    """The device's arithmetic for U = m 2^-24, step by step."""
    m7 = m << 7
    e = 32 - m7.bit_length()                                   # clz
    mn = m7 << e
    inv, b = table[(mn >> 23) & 0xFF]
    r = _fma(float(mn), inv, -1.0)
    base = _fma(float(e), two_ln2, b)
    q = -0.4
    for c in (0.5, -2.0 / 3.0, 1.0, -2.0):
        q = _fma(q, r, c)
    return _fma(r, q, base)


def test_table_driven_log_accuracy(gen):
    getcontext().prec = 40
    table, k = gen.entries(), gen.two_ln2()
    ms = {1, 2, 3, 1 << 23, (1 << 23) + 1, (1 << 24) - 1, (1 << 24) - 2, 1 << 24}
    ms |= {1 << s for s in range(25)} | {(1 << s) - 1 for s in range(2, 25)}
    ms |= {(256 + i) << 15 for i in range(256)} | {((256 + i) << 15) - 1 for i in range(1, 257)}
    ms |= {1 + (j * 2654435761) % (1 << 24) for j in range(1500)}
    for m in sorted(ms):
        got = _device_L(m, table, k)
        if m == 1 << 24:
            assert got == 2.0 ** -400                          # sqrt: 2^-200, a zero in fp32
            continue
        ref = -2 * (Decimal(m) / Decimal(1 << 24)).ln()
        assert abs(Decimal(got) - ref) <= abs(ref) * Decimal(2) ** -45, m


# ------------------------------------------------------------------ angle --

def test_angle_table_is_correctly_rounded(gen):
    t = gen.angle_entries()
    assert len(t) == gen.NA == 512
    quarters = {0: (1.0, 0.0), 128: (-0.0, 1.0), 256: (-1.0, -0.0), 384: (0.0, -1.0)}
    for i, (c, s) in enumerate(t):
        if i in quarters:
            qc, qs = quarters[i]
            assert (c, s) == (qc, qs) and math.copysign(1, c) == math.copysign(1, qc) \
                and math.copysign(1, s) == math.copysign(1, qs), i
            continue
        ref_s, ref_c = _sin_cos(2 * PI * i / 512 if i < 256 else 2 * PI * (i - 512) / 512)
        for got, ref in ((c, ref_c), (s, ref_s)):
            err = abs(Fraction(got) - Fraction(ref))
            half_ulp = Fraction(math.ulp(got)) / 2
            assert err <= half_ulp, (i, got)


def _device_angle(m, table, k):
    """The device's rotation for theta = 2 pi m 2^-24, step by step."""
    b = ((m - 1) << 8) & 0xFFFFFFFF
    s8 = (b + 0x100) & 0xFFFFFFFF
    x = (s8 >> 8) & 0x7FFF
    x = float(x - 0x8000 if x & 0x4000 else x)
    i = (((b + 0x400100) & 0xFFFFFFFF) >> 23) & 0x1FF
    c_i, s_i = table[i]
    x2 = x * x
    sd = x * _fma(x2, _fma(x2, k["A5"], k["A3"]), k["A1"])
    cd = _fma(x2, _fma(x2, k["B4"], k["B2"]), 1.0)
    cos_t = _fma(c_i, cd, -(s_i * sd))
    sin_t = _fma(s_i, cd, c_i * sd)
    return cos_t, sin_t


def _exact_angle(m):
    """cos and sin of pi m 2^-23 with the quadrant taken exactly, as the oracle does."""
    getcontext().prec = 60
    q, rem = (m >> 22) & 3, m & ((1 << 22) - 1)
    s, c = _sin_cos(PI * rem / Decimal(1 << 23))
    return [(c, s), (-s, c), (-c, -s), (s, -c)][q]


def test_angle_rotation_accuracy(gen):
    table, k = gen.angle_entries(), gen.angle_coefficients()
    ms = {1, 2, 3, (1 << 24) - 1, 1 << 24}
    ms |= {q << 22 for q in range(1, 4)} | {(q << 22) + d for q in range(4) for d in (-2, -1, 1, 2) if q or d > 0}
    ms |= {(i << 15) + d for i in range(0, 512, 7) for d in (-(1 << 14) - 1, -(1 << 14), (1 << 14) - 1, 1 << 14)
           if 0 < (i << 15) + d <= 1 << 24}
    ms |= {1 + (j * 2654435761) % (1 << 24) for j in range(1500)}
    for m in sorted(ms):
        got = _device_angle(m, table, k)
        ref = _exact_angle(m)
        for g, r in zip(got, ref):
            if r == 0:
                assert g == 0, m
                continue
            assert abs(Decimal(g) - r) <= abs(r) * Decimal(2) ** -48, (m, g, r)


def test_angle_quarter_turns_keep_the_signs_of_zero(gen):
    """cos(pi/2) = -0, sin(pi) = -0, cos(3 pi/2) = +0, sin(0) = sin(2 pi) = +0,
    as the oracle's exact quadrant reduction gives them."""
    table, k = gen.angle_entries(), gen.angle_coefficients()
    want = {1 << 22: (-0.0, 1.0), 2 << 22: (-1.0, -0.0), 3 << 22: (0.0, -1.0), 1 << 24: (1.0, 0.0)}
    for m, (wc, ws) in want.items():
        c, s = _device_angle(m, table, k)
        assert (c, s) == (wc, ws)
        assert math.copysign(1, c) == math.copysign(1, wc) and math.copysign(1, s) == math.copysign(1, ws), m
