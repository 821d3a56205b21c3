"""Host checks of the table behind the device's -2 ln U (Box-Muller radius).

The header cpes_log_table.hpp must be what gen_log_table.py writes, every
table point must sit in its mantissa interval, and the table-driven formula,
evaluated here with exactly rounded fma (rational arithmetic), must match
-2 ln U to the accuracy the noise needs (2^-45 relative) on the edge cases
and a spread of inputs, with U = 1 giving exactly 0."""
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
    spec = importlib.util.spec_from_file_location("gen_log_table", os.path.join(CSRC, "gen_log_table.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_header_is_generated(gen):
    assert open(os.path.join(CSRC, "cpes_log_table.hpp")).read() == gen.render()


def test_table_points_lie_in_their_intervals(gen):
    t = gen.entries()
    assert len(t) == gen.N == 256
    assert t[0] == (2.0 ** -31, 0.0)                      # c_0 = 1: U = 1 gives L = 0
    assert t[-1] == (2.0 ** -32, -gen.two_ln2())          # c_255 = 2: no cancellation next to U = 1
    for i, (inv, b) in enumerate(t):
        c = 1 / (Fraction(inv) * 2 ** 31)
        assert Fraction(256 + i, 256) <= c <= Fraction(256 + i + 1, 256), i
        assert abs(b + 2 * math.log(float(c))) <= 1e-15 * max(1.0, abs(b))


def _fma(a, b, c):
    return float(Fraction(a) * Fraction(b) + Fraction(c))     # one rounding, like v_fma_f64


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
            assert got == 0.0
            continue
        ref = -2 * (Decimal(m) / Decimal(1 << 24)).ln()
        assert abs(Decimal(got) - ref) <= abs(ref) * Decimal(2) ** -45, m
