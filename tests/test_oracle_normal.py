"""Pins of the oracle's Gaussian noise (eps ~ N(0, I), Eq. 3 and Eq. 8) built by
Box-Muller from Philox words.  The paper only says each perturbation is a seed
that is replayed (Sec. 3.3); the transform itself is our reading, so it is pinned
by closed forms, by independent arbitrary-precision / extended-precision library
evaluation, and by the statistics the paper relies on (E||sigma eps||^2 = d
sigma^2, Eq. 10)."""
import math

import mpmath
import numpy as np
import pytest
from scipy import stats

TWO24 = 1 << 24


def test_uniform_identities(orc):
    assert orc.uniform_open0(0) == 2.0 ** -24
    assert orc.uniform_open0(0xFFFFFFFF) == 1.0
    assert orc.uniform_open0(255) == orc.uniform_open0(0)
    assert orc.uniform_open0(256) == 2.0 * 2.0 ** -24
    assert orc.uniform_open0(0x80000000) == 0.5 + 2.0 ** -24


def test_radius_special_values(orc):
    assert orc.bm_radius(0xFFFFFFFF) == 0.0          # U = 1 -> ln 1 = 0
    assert orc.bm_radius(0) == pytest.approx(math.sqrt(48.0 * math.log(2.0)), rel=1e-15)
    # U = 1/2 -> rho = sqrt(2 ln 2)
    assert orc.bm_radius((TWO24 // 2 - 1) << 8) == pytest.approx(math.sqrt(2.0 * math.log(2.0)), rel=1e-15)


def _b_for_m(m):
    """A word b with (b >> 8) + 1 == m."""
    return (m - 1) << 8


@pytest.mark.parametrize("m,cos_ref,sin_ref", [
    (TWO24, 1.0, 0.0),            # angle 2*pi == 0
    (1 << 22, 0.0, 1.0),          # pi/2
    (1 << 23, -1.0, 0.0),         # pi
    (3 << 22, 0.0, -1.0),         # 3pi/2
])
def test_angle_exact_axes(orc, m, cos_ref, sin_ref):
    c, s = orc.bm_angle(_b_for_m(m))
    assert c == cos_ref and s == sin_ref      # exact, zeros included (+0 == -0)


def test_angle_diagonals(orc):
    for k in range(4):
        m = (1 << 21) + k * (1 << 22)           # pi/4 + k pi/2
        c, s = orc.bm_angle(_b_for_m(m))
        ang = math.pi / 4 + k * math.pi / 2
        assert c == pytest.approx(math.cos(ang), rel=1e-15)
        assert s == pytest.approx(math.sin(ang), rel=1e-15)


def test_radius_exhaustive_vs_extended_precision(orc):
    """All 2^24 radius inputs against x87 extended-precision log/sqrt."""
    m = np.arange(1, TWO24 + 1, dtype=np.uint64)
    a = ((m - 1) << 8).astype(np.uint32)
    rho = orc.bm_radius_many(a)
    u = m.astype(np.longdouble) * np.longdouble(2.0) ** -24
    ref = np.sqrt(np.longdouble(-2.0) * np.log(u))
    err = np.abs(rho.astype(np.longdouble) - ref)
    assert rho[-1] == 0.0
    nz = ref > 0
    assert np.max(err[nz] / ref[nz]) < 4e-16


def test_angle_exhaustive_vs_extended_precision(orc):
    """All 2^24 angle inputs against x87 extended precision.  The reference's
    own argument error is up to ~1e-18 absolute, hence the absolute term."""
    m = np.arange(1, TWO24 + 1, dtype=np.uint64)
    b = ((m - 1) << 8).astype(np.uint32)
    c, s = orc.bm_angle_many(b)
    pi_ld = np.longdouble("3.14159265358979323846264338327950288")
    ang = pi_ld * (m % TWO24).astype(np.longdouble) * np.longdouble(2.0) ** -23
    cref, sref = np.cos(ang), np.sin(ang)
    for got, ref in ((c, cref), (s, sref)):
        err = np.abs(got.astype(np.longdouble) - ref)
        assert np.all(err <= 3e-16 * np.abs(ref) + 2e-18)
        assert np.all(np.sign(got[np.abs(ref) > 1e-15]) == np.sign(ref[np.abs(ref) > 1e-15]))


def test_angle_sample_vs_mpmath(orc):
    """Near the axes the relative error matters; mpmath's cospi/sinpi evaluate
    the dyadic angle exactly at 80 bits."""
    mpmath.mp.prec = 80
    rng = np.random.default_rng(3)
    ms = set(int(x) for x in rng.integers(1, TWO24 + 1, size=3000))
    for axis in range(5):
        for d in range(-40, 41):
            mm = axis * (1 << 22) + d
            if 1 <= mm <= TWO24:
                ms.add(mm)
    for mm in sorted(ms):
        c, s = orc.bm_angle(_b_for_m(mm))
        x = mpmath.mpf(mm % TWO24) / (1 << 23)
        cr, sr = mpmath.cospi(x), mpmath.sinpi(x)
        for got, ref in ((c, cr), (s, sr)):
            if ref == 0:
                assert got == 0.0
            else:
                assert abs((mpmath.mpf(got) - ref) / ref) < 2.5e-16, (mm, got, ref)


def test_normal_equals_rounded_product(orc):
    """z = fp32(rho * cos) for even positions and fp32(rho * sin) for odd ones,
    words (x0, x1) for positions 4q, 4q+1 and (x2, x3) for 4q+2, 4q+3; checked
    against mpmath products (one rounding; the oracle's double product may
    differ by one fp32 ulp only through double rounding)."""
    mpmath.mp.prec = 80
    seed, q0, nb = 77, 1000, 256
    words = orc.blocks(seed, 0, q0, nb).reshape(nb, 4)
    z = orc.normals(seed, 4 * q0, 4 * nb).reshape(nb, 4)
    for q in range(nb):
        for pair in range(2):
            a, b = int(words[q, 2 * pair]), int(words[q, 2 * pair + 1])
            u = mpmath.mpf((a >> 8) + 1) / TWO24
            rho = mpmath.sqrt(-2 * mpmath.log(u))
            x = mpmath.mpf(((b >> 8) + 1) % TWO24) / (1 << 23)
            for odd, trig in ((0, mpmath.cospi(x)), (1, mpmath.sinpi(x))):
                ref = float(np.float32(float(rho * trig)))
                got = float(z[q, 2 * pair + odd])
                ulp = np.spacing(np.float32(abs(ref))) if ref != 0 else 2.0 ** -149
                assert abs(got - ref) <= ulp, (q, pair, odd, got, ref)


def test_normal_moments_and_ks(orc):
    """First four moments of 2^24 draws and a Kolmogorov-Smirnov test against
    Phi.  Bounds are 5 standard errors of each estimator."""
    n = 1 << 24
    z = orc.normals(1, 0, n).astype(np.float64)
    se = 1.0 / math.sqrt(n)
    assert abs(z.mean()) < 5 * se
    assert abs(z.var() - 1.0) < 5 * math.sqrt(2.0) * se
    assert abs(stats.skew(z)) < 5 * math.sqrt(6.0) * se
    assert abs(stats.kurtosis(z)) < 5 * math.sqrt(24.0) * se
    assert stats.kstest(z[: 1 << 20], "norm").pvalue > 1e-3
    assert np.max(np.abs(z)) <= math.sqrt(48 * math.log(2)) + 1e-6  # 24-bit uniform tail cap


def test_normal_positions_are_uncorrelated(orc):
    n = 1 << 22
    z = orc.normals(2, 0, n).reshape(-1, 4).astype(np.float64)
    m = z.shape[0]
    for a, b in ((0, 1), (0, 2), (1, 3), (2, 3)):
        r = np.corrcoef(z[:, a], z[:, b])[0, 1]
        assert abs(r) < 5 / math.sqrt(m)
    # different seeds are independent streams
    z2 = orc.normals(3, 0, n).astype(np.float64)
    assert abs(np.corrcoef(z.reshape(-1), z2)[0, 1]) < 5 / math.sqrt(n)


def test_normal_window_is_prefix_free(orc):
    """Seed replay: any window of the stream is computable on its own."""
    full = orc.normals(9, 0, 4096)
    for j0 in (0, 1, 3, 4, 7, 1001, 4000):
        assert np.array_equal(orc.normals(9, j0, 4096 - j0), full[j0:])
    assert orc.normal(9, 2**40 + 3) == orc.normals(9, 2**40, 8)[3]


# ------------------------------------------------------ seeded normal fill --

def test_fill_normal_reduces_to_the_pinned_noise(orc):
    """Unit scale in fp32 returns the normals themselves: domain 0 is the
    perturbation noise pinned above, and other domains use the same
    transform on their own Philox words."""
    n = 4099
    assert np.array_equal(orc.fill_normal(n, orc.F32, 5, 0, 1.0), orc.normals(5, 0, n))
    for j in (0, 1, 2, 3, 4, 1000, n - 1):
        x = orc.blocks(5, 1, j // 4, 1)
        a, b = (x[0], x[1]) if j % 4 < 2 else (x[2], x[3])
        c, s = orc.bm_angle(int(b))
        ref = np.float32(orc.bm_radius(int(a)) * (s if j % 2 else c))
        assert orc.fill_normal(n, orc.F32, 5, 1, 1.0)[j] == ref
        assert orc.normal_domain(5, 1, j) == ref


def test_fill_normal_scale_rounding_and_zero(orc):
    n = 10000
    z = orc.fill_normal(n, orc.F32, 9, 1, 1.0)
    f = orc.fill_normal(n, orc.F32, 9, 1, 0.02)
    assert np.array_equal(f, (np.float32(0.02) * z).astype(np.float32))          # one fp32 multiply
    h = orc.fill_normal(n, orc.BF16, 9, 1, 0.02)
    assert np.array_equal(h, np.array([orc.f32_to_bf16(float(v)) for v in f], dtype=np.uint16))
    assert not np.any(orc.fill_normal(n, orc.F32, 9, 1, 0.0))


def test_fill_normal_statistics_and_domain_separation(orc):
    n = 1 << 20
    w = orc.fill_normal(n, orc.F32, 0, 1, 0.02).astype(np.float64)
    se = 0.02 / math.sqrt(n)
    assert abs(w.mean()) < 5 * se
    assert abs(w.std() - 0.02) < 5 * 0.02 / math.sqrt(2 * n)
    noise = orc.normals(0, 0, n).astype(np.float64)
    assert abs(np.corrcoef(w, noise)[0, 1]) < 5 / math.sqrt(n)                    # domains are independent
