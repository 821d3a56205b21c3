"""Pins of the oracle's perturb / restore / normalise / update against what the
paper and mathematics fix: Eq. (5), (6), (8), (10)-(13), Alg. 1 and the
weight-backup argument of Sec. 3.3.  Brute-force references are written as
explicit sums over members (no folding of mirrored pairs), in exact rational or
extended-precision arithmetic, with noise vectors taken from the separately
pinned generator."""
import math
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import synthetic as S


def f32(x):
    return np.float32(x)


def _is_correct_rounding_f32(r: float, exact: Fraction) -> bool:
    """r is the round-to-nearest-even fp32 value of `exact`."""
    rf = Fraction(float(r))
    ulp = Fraction(float(np.spacing(np.float32(abs(r))))) if r != 0 else Fraction(2) ** -149
    diff = abs(rf - exact)
    if diff < ulp / 2:
        return True
    if diff == ulp / 2:
        bits = np.array([r], dtype=np.float32).view(np.uint32)[0]
        return (int(bits) & 1) == 0
    return False


# ------------------------------------------------------------- bf16 storage --

def test_bf16_rounding_matches_torch(orc):
    """RNE fp32 -> bf16 (reading A11) against torch's conversion, through the
    master-restore path, on random bit patterns and every tie pattern class."""
    rng = np.random.default_rng(11)
    bits = rng.integers(0, 2**32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    ties = (rng.integers(0, 2**16, size=4096, dtype=np.uint64).astype(np.uint32) << 16) | 0x8000
    near = np.concatenate([ties - 1, ties + 1])
    bits = np.concatenate([bits, ties, near]).astype(np.uint32)
    x = bits.view(np.float32)
    finite = np.isfinite(x)
    master = x.copy()
    w = np.zeros(x.size, dtype=np.uint16)
    orc.restore(w, 0, x.size, 0.0, 0, 1, aux=master, aux_mode=orc.AUX_MASTER)
    ref = S.f32_to_bf16_bits(x)
    assert np.array_equal(w[finite], ref[finite])
    # NaN stays NaN (quiet), infinities stay infinities
    got = orc.bf16_to_f32(w)
    assert np.all(np.isnan(got[np.isnan(x)]))
    assert np.all(got[np.isinf(x)] == x[np.isinf(x)])


# ----------------------------------------------------------------- perturb --

@pytest.mark.parametrize("dtype", [S.F32, S.BF16])
def test_perturb_sigma_zero_is_identity(orc, dtype):
    w = S.host_weights(5000, dtype, 1)
    w0 = w.copy()
    orc.perturb(w, 100, 4000, 0.0, 5, 1)
    assert np.array_equal(w, w0)


def test_perturb_is_one_fp32_fma(orc):
    """theta_{k,i} = theta + sigma_k eps (Eq. 8) with one rounding, checked exactly."""
    n, off, sigma, seed = 3000, 17, f32(2e-3), 42
    w = S.host_weights(n + 50, S.F32, 2)
    w0 = w.copy()
    for sign in (1, -1):
        w[:] = w0
        orc.perturb(w, off, n, sigma, seed, sign)
        z = orc.normals(seed, 0, n)
        for j in range(0, n, 7):
            exact = Fraction(float(w0[off + j])) + sign * Fraction(float(sigma)) * Fraction(float(z[j]))
            assert _is_correct_rounding_f32(w[off + j], exact), j
    assert np.array_equal(w[:off], w0[:off]) and np.array_equal(w[off + n:], w0[off + n:])


def test_perturb_bf16_is_fp32_fma_then_rne(orc):
    n, sigma, seed = 20000, f32(3e-3), 7
    wb = S.host_weights(n, S.BF16, 3)
    wf = orc.bf16_to_f32(wb).copy()
    orc.perturb(wb, 0, n, sigma, seed, -1)
    orc.perturb(wf, 0, n, sigma, seed, -1)
    assert np.array_equal(wb, S.f32_to_bf16_bits(wf))


def test_perturb_touches_only_the_subspace_index_map(orc):
    d = 4096
    rng = np.random.default_rng(5)
    idx = np.sort(rng.choice(d, size=700, replace=False)).astype(np.int64)
    index = np.concatenate([np.zeros(13, dtype=np.int64), idx])  # map entries start at offset 13
    w = S.host_weights(d, S.BF16, 4)
    w0 = w.copy()
    snap = np.empty(idx.size, dtype=np.uint16)
    orc.perturb(w, 13, idx.size, f32(0.05), 3, 1, index=index, aux=snap, aux_mode=orc.AUX_SNAPSHOT)
    outside = np.setdiff1d(np.arange(d), idx)
    assert np.array_equal(w[outside], w0[outside])
    assert np.array_equal(snap, w0[idx])
    assert np.mean(w[idx] != w0[idx]) > 0.9
    # the j-th map entry gets noise position j
    z = orc.normals(3, 0, idx.size)
    expect = S.f32_to_bf16_bits(np.array([np.float32(orc.bf16_to_f32(w0[i])) for i in idx], dtype=np.float32)
                                + np.float32(0.05) * z)
    assert np.mean(w[idx] == expect) > 0.99


def test_perturbation_norm_matches_dimension_aware_scale(orc):
    """E||sigma_k P_k eps||^2 = d_k sigma_k^2 = d sigma^2 (Eq. 10-11), K = 4."""
    K, dk, sigma = 4, 1 << 20, 1e-3
    d = K * dk
    sk = f32(sigma * math.sqrt(K))
    assert sk == f32(2e-3)  # Table S2: sigma_k = 2e-3 for K = 4, sigma = 1e-3
    w = np.zeros(dk, dtype=np.float32)
    orc.perturb(w, 0, dk, sk, 123, 1)
    ratio = float(np.sum(w.astype(np.float64) ** 2)) / (d * sigma * sigma)
    assert abs(ratio - 1.0) < 4 * math.sqrt(2.0 / dk)


# ----------------------------------------------------------------- restore --

@pytest.mark.parametrize("dtype", [S.F32, S.BF16])
def test_snapshot_restore_is_bitwise_identity(orc, dtype):
    w = S.host_weights(10000, dtype, 6)
    w0 = w.copy()
    snap = np.empty(9000, dtype=w.dtype)
    orc.perturb(w, 500, 9000, f32(4e-3), 77, -1, aux=snap, aux_mode=orc.AUX_SNAPSHOT)
    assert not np.array_equal(w, w0)
    orc.restore(w, 500, 9000, f32(4e-3), 77, -1, aux=snap, aux_mode=orc.AUX_SNAPSHOT)
    assert np.array_equal(w, w0)


def test_master_perturb_and_restore(orc):
    n = 8000
    w = S.host_weights(n, S.BF16, 8)
    w0 = w.copy()
    master = orc.stage_master(w, 0, n)
    assert np.array_equal(master, orc.bf16_to_f32(w0))            # staging is exact
    orc.perturb(w, 0, n, f32(4e-3), 9, 1, aux=master, aux_mode=orc.AUX_MASTER)
    m2 = master.copy()
    orc.perturb(m2, 0, n, f32(4e-3), 9, 1)                          # fp32 perturb of the master
    assert np.array_equal(w, S.f32_to_bf16_bits(m2))
    orc.restore(w, 0, n, f32(4e-3), 9, 1, aux=master, aux_mode=orc.AUX_MASTER)
    assert np.array_equal(w, w0)


@pytest.mark.parametrize("dtype", [S.F32, S.BF16])
def test_perturb_from_backup_is_restore_then_perturb(orc, dtype):
    """One backup of the pre-update weights serves every member (Sec. 3.3):
    perturbing from the backup equals restoring from it and perturbing."""
    n, off = 5000, 40
    w = S.host_weights(n + 100, dtype, 12)
    backup = w[off:off + n].copy()
    orc.perturb(w, off, n, f32(3e-3), 5, 1)                         # member 1 perturbed, not restored
    a = w.copy()
    orc.perturb(a, off, n, f32(3e-3), 6, -1, aux=backup, aux_mode=orc.AUX_BACKUP)
    b = w.copy()
    b[off:off + n] = backup
    orc.perturb(b, off, n, f32(3e-3), 6, -1)
    assert np.array_equal(a, b)
    assert np.array_equal(backup, S.host_weights(n + 100, dtype, 12)[off:off + n])  # the backup is read only


def test_replay_restore_is_not_an_identity_but_is_bounded(orc):
    """Sec. 3.3 keeps a backup because (w + d) - d != w in floating point.
    reading A10: replay restore errs by at most one fp32 ulp of max(|w|, |w'|)."""
    n = 1 << 18
    w = S.host_weights(n, S.F32, 10)
    w0 = w.copy()
    orc.perturb(w, 0, n, f32(2e-3), 31, 1)
    wp = w.copy()
    orc.restore(w, 0, n, f32(2e-3), 31, 1)                         # replay-subtract
    diff = np.abs(w.astype(np.float64) - w0.astype(np.float64))
    bound = np.spacing(np.maximum(np.abs(w0), np.abs(wp)).astype(np.float32)).astype(np.float64)
    assert np.all(diff <= bound)
    assert np.count_nonzero(diff) > 0                               # not an identity
    # the textbook counterexample in fp32: (1 + 2^-23) + 2^-24 - 2^-24 != 1 + 2^-23
    a, dlt = f32(1 + 2.0 ** -23), f32(2.0 ** -24)
    assert (a + dlt) - dlt != a


# --------------------------------------------------------------- normalise --

def test_z_normalisation_matches_numpy(orc):
    """Eq. (5)/(12): mean and population std (ddof = 0)."""
    r = S.rewards("uniform", 40, 99)
    out, st = orc.normalize(r, orc.NORM_Z)
    r64 = r.astype(np.float64)
    ref = (r64 - r64.mean()) / r64.std(ddof=0)
    assert st == 0
    assert np.allclose(out, ref, rtol=1e-6, atol=1e-7)
    assert abs(float(np.mean(out.astype(np.float64)))) < 40 * 2.0 ** -23
    assert abs(float(np.var(out.astype(np.float64))) - 1.0) < 40 * 2.0 ** -23


def test_z_normalisation_affine_invariant(orc):
    r = S.rewards("uniform", 64, 5)
    a, _ = orc.normalize(r, orc.NORM_Z)
    b, _ = orc.normalize((3.5 * r.astype(np.float64) - 2.0).astype(np.float32), orc.NORM_Z)
    assert np.allclose(a, b, rtol=1e-5, atol=1e-6)


def test_z_normalisation_constant_and_nonfinite(orc):
    out, st = orc.normalize(np.full(10, 0.3, dtype=np.float32), orc.NORM_Z)
    assert st == 0 and np.all(out == 0)
    r = S.rewards("uniform", 10, 1)
    for bad in (np.nan, np.inf, -np.inf):
        rr = r.copy()
        rr[4] = bad
        out, st = orc.normalize(rr, orc.NORM_Z)
        assert st == 1 and np.all(out == 0)


def test_rank_normalisation_matches_scipy(orc):
    """reading A7: centred average ranks, ties averaged."""
    for kind, n in (("bernoulli", 32), ("uniform", 33), ("mean_bernoulli", 128)):
        r = S.rewards(kind, n, 3)
        out, st = orc.normalize(r, orc.NORM_RANK)
        ref = (stats.rankdata(r, method="average") - 1.0) / (n - 1) - 0.5
        assert st == 0
        assert np.array_equal(out, ref.astype(np.float32))
        assert abs(float(out.astype(np.float64).sum())) < 1e-5
        assert out.min() >= -0.5 and out.max() <= 0.5
    out, _ = orc.normalize(np.array([0.7], dtype=np.float32), orc.NORM_RANK)
    assert out[0] == 0.0


@pytest.mark.parametrize("mode", [0, 1])
def test_grouped_normalisation_equals_per_group_joint(orc, mode):
    """Independent standardisation (the ablation of Sec. 4.4) = joint
    standardisation applied to each group alone."""
    n, K = 40, 4
    r = S.rewards("uniform", n, 12)
    group = np.repeat(np.arange(K), n // K)[np.random.default_rng(1).permutation(n)].astype(np.int32)
    out, _ = orc.normalize(r, mode, group)
    for g in range(K):
        sel = group == g
        ref, _ = orc.normalize(r[sel], mode)
        assert np.array_equal(out[sel], ref)


# ------------------------------------------------------------------ update --

@pytest.mark.parametrize("scale_mode", [0, 1])
@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_update_brute_force_fp32(orc, n, scale_mode):
    rng = np.random.default_rng(100 + n + 10 * scale_mode)
    L = 64
    seeds = [int(x) for x in rng.integers(1, 2**63, size=n)]
    if n >= 3:
        seeds[2] = seeds[1]                      # a mirrored pair shares its seed
    signs = [1] * n
    if n >= 3:
        signs[2] = -1
    rnorm = rng.standard_normal(n).astype(np.float32)
    alpha, sigma = f32(5e-4), f32(2e-3)
    j0 = int(rng.integers(0, 2**40))
    w = S.host_weights(L, S.F32, n)
    w0 = w.copy()
    orc.update(w, 0, L, seeds, signs, rnorm, alpha, sigma, scale_mode, j0=j0)
    step = (Fraction(float(alpha)) / (n * Fraction(float(sigma)))) if scale_mode == 0 else \
        Fraction(float(alpha)) / n
    z = [orc.normals(s, j0, L) for s in seeds]
    for j in range(L):
        acc = sum(Fraction(sg) * Fraction(float(rn)) * Fraction(float(zz[j]))
                  for sg, rn, zz in zip(signs, rnorm, z))
        exact = Fraction(float(w0[j])) + step * acc
        ref = np.float32(float(exact))
        ulp = np.spacing(np.float32(abs(ref)))
        assert abs(float(w[j]) - float(exact)) <= float(ulp), (j, w[j], float(exact))


def test_update_bf16_and_master(orc):
    n, L = 4, 64
    seeds, signs = [5, 5, 9, 11], [1, -1, 1, 1]
    rnorm = np.array([0.9, -1.3, 0.2, 0.4], dtype=np.float32)
    wb = S.host_weights(L, S.BF16, 21)
    wf = orc.bf16_to_f32(wb).copy()
    master = wf.copy()
    wm = wb.copy()
    orc.update(wb, 0, L, seeds, signs, rnorm, f32(5e-4), f32(4e-3))
    orc.update(wf, 0, L, seeds, signs, rnorm, f32(5e-4), f32(4e-3))
    assert np.array_equal(wb, S.f32_to_bf16_bits(wf))              # bf16 = fp32 result rounded
    orc.update(wm, 0, L, seeds, signs, rnorm, f32(5e-4), f32(4e-3), master=master)
    assert np.array_equal(master, wf)                               # master carries the fp32 value
    assert np.array_equal(wm, S.f32_to_bf16_bits(master))


def test_update_one_hot_reward(orc):
    L = 256
    w = S.host_weights(L, S.F32, 30)
    w0 = w.copy()
    seeds, signs = [3, 4, 5], [1, 1, -1]
    rn = np.array([0.0, 0.0, 1.0], dtype=np.float32)
    orc.update(w, 0, L, seeds, signs, rn, f32(5e-4), f32(2e-3), 1)
    step = 5e-4 / 3
    z = orc.normals(5, 0, L).astype(np.float64)
    ref = (w0.astype(np.float64) - step * z).astype(np.float32)
    assert np.max(np.abs(w - ref)) <= np.max(np.spacing(np.abs(ref)))


def test_update_mirrored_equal_rewards_leave_theta_unchanged(orc):
    L = 1000
    w = S.host_weights(L, S.BF16, 31)
    w0 = w.copy()
    orc.update(w, 0, L, [7, 7, 8, 8], [1, -1, 1, -1], np.array([0.5, 0.5, -2.0, -2.0], np.float32),
               f32(5e-4), f32(4e-3))
    assert np.array_equal(w, w0)


def test_update_equal_rewards_leave_theta_unchanged(orc):
    L = 1000
    w = S.host_weights(L, S.F32, 32)
    w0 = w.copy()
    rn, _ = orc.normalize(np.full(6, 0.25, dtype=np.float32), orc.NORM_Z)
    orc.update(w, 0, L, [1, 2, 3, 4, 5, 6], [1] * 6, rn, f32(5e-4), f32(2e-3))
    assert np.array_equal(w, w0)


def test_k1_paper_scale_is_standard_es(orc):
    """K = 1 with step alpha / N is the standard ES update of Eq. (6)
    (Table 3: 'K=1 (Std. ES)')."""
    d, N = 512, 8
    w = S.host_weights(d, S.F32, 40)
    w0 = w.copy()
    seeds = list(range(101, 101 + N))
    r = S.rewards("uniform", N, 4)
    rhat, _ = orc.normalize(r, orc.NORM_Z)
    offsets, _ = orc.partition(orc.PART_CONTIGUOUS, d, 1)
    assert list(offsets) == [0, d]
    orc.update(w, 0, d, seeds, [1] * N, rhat, f32(5e-4), f32(1e-3), orc.SCALE_ALPHA_OVER_N)
    eps = np.stack([orc.normals(s, 0, d).astype(np.longdouble) for s in seeds])
    ref = w0.astype(np.longdouble) + np.longdouble(float(f32(5e-4))) / N * (rhat.astype(np.longdouble) @ eps)
    assert np.max(np.abs(w.astype(np.longdouble) - ref) / np.spacing(np.abs(ref.astype(np.float32)))) <= 1.0


def test_copes_step_composition(orc):
    """One CoPES step (Alg. 1; Eq. 12-13) on a permutation partition: K = 4,
    N = 40 (N_k = 10), sigma_k = 2e-3, alpha = 5e-4, joint z-score, step
    alpha / N_k.  The per-subspace updates compose in any order to the same
    parameters (disjoint supports), equal to the explicit sum."""
    d, K, Nk = 1 << 14, 4, 10
    N = K * Nk
    offsets, index = orc.partition(orc.PART_PERMUTATION, d, K, seed=33)
    seeds = list(range(1, N + 1))
    r = S.rewards("uniform", N, 99)
    rhat, _ = orc.normalize(r, orc.NORM_Z)                # joint over all N (Eq. 12)
    w0 = S.host_weights(d, S.F32, 50)

    def step_in_order(order):
        w = w0.copy()
        for k in order:
            sl = slice(k * Nk, (k + 1) * Nk)
            orc.update(w, int(offsets[k]), int(offsets[k + 1] - offsets[k]), seeds[sl], [1] * Nk,
                       rhat[sl], f32(5e-4), f32(2e-3), orc.SCALE_ALPHA_OVER_N, index=index)
        return w

    a = step_in_order([0, 1, 2, 3])
    b = step_in_order([3, 1, 0, 2])
    assert np.array_equal(a, b)
    c = w0.copy()                                         # the one-call form of the same step
    orc.update_step(c, offsets, seeds, [1] * N, np.repeat(np.arange(K), Nk), rhat, f32(5e-4), [f32(2e-3)] * K,
                    orc.SCALE_ALPHA_OVER_N, index=index)
    assert np.array_equal(a, c)
    ref = w0.astype(np.longdouble).copy()
    for k in range(K):
        pos = index[offsets[k]:offsets[k + 1]]
        g = np.zeros(pos.size, dtype=np.longdouble)
        for i in range(Nk):
            m = k * Nk + i
            g += np.longdouble(float(rhat[m])) * orc.normals(seeds[m], 0, pos.size).astype(np.longdouble)
        ref[pos] += np.longdouble(float(f32(5e-4))) * g / Nk
    err = np.abs(a.astype(np.longdouble) - ref) / np.spacing(np.abs(ref.astype(np.float32)))
    assert np.max(err) <= 1.0


def test_update_step_k1_is_standard_es_and_skips_empty_subspaces(orc):
    """K = 1 with alpha / N is Eq. 6; a subspace without members is unchanged."""
    d, N = 300, 6
    w0 = S.host_weights(d, S.F32, 60)
    seeds = list(range(7, 7 + N))
    rhat, _ = orc.normalize(S.rewards("uniform", N, 8), orc.NORM_Z)
    a = w0.copy()
    orc.update_step(a, [0, d], seeds, [1] * N, [0] * N, rhat, f32(5e-4), [f32(1e-3)], orc.SCALE_ALPHA_OVER_N)
    b = w0.copy()
    orc.update(b, 0, d, seeds, [1] * N, rhat, f32(5e-4), f32(1e-3), orc.SCALE_ALPHA_OVER_N)
    assert np.array_equal(a, b)
    eps = np.stack([orc.normals(s, 0, d).astype(np.longdouble) for s in seeds])
    ref = w0.astype(np.longdouble) + np.longdouble(float(f32(5e-4))) / N * (rhat.astype(np.longdouble) @ eps)
    assert np.max(np.abs(a.astype(np.longdouble) - ref) / np.spacing(np.abs(ref.astype(np.float32)))) <= 1.0
    c = w0.copy()
    orc.update_step(c, [0, 100, 200, 300], seeds, [1] * N, [0, 0, 2, 2, 0, 2], rhat, f32(5e-4), [f32(2e-3)] * 3)
    assert np.array_equal(c[100:200], w0[100:200]) and not np.array_equal(c[:100], w0[:100])
