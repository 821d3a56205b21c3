"""Host checks of the tolerance helpers the GPU tests use: each accepts a
result computed correctly in another rounding order and rejects a plausible
mistake."""
import numpy as np
import pytest

import oracle as O
import synthetic as S
from tests.gpu_helpers import zscore_close


def _device_order_zscores(r, group=None):
    """Z-scores summed the way the device does (sort by group and value;
    lane l of a wave takes entries l, l + 64, ... of the group's run; a
    butterfly over the 64 partial sums), in fp64, rounded to fp32."""
    r = np.asarray(r, dtype=np.float32)
    g = np.zeros(len(r), dtype=np.int64) if group is None else np.asarray(group, dtype=np.int64)
    out = np.zeros(len(r), dtype=np.float32)

    def wave_sum(vals):
        part = np.zeros(64)
        for p, v in enumerate(vals):
            part[p % 64] += v
        m = 32
        while m:
            part = part + part[np.arange(64) ^ m]
            m //= 2
        return part[0]

    for k in np.unique(g):
        idx = np.nonzero(g == k)[0]
        run = np.sort(r[idx].astype(np.float64))
        mu = wave_sum(run) / len(run)
        sd = np.sqrt(wave_sum((run - mu) * (run - mu)) / len(run))
        if sd > 0:
            out[idx] = ((r[idx].astype(np.float64) - mu) / sd).astype(np.float32)
    return out


@pytest.mark.parametrize("kind,n", [("uniform", 8), ("uniform", 30), ("mean_bernoulli", 128), ("uniform", 4096)])
def test_zscore_bound_accepts_another_summation_order(kind, n):
    r = S.rewards(kind, n, 5 + n)
    ref, _ = O.normalize(r, O.NORM_Z)
    got = _device_order_zscores(r)
    assert zscore_close(got, ref, r)
    g = (np.arange(n) % 4).astype(np.int32)
    ref_g, _ = O.normalize(r, O.NORM_Z, g)
    assert zscore_close(_device_order_zscores(r, g), ref_g, r, g)


def test_zscore_bound_rejects_plausible_mistakes():
    r = S.rewards("uniform", 512, 3)
    ref, _ = O.normalize(r, O.NORM_Z)
    r64 = r.astype(np.float64)
    sample_std = ((r64 - r64.mean()) / r64.std(ddof=1)).astype(np.float32)
    assert not zscore_close(sample_std, ref, r)
    fp32_mean = ((r - np.float32(r.mean(dtype=np.float32))) / np.float32(r.std(dtype=np.float32))).astype(np.float32)
    assert not zscore_close(fp32_mean, ref, r) or np.array_equal(fp32_mean, ref)
    off_by_one = ref.copy()
    off_by_one[17] = np.nextafter(np.nextafter(ref[17], np.float32(9)), np.float32(9))   # two ulps
    assert not zscore_close(off_by_one, ref, r)
    const = np.full(16, 0.25, np.float32)
    zero_ref, _ = O.normalize(const, O.NORM_Z)
    assert zscore_close(np.zeros(16, np.float32), zero_ref, const)
    assert not zscore_close(np.full(16, 1e-30, np.float32), zero_ref, const)


def _device_order_update(w_bits, seeds, signs, rnorm, step, j0=0):
    """An update evaluated the way the device does it: fp64 coefficients
    rounded to fp32, an fp32 multiply-add chain over the streams in order of
    first appearance (each step rounded once), one fp32 fma with the fp32
    step, round to bf16."""
    coef = {}
    for sd, sg, r in zip(seeds, signs, rnorm):
        coef[sd] = coef.get(sd, 0.0) + float(sg) * float(r)
    n = len(w_bits)
    acc = np.zeros(n, dtype=np.float32)
    for sd, c in coef.items():
        z = O.normals(sd, j0, n).astype(np.float64)
        acc = (np.float64(np.float32(c)) * z + acc.astype(np.float64)).astype(np.float32)
    w = (w_bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    x = (np.float64(np.float32(step)) * acc.astype(np.float64) + w).astype(np.float32)
    return S.f32_to_bf16_bits(x)


@pytest.mark.parametrize("n,antithetic", [(30, False), (64, True)])
def test_bf16_update_bound_accepts_fp32_accumulation(n, antithetic):
    from tests.gpu_helpers import bf16_update_close, update_slack, update_step_size

    seeds = [s for s in range(1, n // 2 + 1) for _ in (0, 1)] if antithetic else list(range(1, n + 1))
    signs = [1, -1] * (n // 2) if antithetic else [1] * n
    rnorm, _ = O.normalize(S.rewards("uniform", n, 17), O.NORM_Z)
    w = S.host_weights(1 << 14, S.BF16, 3)
    alpha, sigma = np.float32(5e-4), np.float32(2.25e-3)
    step = update_step_size(alpha, sigma, n, 0)
    ref = w.copy()
    O.update(ref, 0, len(w), seeds, signs, rnorm, alpha, sigma, 0)
    got = _device_order_update(w, seeds, signs, rnorm, step)
    slack = lambda k: update_slack(O, seeds, signs, rnorm, step, k)
    assert bf16_update_close(got, ref, slack)
    wrong = _device_order_update(w, seeds, [-signs[0]] + signs[1:], rnorm, step)     # one member's sign flipped
    assert not bf16_update_close(wrong, ref, slack)
