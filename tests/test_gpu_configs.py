"""Parity on the two small benchmark configurations, end to end, on every
output of the step: the 1,048,576-parameter fp32 workload's active subspace
(8 members), and subspace 3 of the 150,994,944-parameter bf16 workload (32
antithetic members, rank-normalised Bernoulli rewards).  The device runs the
sequence bench.py times -- the first member writes the backup, later members
perturb the restored weights in place, a restore follows every member, then
normalise and update -- and the oracle runs the same sequence on the host.
Restores and normalised rewards must match bit for bit; perturbed and updated
weights within the bar of the other parity tests."""
import numpy as np
import pytest

import paper_2608_02391_amd as cp
import synthetic as S
from tests.gpu_helpers import (bf16_close, bf16_update_close, bf16_value, describe_mismatch, f32_close, to_dev, to_host,
                               torch, ulp_bf16, update_slack, update_step_size, zscore_close)

pytestmark = pytest.mark.gpu


def _check_close(dtype, got, ref, what):
    if dtype == S.BF16:
        assert ulp_bf16(got, ref).max() <= 1, what
    else:
        assert f32_close(got, ref), (what, describe_mismatch(got, ref))


@pytest.mark.parametrize("name,k", [("c1", 0), ("c2", 3)])
def test_benchmark_config_step(orc, name, k):
    T = torch()
    assert T.cuda.is_available(), "GPU tests need an MI355X"
    cp.load()
    W = S.workload(name)
    offs = cp.cpes_partition(cp.PART_CONTIGUOUS, W.d, W.K, bounds=W.bounds)
    off, L = offs[k], offs[k + 1] - offs[k]
    w = S.host_weights(W.d, W.dtype, 7)
    dw = to_dev(w)
    s = cp.subspace(off, L)
    sigma = np.float32(W.sigma_k(k))
    backup_d = T.empty(L, dtype=dw.dtype, device="cuda")
    backup_h = np.zeros(L, dtype=w.dtype)
    seeds, signs = W.member_seeds(0), W.signs
    for m, (seed, sign) in enumerate(zip(seeds, signs)):
        mode = cp.AUX_SNAPSHOT if m == 0 else cp.AUX_NONE
        cp.cpes_perturb(dw, s, float(sigma), seed, sign, aux=backup_d, aux_mode=mode)
        orc.perturb(w, off, L, sigma, seed, sign, aux=backup_h if m == 0 else None,
                    aux_mode=orc.AUX_SNAPSHOT if m == 0 else orc.AUX_NONE)
        T.cuda.synchronize()
        _check_close(W.dtype, to_host(dw)[off:off + L], w[off:off + L], f"member {m} perturbed")
        cp.cpes_restore(dw, s, aux=backup_d, aux_mode=cp.AUX_SNAPSHOT)
        orc.restore(w, off, L, 0.0, 0, 1, aux=backup_h, aux_mode=orc.AUX_SNAPSHOT)
        T.cuda.synchronize()
        assert np.array_equal(to_host(dw), w), f"member {m} restored"
    r = W.rewards(0)
    rn_d = T.empty(len(r), dtype=T.float32, device="cuda")
    cp.cpes_normalize_rewards(T.from_numpy(r).cuda(), rn_d, W.norm_mode)
    rn_h, status = orc.normalize(r, W.norm_mode)
    T.cuda.synchronize()
    assert status == 0
    if W.norm_mode == cp.NORM_RANK:
        assert np.array_equal(to_host(rn_d), rn_h)
    else:
        assert zscore_close(to_host(rn_d), rn_h, r)
    cp.cpes_update(dw, s, seeds, signs, rn_d, W.alpha, float(sigma), W.scale_mode)
    orc.update(w, off, L, seeds, signs, rn_h, np.float32(W.alpha), sigma, W.scale_mode)
    T.cuda.synchronize()
    got = to_host(dw)
    if W.dtype == S.BF16:
        step = update_step_size(W.alpha, sigma, W.n, W.scale_mode)
        slack = lambda k: update_slack(orc, seeds, signs, rn_h, step, k)
        assert bf16_update_close(got[off:off + L], w[off:off + L], slack), \
            describe_mismatch(bf16_value(got[off:off + L]), bf16_value(w[off:off + L]))
    else:
        assert f32_close(got[off:off + L], w[off:off + L])
    outside = np.ones(W.d, dtype=bool)
    outside[off:off + L] = False
    assert np.array_equal(got[outside], w[outside])             # nothing outside the subspace moved
