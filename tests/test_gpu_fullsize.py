"""GPU parity at the benchmark's full sizes (4,022,468,096 bf16 parameters),
through the same calls bench.py times.  The oracle cannot process 4 G
parameters, so it checks sampled windows of positions (the counter-based
generator lets it start anywhere: j0 = window start), and properties that hold
at any size are checked on the device: snapshot / master restore is the bitwise
identity over the whole buffer, parameters outside the subspace never change,
and a permutation partition lists every index exactly once, ascending within
each subspace, each entry in the subspace the oracle assigns it to."""
import numpy as np
import pytest

import paper_2608_02391_amd as cp
import synthetic as S
from tests.gpu_helpers import (bf16_close, bf16_update_close, describe_mismatch, bf16_value, f32_close, to_host, torch,
                               ulp_bf16, update_slack, update_step_size, zscore_close)

pytestmark = pytest.mark.gpu

WIN = 1 << 16


@pytest.fixture(scope="module")
def T():
    t = torch()
    assert t.cuda.is_available(), "GPU tests need an MI355X"
    cp.load()
    return t


def _windows(length, rng, n_random=6):
    starts = {0, max(0, length - WIN)}
    for _ in range(n_random):
        starts.add(int(rng.integers(0, max(1, length - WIN))))
    return sorted(starts)


def _say(msg):
    print(msg, flush=True)


def _host_bits(x):
    return to_host(x)


@pytest.fixture(scope="module")
def big(T):
    W = S.workload("c3")
    _say(f"allocating {W.d} bf16 weights")
    w = S.device_weights(W.d, S.BF16, 0)
    T.cuda.synchronize()
    return W, w


def test_c3_layer_group_subspace(orc, T, big):
    W, w = big
    k = 4
    off, L = W.bounds[k], W.sizes()[k]
    sigma = W.sigma_k(k)
    rng = np.random.default_rng(3)
    wins = _windows(L, rng)
    before = {p: _host_bits(w[off + p: off + p + WIN]) for p in wins}
    outside = (_host_bits(w[off - WIN: off]), _host_bits(w[off + L: off + L + WIN]))
    full_before = w.clone()
    s = cp.subspace(off, L)
    snap = T.empty(L, dtype=T.bfloat16, device="cuda")
    _say("c3: perturb with backup")
    cp.cpes_perturb(w, s, sigma, 7, 1, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    T.cuda.synchronize()
    for p in wins:
        ref = before[p].copy()
        orc.perturb(ref, 0, WIN, np.float32(sigma), 7, 1, j0=p)
        got = _host_bits(w[off + p: off + p + WIN])
        assert ulp_bf16(got, ref).max() <= 1, p
    assert np.array_equal(_host_bits(w[off - WIN: off]), outside[0])
    assert np.array_equal(_host_bits(w[off + L: off + L + WIN]), outside[1])
    assert T.equal(snap, full_before[off:off + L])
    _say("c3: perturb from backup, restore")
    cp.cpes_perturb(w, s, sigma, 8, -1, aux=snap, aux_mode=cp.AUX_BACKUP)
    T.cuda.synchronize()
    p = wins[1]
    ref = before[p].copy()
    orc.perturb(ref, 0, WIN, np.float32(sigma), 8, -1, j0=p)
    assert ulp_bf16(_host_bits(w[off + p: off + p + WIN]), ref).max() <= 1
    cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    T.cuda.synchronize()
    assert T.equal(w, full_before)                       # bitwise identity over all 4 G parameters
    _say("c3: update with 30 members")
    seeds, signs = W.member_seeds(0), W.signs
    r = W.rewards(0)
    rn = T.empty(W.n, dtype=T.float32, device="cuda")
    cp.cpes_normalize_rewards(T.from_numpy(r).cuda(), rn, W.norm_mode)
    rn_ref, _ = orc.normalize(r, W.norm_mode)
    cp.cpes_update(w, s, seeds, signs, rn, W.alpha, sigma, W.scale_mode)
    T.cuda.synchronize()
    assert zscore_close(rn.cpu().numpy(), rn_ref, r)
    for p in wins[:4]:
        ref = before[p].copy()
        orc.update(ref, 0, WIN, seeds, signs, rn_ref, np.float32(W.alpha), np.float32(sigma), W.scale_mode, j0=p)
        got = _host_bits(w[off + p: off + p + WIN])
        step = update_step_size(W.alpha, sigma, W.n, W.scale_mode)
        slack = lambda k: update_slack(orc, seeds, signs, rn_ref, step, p + k)
        assert bf16_update_close(got, ref, slack), describe_mismatch(bf16_value(got), bf16_value(ref))
    assert T.equal(w[:off], full_before[:off]) and T.equal(w[off + L:], full_before[off + L:])
    w.copy_(full_before)
    del full_before


def test_c4_permutation_partition_and_gather(orc, T, big):
    W3, w = big
    W = S.workload("c4")
    d, K = W.d, W.K
    _say("c4: partition 4 G indices into 8 subspaces")
    index = T.empty(d, dtype=T.int64, device="cuda")
    ws = T.empty(cp.cpes_partition_workspace_bytes(cp.PART_PERMUTATION, d, K), dtype=T.uint8, device="cuda")
    st = T.full((1,), -1, dtype=T.int32, device="cuda")
    offsets = cp.cpes_partition(cp.PART_PERMUTATION, d, K, W.partition_seed, index=index, workspace=ws, status=st)
    T.cuda.synchronize()
    del ws
    assert int(st.item()) == 0
    assert offsets == [-(-k * d // K) for k in range(K + 1)]
    # every entry sampled lies in the subspace the oracle assigns it to
    rng = np.random.default_rng(5)
    pos = np.sort(rng.integers(0, d, size=20000))
    vals = index[T.from_numpy(pos).cuda()].cpu().numpy()
    ks = np.searchsorted(np.array(offsets), pos, side="right") - 1
    for p, v, k in zip(pos, vals, ks):
        assert orc.bucket(W.partition_seed, d, K, int(v)) == k, (p, v, k)
    # ascending within every subspace, and every index present exactly once
    _say("c4: checking the maps on the device")
    chunk = 1 << 28
    for k in range(K):
        a, b = offsets[k], offsets[k + 1]
        for s0 in range(a, b - 1, chunk):
            e0 = min(b, s0 + chunk + 1)
            seg = index[s0:e0]
            assert bool((seg[1:] > seg[:-1]).all()), (k, s0)
    seen = T.zeros(d, dtype=T.uint8, device="cuda")
    for s0 in range(0, d, chunk):
        seen.index_fill_(0, index[s0:s0 + chunk], 1)
    assert bool(seen.all())
    del seen
    # gather perturb / restore / update on subspace 3
    k = 3
    off, L = offsets[k], offsets[k + 1] - offsets[k]
    sigma = W.sigma_k(k)
    wins = _windows(L, rng, n_random=3)
    idx_w = {p: index[off + p: off + p + WIN].cpu().numpy() for p in wins}
    before = {p: _host_bits(w[T.from_numpy(idx_w[p]).cuda()]) for p in wins}
    full_before = w.clone()
    s = cp.subspace(off, L, index, ascending=True)       # the partition's map is ascending, as bench.py passes it
    snap = T.empty(L, dtype=T.bfloat16, device="cuda")
    _say("c4: gather perturb")
    cp.cpes_perturb(w, s, sigma, 11, 1, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    T.cuda.synchronize()
    for p in wins:
        ref = before[p].copy()
        orc.perturb(ref, 0, WIN, np.float32(sigma), 11, 1, j0=p)
        got = _host_bits(w[T.from_numpy(idx_w[p]).cuda()])
        assert ulp_bf16(got, ref).max() <= 1, p
    changed = (w != full_before)
    mask = T.zeros(d, dtype=T.bool, device="cuda")
    mask[index[off:off + L]] = True
    assert not bool((changed & ~mask).any())               # nothing outside the subspace moved
    del changed, mask
    cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    T.cuda.synchronize()
    assert T.equal(w, full_before)
    _say("c4: whole-line windows and entry-by-entry stores give the same bits")
    plain = cp.subspace(off, L, index)
    cp.cpes_perturb(w, plain, sigma, 13, -1, aux=snap, aux_mode=cp.AUX_BACKUP)
    T.cuda.synchronize()
    via_entries = w.clone()
    cp.cpes_restore(w, plain, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    cp.cpes_perturb(w, s, sigma, 13, -1, aux=snap, aux_mode=cp.AUX_BACKUP)
    T.cuda.synchronize()
    assert T.equal(w, via_entries)
    del via_entries
    cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    T.cuda.synchronize()
    assert T.equal(w, full_before)
    _say("c4: gather update")
    r = W.rewards(0)
    rn = T.from_numpy(orc.normalize(r, W.norm_mode)[0]).cuda()
    cp.cpes_update(w, s, W.member_seeds(0), W.signs, rn, W.alpha, sigma, W.scale_mode)
    T.cuda.synchronize()
    rn_ref = rn.cpu().numpy()
    for p in wins[:3]:
        ref = before[p].copy()
        orc.update(ref, 0, WIN, W.member_seeds(0), W.signs, rn_ref, np.float32(W.alpha), np.float32(sigma),
                   W.scale_mode, j0=p)
        got = _host_bits(w[T.from_numpy(idx_w[p]).cuda()])
        step = update_step_size(W.alpha, sigma, W.n, W.scale_mode)
        slack = lambda k: update_slack(orc, W.member_seeds(0), W.signs, rn_ref, step, p + k)
        assert bf16_update_close(got, ref, slack), describe_mismatch(bf16_value(got), bf16_value(ref))
    w.copy_(full_before)
    # the same partition as a uint32 map (4,022,468,096 < 2^32): identical entries,
    # and a gather perturbation through it gives the same bits as through the int64 map
    _say("c4: uint32 map of the same partition")
    index32 = T.empty(d, dtype=T.int32, device="cuda")
    ws = T.empty(cp.cpes_partition_workspace_bytes(cp.PART_PERMUTATION, d, K), dtype=T.uint8, device="cuda")
    offsets32 = cp.cpes_partition32(d, K, W.partition_seed, index32, ws)
    T.cuda.synchronize()
    del ws
    assert offsets32 == offsets
    for s0 in range(0, d, chunk):
        assert T.equal(index32[s0:s0 + chunk].to(T.int64) & 0xFFFFFFFF, index[s0:s0 + chunk]), s0
    cp.cpes_perturb(w, s, sigma, 12, -1)
    T.cuda.synchronize()
    via64 = w.clone()
    w.copy_(full_before)
    cp.cpes_perturb(w, cp.subspace(off, L, index32, ascending=True), sigma, 12, -1)
    T.cuda.synchronize()
    assert T.equal(w, via64)
    w.copy_(full_before)
    del full_before, index, index32, via64


def test_c5_master_iteration(orc, T, big):
    W3, w = big
    W = S.workload("c5")
    t = 5
    k = W.active[t]
    off, L = W.bounds[k], W.sizes()[k]
    sigma = W.sigma_k(k)
    rng = np.random.default_rng(9)
    wins = _windows(L, rng, n_random=2)
    before = {p: _host_bits(w[off + p: off + p + WIN]) for p in wins}
    full_before = w.clone()
    s = cp.subspace(off, L)
    master = T.empty(L, dtype=T.float32, device="cuda")
    _say("c5: stage master and bf16 backup; perturb from the backup (as bench.py) and from the master; restore")
    cp.cpes_stage_master(w, s, master)
    backup = T.empty(L, dtype=T.bfloat16, device="cuda")
    cp.cpes_backup(w, s, backup)                       # the schedule bench.py times
    T.cuda.synchronize()
    assert T.equal(master, full_before[off:off + L].float())
    assert T.equal(backup, full_before[off:off + L])
    seeds = W.member_seeds(t)
    for m in (0, 1, 127):
        # members perturb from the bf16 backup, the schedule bench.py times; member 1 also
        # from the master, which must give the same 4 G weights bit for bit
        cp.cpes_perturb(w, s, sigma, seeds[m], W.signs[m], aux=backup, aux_mode=cp.AUX_BACKUP)
        if m == 1:
            via_backup = w.clone()
            cp.cpes_perturb(w, s, sigma, seeds[m], W.signs[m], aux=master, aux_mode=cp.AUX_MASTER)
            T.cuda.synchronize()
            assert T.equal(w, via_backup)
            del via_backup
        T.cuda.synchronize()
        p = wins[m % len(wins)]
        ref = before[p].copy()
        mref = orc.bf16_to_f32(before[p]).copy()
        orc.perturb(ref, 0, WIN, np.float32(sigma), seeds[m], W.signs[m], j0=p, aux=mref, aux_mode=orc.AUX_MASTER)
        assert ulp_bf16(_host_bits(w[off + p: off + p + WIN]), ref).max() <= 1
        if m == 1:
            cp.cpes_restore(w, s, aux=master, aux_mode=cp.AUX_MASTER)
        else:
            cp.cpes_restore(w, s, aux=backup, aux_mode=cp.AUX_SNAPSHOT)
        T.cuda.synchronize()
        assert T.equal(w, full_before)
    del backup
    _say("c5: update of master and bf16 weights with 128 antithetic members")
    r = W.rewards(t)
    rn_ref, _ = orc.normalize(r, W.norm_mode)
    cp.cpes_update(w, s, seeds, W.signs, T.from_numpy(rn_ref).cuda(), W.alpha, sigma, W.scale_mode, master=master)
    T.cuda.synchronize()
    for p in wins[:2]:
        mref = orc.bf16_to_f32(before[p]).copy()
        ref = before[p].copy()
        orc.update(ref, 0, WIN, seeds, W.signs, rn_ref, np.float32(W.alpha), np.float32(sigma), W.scale_mode,
                   j0=p, master=mref)
        got_m = master[p:p + WIN].cpu().numpy()
        assert f32_close(got_m, mref), describe_mismatch(got_m, mref)
        got = _host_bits(w[off + p: off + p + WIN])
        step = update_step_size(W.alpha, sigma, W.n, W.scale_mode)
        slack = lambda k: update_slack(orc, seeds, W.signs, rn_ref, step, p + k)
        assert bf16_update_close(got, ref, slack), describe_mismatch(bf16_value(got), bf16_value(ref))
    w.copy_(full_before)


def _chunk_positions(chunks, off, p, n, chunk):
    j = np.arange(p, p + n, dtype=np.int64)
    return chunks[off + j // chunk] * chunk + j % chunk


def test_c4c_chunked_subspaces_and_paper_step(orc, T, big):
    _, w = big
    W = S.workload("c4c")
    d, K, C = W.d, W.K, W.chunk
    _say("c4c: chunk partition of 4 G parameters (chunks of 65,536)")
    n_chunks = -(-d // C)
    chunks = T.empty(n_chunks, dtype=T.int64, device="cuda")
    ws = T.empty(cp.cpes_partition_chunks_workspace_bytes(d, C, K), dtype=T.uint8, device="cuda")
    offs, lens = cp.cpes_partition_chunks(d, C, K, W.partition_seed, chunks, ws)
    r_offs, r_lens, r_chunks = orc.partition_chunks(d, C, K, W.partition_seed)
    T.cuda.synchronize()
    assert offs == [int(x) for x in r_offs] and lens == [int(x) for x in r_lens]
    h_chunks = to_host(chunks)
    assert np.array_equal(h_chunks, r_chunks)
    rng = np.random.default_rng(11)
    k = 2
    off, L = offs[k], lens[k]
    sigma = float(np.float32(W.sigma * np.sqrt(d / L)))
    wins = _windows(L, rng, n_random=4)
    pos = {p: _chunk_positions(h_chunks, off, p, WIN, C) for p in wins}
    before = {p: _host_bits(w[T.from_numpy(pos[p]).cuda()]) for p in wins}
    full_before = w.clone()
    s = cp.subspace(off, L, chunks, C)
    snap = T.empty(L, dtype=T.bfloat16, device="cuda")
    _say("c4c: chunked perturb with backup, from backup, restore")
    cp.cpes_perturb(w, s, sigma, 21, 1, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    T.cuda.synchronize()
    for p in wins:
        ref = before[p].copy()
        orc.perturb(ref, 0, WIN, np.float32(sigma), 21, 1, j0=p)
        assert ulp_bf16(_host_bits(w[T.from_numpy(pos[p]).cuda()]), ref).max() <= 1, p
    cp.cpes_perturb(w, s, sigma, 22, -1, aux=snap, aux_mode=cp.AUX_BACKUP)
    cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    T.cuda.synchronize()
    assert T.equal(w, full_before)
    # one CoPES step as the paper runs it: K = 4, N = 40, joint z-score, alpha / N_k
    P = S.workload("p0")
    _say("p0: one step update over 4 chunked subspaces, 40 members")
    p_chunks = T.empty(-(-d // P.chunk), dtype=T.int64, device="cuda")
    p_ws = T.empty(cp.cpes_partition_chunks_workspace_bytes(d, P.chunk, P.K), dtype=T.uint8, device="cuda")
    p_offs, p_lens = cp.cpes_partition_chunks(d, P.chunk, P.K, P.partition_seed, p_chunks, p_ws)
    T.cuda.synchronize()
    hp = to_host(p_chunks)
    seeds, ks = P.member_seeds(0), P.member_subspaces()
    rhat, _ = orc.normalize(P.rewards(0), P.norm_mode)
    sigmas = [float(np.float32(P.sigma * np.sqrt(d / p_lens[k]))) for k in range(P.K)]
    p_pos, p_before = {}, {}
    for kk in range(P.K):
        p = int(rng.integers(0, p_lens[kk] - WIN))
        p_pos[kk] = (p, _chunk_positions(hp, p_offs[kk], p, WIN, P.chunk))
        p_before[kk] = _host_bits(w[T.from_numpy(p_pos[kk][1]).cuda()])
    cp.cpes_update_step(w, p_offs, seeds, P.signs, ks, T.from_numpy(rhat).cuda(), P.alpha, sigmas, P.scale_mode,
                        index=p_chunks, chunk=P.chunk, lengths=p_lens)
    T.cuda.synchronize()
    for kk in range(P.K):
        p, ps = p_pos[kk]
        sel = [i for i in range(P.n) if ks[i] == kk]
        ref = p_before[kk].copy()
        orc.update(ref, 0, WIN, [seeds[i] for i in sel], [P.signs[i] for i in sel], rhat[sel], np.float32(P.alpha),
                   np.float32(sigmas[kk]), P.scale_mode, j0=p)
        got = _host_bits(w[T.from_numpy(ps).cuda()])
        step = update_step_size(P.alpha, sigmas[kk], len(sel), P.scale_mode)
        slack = lambda k: update_slack(orc, [seeds[i] for i in sel], [P.signs[i] for i in sel], rhat[sel], step, p + k)
        assert bf16_update_close(got, ref, slack), describe_mismatch(bf16_value(got), bf16_value(ref))
    w.copy_(full_before)


def test_host_backup_full_size(orc, T, big):
    """The weight backup in pinned host memory at full subspace sizes: a c3
    layer group (one DMA copy each way) and a c4c chunked subspace (kernels
    reading and writing the pinned buffer).  Sampled windows of the backup
    equal the weights they were taken from; after a perturbation, the restore
    from host memory returns the whole 4 G buffer to its bits."""
    W, w = big
    full_before = w.clone()
    rng = np.random.default_rng(5)
    k = 4
    off, L = W.bounds[k], W.sizes()[k]
    hb = T.empty(L, dtype=T.bfloat16, pin_memory=True)
    _say("host backup: c3 layer group, DMA")
    cp.cpes_backup_to_host(w, cp.subspace(off, L), hb)
    T.cuda.synchronize()
    hbits = to_host(hb)
    for p in _windows(L, rng, n_random=3):
        assert np.array_equal(hbits[p:p + WIN], _host_bits(w[off + p: off + p + WIN])), p
    cp.cpes_perturb(w, cp.subspace(off, L), W.sigma_k(k), 31, 1)
    cp.cpes_restore_from_host(w, cp.subspace(off, L), hb)
    T.cuda.synchronize()
    assert T.equal(w, full_before)
    del hb, hbits
    C4 = S.workload("c4c")
    _say("host backup: c4c chunked subspace, zero-copy kernels")
    chunks = T.empty(-(-C4.d // C4.chunk), dtype=T.int64, device="cuda")
    ws = T.empty(cp.cpes_partition_chunks_workspace_bytes(C4.d, C4.chunk, C4.K), dtype=T.uint8, device="cuda")
    offs, lens = cp.cpes_partition_chunks(C4.d, C4.chunk, C4.K, C4.partition_seed, chunks, ws)
    T.cuda.synchronize()
    h_chunks = to_host(chunks)
    k = C4.K - 1                                     # holds the short last chunk or not; either way ragged-safe
    off, L = offs[k], lens[k]
    s = cp.subspace(off, L, chunks, C4.chunk)
    hb = T.empty(L, dtype=T.bfloat16, pin_memory=True)
    cp.cpes_backup_to_host(w, s, hb)
    T.cuda.synchronize()
    hbits = to_host(hb)
    for p in _windows(L, rng, n_random=3):
        pos = _chunk_positions(h_chunks, off, p, WIN, C4.chunk)
        assert np.array_equal(hbits[p:p + WIN], _host_bits(w[T.from_numpy(pos).cuda()])), p
    cp.cpes_perturb(w, s, float(np.float32(C4.sigma * np.sqrt(C4.d / L))), 32, -1)
    T.cuda.synchronize()
    assert not T.equal(w, full_before)
    cp.cpes_restore_from_host(w, s, hb)
    T.cuda.synchronize()
    assert T.equal(w, full_before)
