"""GPU parity: every entry point of libcpes (called through the C ABI) against
the CPU oracle, element by element, on the same seeded inputs.  Sizes span many
workgroups and a ragged tail; offsets include unaligned ones; index-map
(gather/scatter) subspaces come from the oracle's own partition.

Tolerances: Philox words, index maps, snapshots and restores bit-exact;
normals within 2 fp32 ulp; bf16 results within 1 bf16 ulp; fp32 results within
1e-5 relative + 1e-7 absolute."""
import functools

import numpy as np
import pytest

import paper_2608_02391_amd as cp
import synthetic as S
from tests.gpu_helpers import (bf16_close, bf16_update_close, bf16_value, describe_mismatch, f32_close,
                               normals_within_2ulp, to_dev, update_slack, update_step_size, zscore_close,
                               to_host, torch, ulp_bf16, ulp_f32)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    t = torch()
    assert t.cuda.is_available(), "GPU tests need an MI355X"
    cp.load()
    return t


def _sync(T):
    T.cuda.synchronize()


# ------------------------------------------------------------------ Philox --

@pytest.mark.parametrize("seed,domain,q0,nb", [
    (0, 0, 0, 1 << 16),
    (33, 3, (5 << 32) - 100, 4096),          # crosses the hi word of the counter
    (2**64 - 1, 0, 2**40 + 7, 1000),
    (123456789012345, 2, 17, 77777),
])
def test_philox_streams_bit_exact(orc, T, seed, domain, q0, nb):
    out = T.empty(4 * nb, dtype=T.int32, device="cuda")
    cp.cpes_debug_philox(seed, domain, q0, nb, out)
    got = to_host(out).view(np.uint32)
    ref = orc.blocks(seed, domain, q0, nb)
    assert np.array_equal(got, ref)


# -------------------------------------------------------------- transform --

def test_box_muller_halves_exhaustive(orc, T):
    """Radius and angle on the whole 2^24-point uniform grid against the oracle."""
    n = 1 << 24
    rho = T.empty(n, dtype=T.float64, device="cuda")
    c = T.empty(n, dtype=T.float64, device="cuda")
    s = T.empty(n, dtype=T.float64, device="cuda")
    cp.cpes_debug_bm_grid(1, n, rho, c, s)
    words = ((np.arange(1, n + 1, dtype=np.uint64) - 1) << 8).astype(np.uint32)
    r_ref = orc.bm_radius_many(words)
    c_ref, s_ref = orc.bm_angle_many(words)
    g_rho, g_c, g_s = to_host(rho), to_host(c), to_host(s)
    # U = 1 has radius 0; the device returns about 2^-200 there (the square
    # root of the log table's 2^-400), which still gives a zero normal in fp32.
    # The angle's zeros are exact.
    at_one = g_rho[r_ref == 0]
    assert at_one.size == 1 and 0 < at_one[0] < 2.0 ** -150
    for got, ref in ((g_c, c_ref), (g_s, s_ref)):
        assert np.all(got[ref == 0] == 0)
    for name, got, ref in (("rho", g_rho, r_ref), ("cos", g_c, c_ref), ("sin", g_s, s_ref)):
        nz = ref != 0
        rel = np.abs(got[nz] - ref[nz]) / np.abs(ref[nz])
        assert rel.max() < 2.0 ** -45, (name, np.log2(rel.max()))


@pytest.mark.parametrize("seed,j0,n", [
    (1, 0, (1 << 20) + 3),
    (2**33 + 5, 3, 100001),
    (2**64 - 1, (1 << 34) - 6, 4099),         # block index crosses 2^32
    (7, 1, 1),
])
def test_normals_within_two_ulp(orc, T, seed, j0, n):
    out = T.empty(n, dtype=T.float32, device="cuda")
    cp.cpes_debug_normals(seed, j0, n, out)
    got = to_host(out)
    ref = orc.normals(seed, j0, n)
    assert normals_within_2ulp(got, ref)
    assert np.mean(got == ref) > 0.999


def test_gpu_normal_statistics(T):
    n = 1 << 26
    out = T.empty(n, dtype=T.float32, device="cuda")
    cp.cpes_debug_normals(11, 0, n, out)
    z = out.double()
    se = 1.0 / np.sqrt(n)
    assert abs(z.mean().item()) < 5 * se
    assert abs(z.var(unbiased=False).item() - 1.0) < 5 * np.sqrt(2.0) * se
    assert abs(((z - z.mean()) ** 3).mean().item()) < 5 * np.sqrt(15.0) * se
    assert abs(((z - z.mean()) ** 4).mean().item() - 3.0) < 5 * np.sqrt(96.0) * se
    # Kolmogorov-Smirnov against the standard normal CDF over all 2^26 values:
    # the statistic stays below the 0.1 % critical value 1.95 / sqrt(n)
    zs = T.sort(out).values.double()
    cdf = T.special.ndtr(zs)
    upper = T.arange(1, n + 1, dtype=T.float64, device="cuda") / n
    ks = max((upper - cdf).max().item(), (cdf - (upper - 1.0 / n)).max().item())
    assert ks < 1.95 / np.sqrt(n), ks


@pytest.mark.parametrize("dtype", [S.BF16, S.F32])
@pytest.mark.parametrize("n,shift,seed,domain", [(1, 0, 3, 1), (7, 3, 4, 1), (4095, 1, 5, 0), ((1 << 20) + 5, 3, 6, 7)])
def test_fill_normal_matches_oracle(orc, T, dtype, n, shift, seed, domain):
    """Seeded fill against the oracle's, at an aligned or unaligned start."""
    tdt = T.bfloat16 if dtype == S.BF16 else T.float32
    buf = T.zeros(n + shift, dtype=tdt, device="cuda")
    w = buf[shift:]
    cp.cpes_fill_normal(w, seed, domain, 0.02)
    _sync(T)
    got = to_host(w)
    ref = orc.fill_normal(n, dtype, seed, domain, 0.02)
    if dtype == S.BF16:
        assert ulp_bf16(got, ref).max() <= 1
    else:
        assert ulp_f32(got, ref).max() <= 3
    assert not to_host(buf[:shift]).any()                       # nothing written before the start


# ------------------------------------------------------------ perturb etc --

LAYOUTS = ["aligned", "unaligned", "gather", "gather_v", "gather32", "chunked", "chunked_wave",
           "dense", "dense_v", "dense32", "dense_mixed"]
DENSE = ("dense", "dense_v", "dense32", "dense_mixed")   # maps flagged strictly ascending (CPES_SUB_ASCENDING)
CHUNK = 64              # chunks shorter than a wave's 64 units: per-lane chunk ids
CHUNK_WAVE = 1024       # a wave's units share a chunk (64 x 8 bf16 or 64 x 4 fp32 positions): one scalar id
LENGTHS = [1, 7, 9, 4095, (1 << 20) + 5]


@functools.lru_cache(maxsize=None)
def _perm_partition(d):
    import oracle as O

    return O.partition(O.PART_PERMUTATION, d, 4, seed=33)


@functools.lru_cache(maxsize=None)
def _chunk_partition(d, chunk=CHUNK):
    import oracle as O

    return O.partition_chunks(d, chunk, 4, 33)


def _layout(layout, length):
    """(numel, offset, host index map or None) for a subspace of `length`:
    a contiguous range at an aligned or unaligned offset, or a subspace of a
    4-way permutation partition of 4 * length indices: subspace 1 ("gather",
    its map starts at an odd entry, so units take the element path) or
    subspace 0 ("gather_v", "gather32": 16-byte map vectors; gather32 passes
    the map as uint32).  The "dense" layouts are the same maps flagged
    ascending ("dense_v" at the 16-byte aligned subspace 0), and "dense_mixed"
    one whose density alternates."""
    if layout == "aligned":
        return length + 64, 16, None
    if layout == "unaligned":
        return length + 64, 3, None
    if layout == "dense_mixed":
        index = _mixed_map(length)
        return int(index[-1]) + 70, 0, index
    d = max(4 * length, 8)
    offsets, index = _perm_partition(d)
    k = 1 if layout in ("gather", "dense") else 0
    assert offsets[k + 1] - offsets[k] >= length
    return d, int(offsets[k]), index


@functools.lru_cache(maxsize=None)
def _mixed_map(length):
    """A strictly ascending map whose density changes every 300 entries:
    gaps of 1-3 parameters, then gaps of 20-40.  Tiles of 256 entries then
    alternate between windows that fit the dense path and windows too sparse
    for it, and lines are shared between the two kinds of tile."""
    rng = np.random.default_rng(length)
    blocks = np.arange(length) // 300
    gaps = np.where(blocks % 2 == 0, rng.integers(1, 4, length), rng.integers(20, 41, length))
    return np.cumsum(gaps).astype(np.int64) + 5


def _setup(orc, T, dtype, layout, length, wseed):
    """Host weights, device weights, host (offset, element map) for the oracle,
    and the device subspace.  A chunked subspace is subspace 1 of a 4-way
    chunk partition (chunks of 64, or of 1,024 so that a wave shares one chunk
    id): the device gets its chunk list, the oracle the element map the chunk
    list expands to."""
    if layout in ("chunked", "chunked_wave"):
        C = CHUNK if layout == "chunked" else CHUNK_WAVE
        d = 4 * (length + 2 * C)
        offs, lens, chunks = _chunk_partition(d, C)
        assert lens[1] >= length
        w = S.host_weights(d, dtype, wseed)
        index = orc.expand_chunks(chunks, int(offs[1]), length, C)
        sub = cp.subspace(int(offs[1]), length, to_dev(chunks), C)
        return w, to_dev(w), 0, index, sub
    numel, offset, index = _layout(layout, length)
    w = S.host_weights(numel, dtype, wseed)
    if layout in ("gather32", "dense32"):
        dev_map = to_dev(index.astype(np.uint32).view(np.int32))
    else:
        dev_map = to_dev(index) if index is not None else None
    return w, to_dev(w), offset, index, cp.subspace(offset, length, dev_map, ascending=layout in DENSE)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("length", LENGTHS)
@pytest.mark.parametrize("dtype,aux", [(S.BF16, 0), (S.BF16, 1), (S.BF16, 2), (S.BF16, 3), (S.F32, 0), (S.F32, 1),
                                       (S.F32, 3)])
def test_perturb_matches_oracle(orc, T, dtype, aux, layout, length):
    w, dw, off, index, s = _setup(orc, T, dtype, layout, length, 1000 + length)
    sigma, seed, sign = np.float32(2.8284e-3), 17 + length, (-1 if length % 2 else 1)
    w0 = w.copy()
    snap_h = snap_d = master_h = master_d = None
    if aux == 1:
        snap_h = np.zeros(length, dtype=w.dtype)
        snap_d = to_dev(snap_h)
    if aux == 2:
        master_h = S.host_weights(length, S.F32, 7 + length)
        master_d = to_dev(master_h)
    if aux == 3:                                                      # an existing backup (other values)
        master_h = S.host_weights(length, dtype, 9 + length)
        master_d = to_dev(master_h)
    cp.cpes_perturb(dw, s, float(sigma), seed, sign, aux=snap_d if aux == 1 else master_d, aux_mode=aux)
    orc.perturb(w, off, length, sigma, seed, sign, index=index, aux=snap_h if aux == 1 else master_h, aux_mode=aux)
    _sync(T)
    got = to_host(dw)
    touched = np.zeros(w.size, dtype=bool)
    pos = index[off:off + length] if index is not None else np.arange(off, off + length)
    touched[pos] = True
    assert np.unique(pos).size == length
    assert np.array_equal(got[~touched], w0[~touched])              # outside: bitwise untouched
    if dtype == S.BF16:
        assert ulp_bf16(got[touched], w[touched]).max() <= 1
    else:
        assert f32_close(got[touched], w[touched])
        assert ulp_f32(got[touched], w[touched]).max() <= 1
    if aux == 1:
        assert np.array_equal(to_host(snap_d), snap_h)              # the backup is exact


@pytest.mark.parametrize("layout", DENSE)
@pytest.mark.parametrize("aux", [1, 2, 3])
@pytest.mark.parametrize("length", [4095, 70001])
def test_perturb_side_buffer_at_odd_offset(orc, T, aux, layout, length):
    """A snapshot, master or backup that starts one element past an aligned
    address (a view into a larger buffer): the side buffer moves element by
    element and the results are those of the oracle."""
    w, dw, off, index, s = _setup(orc, T, S.BF16, layout, length, 2000 + length)
    sigma, seed = np.float32(2.8284e-3), 23 + length
    w0 = w.copy()
    if aux == 1:
        side_h = np.zeros(length, dtype=w.dtype)
    else:
        side_h = S.host_weights(length, S.F32 if aux == 2 else S.BF16, 11 + length)
    big = to_dev(np.concatenate([side_h[:1], side_h]))
    side_d = big[1:]
    assert side_d.data_ptr() % 8 != 0
    cp.cpes_perturb(dw, s, float(sigma), seed, 1, aux=side_d, aux_mode=aux)
    orc.perturb(w, off, length, sigma, seed, 1, index=index, aux=side_h, aux_mode=aux)
    _sync(T)
    got = to_host(dw)
    touched = np.zeros(w.size, dtype=bool)
    touched[index[off:off + length]] = True
    assert np.array_equal(got[~touched], w0[~touched])
    assert ulp_bf16(got[touched], w[touched]).max() <= 1
    if aux == 1:
        assert np.array_equal(to_host(side_d), side_h)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("dtype", [S.BF16, S.F32])
def test_snapshot_and_master_restore_are_identities(orc, T, dtype, layout):
    length = (1 << 20) + 5
    w, dw, off, index, s = _setup(orc, T, dtype, layout, length, 5)
    snap = T.empty(length, dtype=dw.dtype, device="cuda")
    cp.cpes_perturb(dw, s, 4e-3, 99, 1, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    _sync(T)
    assert not np.array_equal(to_host(dw), w)
    cp.cpes_restore(dw, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
    _sync(T)
    assert np.array_equal(to_host(dw), w)
    if dtype == S.BF16:
        master = T.empty(length, dtype=T.float32, device="cuda")
        cp.cpes_stage_master(dw, s, master)
        pos = index[off:off + length] if index is not None else np.arange(off, off + length)
        _sync(T)
        assert np.array_equal(to_host(master), orc.bf16_to_f32(w[pos]))  # staging is exact
        cp.cpes_perturb(dw, s, 4e-3, 5, -1, aux=master, aux_mode=cp.AUX_MASTER)
        cp.cpes_restore(dw, s, aux=master, aux_mode=cp.AUX_MASTER)
        _sync(T)
        assert np.array_equal(to_host(dw), w)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("dtype", [S.BF16, S.F32])
def test_replay_restore_matches_oracle(orc, T, dtype, layout):
    length = 300007
    w, dw, off, index, s = _setup(orc, T, dtype, layout, length, 6)
    cp.cpes_perturb(dw, s, 2e-3, 3, -1)
    cp.cpes_restore(dw, s, 2e-3, 3, -1, aux=None, aux_mode=cp.AUX_NONE)
    orc.perturb(w, off, length, np.float32(2e-3), 3, -1, index=index)
    orc.restore(w, off, length, np.float32(2e-3), 3, -1, index=index)
    _sync(T)
    got = to_host(dw)
    if dtype == S.BF16:
        assert ulp_bf16(got, w).max() <= 1
    else:
        assert f32_close(got, w)


# ------------------------------------------------------------ device backup --

@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("length", [1, 7, 4095, (1 << 20) + 5])
@pytest.mark.parametrize("dtype", [S.BF16, S.F32])
def test_device_backup_is_the_oracle_snapshot(orc, T, dtype, layout, length):
    """cpes_backup writes the oracle's snapshot bit for bit and leaves w alone;
    restoring from it undoes a perturbation exactly."""
    w, dw, off, index, s = _setup(orc, T, dtype, layout, length, 60 + length)
    w0 = w.copy()
    b = T.full((length,), 3, dtype=dw.dtype, device="cuda")
    cp.cpes_backup(dw, s, b)
    snap = np.zeros(length, dtype=w.dtype)
    orc.perturb(w.copy(), off, length, np.float32(0.0), 1, 1, index=index, aux=snap, aux_mode=orc.AUX_SNAPSHOT)
    _sync(T)
    assert np.array_equal(to_host(b), snap)
    assert np.array_equal(to_host(dw), w0)
    cp.cpes_perturb(dw, s, 3e-3, 8, 1)
    cp.cpes_restore(dw, s, aux=b, aux_mode=cp.AUX_SNAPSHOT)
    _sync(T)
    assert np.array_equal(to_host(dw), w0)


@pytest.mark.parametrize("layout", ["aligned", "gather", "chunked"])
def test_master_loop_restores_from_a_bf16_backup(orc, T, layout):
    """With an fp32 master staged from w, a bf16 backup of w taken at the
    same time holds the master's values exactly (w is the master rounded to
    bf16, the master f32 of w).  So perturbing each member from the backup
    and restoring from it -- the schedule bench.py times for c5 -- gives the
    same bits as perturbing from and restoring from the master, member by
    member and after the update."""
    length = 200003
    w, dw, off, index, s = _setup(orc, T, S.BF16, layout, length, 91)
    dw2 = dw.clone()
    master = T.empty(length, dtype=T.float32, device="cuda")
    master2 = T.empty_like(master)
    b = T.empty(length, dtype=T.bfloat16, device="cuda")
    members = [(21, 1), (21, -1), (22, 1), (22, -1)]
    rn = to_dev(np.array([0.5, -1.0, 1.5, -1.0], np.float32))
    for it in range(2):
        cp.cpes_stage_master(dw, s, master)
        cp.cpes_stage_master(dw2, s, master2)
        cp.cpes_backup(dw2, s, b)
        for seed, sign in members:
            cp.cpes_perturb(dw, s, 2e-3, seed + it, sign, aux=master, aux_mode=cp.AUX_MASTER)
            cp.cpes_perturb(dw2, s, 2e-3, seed + it, sign, aux=b, aux_mode=cp.AUX_BACKUP)
            _sync(T)
            assert T.equal(dw.view(T.int16), dw2.view(T.int16))
            cp.cpes_restore(dw, s, aux=master, aux_mode=cp.AUX_MASTER)
            cp.cpes_restore(dw2, s, aux=b, aux_mode=cp.AUX_SNAPSHOT)
            _sync(T)
            assert T.equal(dw.view(T.int16), dw2.view(T.int16))
        seeds = [m[0] + it for m in members]
        signs = [m[1] for m in members]
        cp.cpes_update(dw, s, seeds, signs, rn, 5e-4, 2e-3, master=master)
        cp.cpes_update(dw2, s, seeds, signs, rn, 5e-4, 2e-3, master=master2)
        _sync(T)
        assert T.equal(dw.view(T.int16), dw2.view(T.int16))
        assert T.equal(master, master2)


# ------------------------------------------------------ host-memory backup --

@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("length", [1, 7, 4095, (1 << 20) + 5])
@pytest.mark.parametrize("dtype", [S.BF16, S.F32])
def test_host_backup_round_trip(orc, T, dtype, layout, length):
    """The backup written to pinned host memory is the oracle's snapshot, bit
    for bit, and restoring from it undoes a perturbation exactly."""
    w, dw, off, index, s = _setup(orc, T, dtype, layout, length, 40 + length)
    w0 = w.copy()
    hb = T.full((length,), 7, dtype=dw.dtype, pin_memory=True)
    cp.cpes_backup_to_host(dw, s, hb)
    snap = np.zeros(length, dtype=w.dtype)
    orc.perturb(w, off, length, np.float32(3e-3), 8, 1, index=index, aux=snap, aux_mode=orc.AUX_SNAPSHOT)
    cp.cpes_perturb(dw, s, 3e-3, 8, 1)
    _sync(T)
    assert np.array_equal(to_host(hb), snap)
    got = to_host(dw)
    if dtype == S.BF16:
        assert ulp_bf16(got, w).max() <= 1
    else:
        assert f32_close(got, w)
    cp.cpes_restore_from_host(dw, s, hb)
    orc.restore(w, off, length, 0.0, 0, 1, index=index, aux=snap, aux_mode=orc.AUX_SNAPSHOT)
    _sync(T)
    assert np.array_equal(w, w0)
    assert np.array_equal(to_host(dw), w0)


@pytest.mark.parametrize("layout", ["unaligned", "chunked", "dense_v"])
def test_host_backup_member_loop(orc, T, layout):
    """One host backup per step, then perturb / restore for every member: each
    member is perturbed from the same pre-update weights (the oracle perturbs
    a fresh copy of them), and the weights return to them bit for bit."""
    length = 300007
    w, dw, off, index, s = _setup(orc, T, S.BF16, layout, length, 77)
    hb = T.empty((length,), dtype=dw.dtype, pin_memory=True)
    cp.cpes_backup_to_host(dw, s, hb)
    for m, (seed, sign) in enumerate([(11, 1), (11, -1), (12, 1), (13, -1)]):
        cp.cpes_perturb(dw, s, 2e-3, seed, sign)
        _sync(T)
        ref = w.copy()
        orc.perturb(ref, off, length, np.float32(2e-3), seed, sign, index=index)
        assert ulp_bf16(to_host(dw), ref).max() <= 1, f"member {m}"
        cp.cpes_restore_from_host(dw, s, hb)
    _sync(T)
    assert np.array_equal(to_host(dw), w)


def test_host_backup_rejects_unpinned_and_device_buffers(orc, T):
    w, dw, off, index, s = _setup(orc, T, S.BF16, "aligned", 4096, 3)
    pageable = T.empty((4096,), dtype=dw.dtype)
    assert not pageable.is_pinned()
    with pytest.raises(cp.CpesError, match="not pinned host memory"):
        cp.cpes_backup_to_host(dw, s, pageable)
    with pytest.raises(cp.CpesError, match="not pinned host memory"):
        cp.cpes_restore_from_host(dw, s, pageable)
    dev = T.empty((4096,), dtype=dw.dtype, device="cuda")
    rc = cp.load().cpes_restore_from_host(dw.data_ptr(), dw.numel(), cp.BF16, cp.ctypes.byref(s), dev.data_ptr(),
                                          None)
    assert rc == cp.ERR_INVALID_ARGUMENT and "not pinned" in cp.last_error()
    with pytest.raises(ValueError):
        cp.cpes_backup_to_host(dw, s, dev)
    _sync(T)
    assert np.array_equal(to_host(dw), w)                           # nothing was written


# --------------------------------------------------------------- normalise --

@pytest.mark.parametrize("n", [1, 2, 8, 30, 32, 40, 128, 1000, 4096])
@pytest.mark.parametrize("mode", [S.NORM_Z, S.NORM_RANK])
@pytest.mark.parametrize("kind", ["uniform", "bernoulli", "mean_bernoulli"])
def test_normalize_matches_oracle(orc, T, n, mode, kind):
    r = S.rewards(kind, n, 99 + n)
    out = T.empty(n, dtype=T.float32, device="cuda")
    st = T.full((1,), -7, dtype=T.int32, device="cuda")
    cp.cpes_normalize_rewards(to_dev(r), out, mode, status=st)
    ref, rst = orc.normalize(r, mode)
    _sync(T)
    assert int(st.item()) == rst == 0
    _normalized_match(to_host(out), ref, r, mode)


def _normalized_match(got, ref, r, mode, group=None):
    """Ranks bit-exact; z-scores within the bound of zscore_close (and, over
    many rewards, nearly all bit-identical)."""
    if mode == S.NORM_RANK:
        assert np.array_equal(got, ref)
        return
    assert zscore_close(got, ref, r, group), describe_mismatch(got, ref)
    if len(r) >= 1000:
        assert np.mean(got == ref) > 0.99


@pytest.mark.parametrize("mode", [S.NORM_Z, S.NORM_RANK])
def test_normalize_grouped_and_failures(orc, T, mode):
    n, K = 40, 4
    r = S.rewards("uniform", n, 12)
    g = np.repeat(np.arange(K), n // K).astype(np.int32)[np.random.default_rng(2).permutation(n)]
    out = T.empty(n, dtype=T.float32, device="cuda")
    st = T.zeros(1, dtype=T.int32, device="cuda")
    cp.cpes_normalize_rewards(to_dev(r), out, mode, group=to_dev(g), n_groups=K, status=st)
    ref, _ = orc.normalize(r, mode, g)
    _sync(T)
    assert int(st.item()) == 0
    _normalized_match(to_host(out), ref, r, mode, g)
    # constant rewards -> zeros; a NaN -> zeros + status 1; a bad group id -> zeros + status 2
    cp.cpes_normalize_rewards(to_dev(np.full(n, 0.5, np.float32)), out, mode, status=st)
    _sync(T)
    assert np.all(to_host(out) == 0) and int(st.item()) == 0
    rr = r.copy()
    rr[7] = np.nan
    cp.cpes_normalize_rewards(to_dev(rr), out, mode, status=st)
    _sync(T)
    assert np.all(to_host(out) == 0) and int(st.item()) == 1
    gg = g.copy()
    gg[3] = K
    cp.cpes_normalize_rewards(to_dev(r), out, mode, group=to_dev(gg), n_groups=K, status=st)
    _sync(T)
    assert np.all(to_host(out) == 0) and int(st.item()) == 2


def test_normalize_at_the_limits(orc, T):
    """4096 rewards (CPES_MAX_REWARDS) in 1024 groups (CPES_MAX_GROUPS) of 4."""
    n, K = 4096, 1024
    for mode in (S.NORM_Z, S.NORM_RANK):
        r = S.rewards("mean_bernoulli", n, 31)
        g = (np.arange(n) % K).astype(np.int32)
        out = T.empty(n, dtype=T.float32, device="cuda")
        cp.cpes_normalize_rewards(to_dev(r), out, mode, group=to_dev(g), n_groups=K)
        ref, st = orc.normalize(r, mode, g)
        _sync(T)
        assert st == 0
        _normalized_match(to_host(out), ref, r, mode, g)


# ------------------------------------------------------------------ update --

MEMBER_SETS = {
    "one": ([5], [1]),
    "pairs4": ([9, 9, 12, 40], [1, -1, 1, 1]),
    "n30": (list(range(1, 31)), [1] * 30),
    "n128_antithetic": ([s for s in range(1001, 1065) for _ in (0, 1)], [1, -1] * 64),
    "n256_max": (list(range(2001, 2257)), [1, -1] * 128),             # CPES_MAX_MEMBERS distinct streams
}


@pytest.mark.parametrize("members", list(MEMBER_SETS))
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("kind", ["bf16", "f32", "master"])
def test_update_matches_oracle(orc, T, kind, layout, members):
    seeds, signs = MEMBER_SETS[members]
    n = len(seeds)
    length = (1 << 18) + 5 if n > 30 else (1 << 20) + 3
    dtype = S.F32 if kind == "f32" else S.BF16
    w, dw, off, index, s = _setup(orc, T, dtype, layout, length, 20 + n)
    r = S.rewards("uniform", n, 7 + n)
    rnorm, _ = orc.normalize(r, S.NORM_Z)
    scale = S.SCALE_ALPHA_OVER_N if members == "pairs4" else S.SCALE_ALPHA_OVER_N_SIGMA
    alpha, sigma = np.float32(5e-4), np.float32(2.25e-3)
    master_h = master_d = None
    if kind == "master":
        pos = index[off:off + length] if index is not None else np.arange(off, off + length)
        master_h = orc.bf16_to_f32(w[pos]).copy()
        master_d = to_dev(master_h)
    w0 = w.copy()
    cp.cpes_update(dw, s, seeds, signs, to_dev(rnorm), float(alpha), float(sigma), scale, master=master_d)
    orc.update(w, off, length, seeds, signs, rnorm, alpha, sigma, scale, index=index, master=master_h)
    _sync(T)
    got = to_host(dw)
    changed = np.zeros(w.size, dtype=bool)
    pos = index[off:off + length] if index is not None else np.arange(off, off + length)
    changed[pos] = True
    assert np.array_equal(got[~changed], w0[~changed])
    if dtype == S.BF16:
        step = update_step_size(alpha, sigma, n, scale)
        inv = np.full(w.size, -1, dtype=np.int64)
        inv[pos] = np.arange(length)
        slack = lambda k: update_slack(orc, seeds, signs, rnorm, step, inv[k])
        assert bf16_update_close(got, w, slack), describe_mismatch(bf16_value(got), bf16_value(w))
        assert np.mean(ulp_bf16(got, w) <= 1) > 0.9999
    else:
        assert f32_close(got, w), describe_mismatch(got, w)
    if kind == "master":
        assert f32_close(to_host(master_d), master_h), describe_mismatch(to_host(master_d), master_h)


def test_update_mirrored_equal_rewards_is_identity(T):
    w = S.host_weights(100003, S.BF16, 3)
    dw = to_dev(w)
    rn = to_dev(np.array([0.7, 0.7, -1.1, -1.1], np.float32))
    cp.cpes_update(dw, cp.subspace(0, 100003), [4, 4, 8, 8], [1, -1, 1, -1], rn, 5e-4, 4e-3)
    _sync(T)
    assert np.array_equal(to_host(dw), w)


@pytest.mark.parametrize("dtype", [S.BF16, S.F32])
def test_degenerate_calls_leave_weights_untouched(T, dtype):
    """sigma = 0 perturbs to the same bits (one fp32 FMA with a zero product,
    then the exact bf16 rounding of an exact value), an empty subspace and a
    zero step do nothing, and neither do mirrored pairs with equal rewards
    (each stream's folded coefficient is exactly zero)."""
    w = S.host_weights(70001, dtype, 12)
    dw = to_dev(w)
    s = cp.subspace(1, 70000)
    cp.cpes_perturb(dw, s, 0.0, 3, 1)
    cp.cpes_perturb(dw, cp.subspace(9, 0), 1e-2, 3, 1)
    cp.cpes_update(dw, s, [1, 2], [1, 1], to_dev(np.array([0.3, -0.3], np.float32)), 0.0, 1e-3)
    cp.cpes_update(dw, s, [5, 5, 6, 6], [1, -1, 1, -1], to_dev(np.array([0.7, 0.7, -0.2, -0.2], np.float32)),
                   5e-4, 1e-3)
    cp.cpes_restore(dw, cp.subspace(70001, 0), aux=None, aux_mode=cp.AUX_NONE, sigma=1e-3)
    _sync(T)
    assert np.array_equal(to_host(dw), w)


# --------------------------------------------------------------- partition --

@pytest.mark.parametrize("d,K", [(1, 1), (2, 2), (7, 3), (1000, 8), (4096, 4), (100003, 8), ((1 << 20) + 3, 256),
                                 ((1 << 21) + 1, 16)])
def test_permutation_partition_bit_exact(orc, T, d, K):
    ws = T.empty(cp.cpes_partition_workspace_bytes(cp.PART_PERMUTATION, d, K), dtype=T.uint8, device="cuda")
    index = T.full((d,), -1, dtype=T.int64, device="cuda")
    st = T.full((1,), -7, dtype=T.int32, device="cuda")
    offsets = cp.cpes_partition(cp.PART_PERMUTATION, d, K, seed=33, index=index, workspace=ws, status=st)
    ref_off, ref_index = orc.partition(orc.PART_PERMUTATION, d, K, seed=33)
    _sync(T)
    assert offsets == [int(x) for x in ref_off]
    assert int(st.item()) == 0
    assert np.array_equal(to_host(index), ref_index)


@pytest.mark.parametrize("d,K", [(1, 1), (7, 3), (100003, 8), ((1 << 20) + 3, 256)])
def test_permutation_partition32_bit_exact(orc, T, d, K):
    ws = T.empty(cp.cpes_partition_workspace_bytes(cp.PART_PERMUTATION, d, K), dtype=T.uint8, device="cuda")
    index = T.full((d,), -1, dtype=T.int32, device="cuda")
    offsets = cp.cpes_partition32(d, K, 33, index, ws)
    ref_off, ref_index = orc.partition(orc.PART_PERMUTATION, d, K, seed=33)
    _sync(T)
    assert offsets == [int(x) for x in ref_off]
    assert np.array_equal(to_host(index).view(np.uint32).astype(np.int64), ref_index)


def test_prp_values_bit_exact(orc, T):
    for d, K in ((4022468096, 8), (1 << 20, 4), (12345, 7)):
        i0 = max(0, d - 5000)
        n = min(d, 5000)
        perm = T.empty(n, dtype=T.int64, device="cuda")
        bucket = T.empty(n, dtype=T.int32, device="cuda")
        cp.cpes_debug_prp(33, d, K, i0, n, perm, bucket)
        _sync(T)
        p, b = to_host(perm), to_host(bucket)
        for k in range(0, n, 37):
            assert p[k] == orc.prp(33, d, i0 + k)
            assert b[k] == orc.bucket(33, d, K, i0 + k)


# ------------------------------------------------------------ step update --

STEP_CASES = {
    # name: (d, K, partition, members per subspace)
    "paper_perm_k4_n40": ((1 << 20) + 3, 4, "perm", [10, 10, 10, 10]),
    "paper_chunk_k4_n40": ((1 << 20) + 3, 4, "chunk", [10, 10, 10, 10]),
    "paper_perm32_k4_n40": ((1 << 20) + 3, 4, "perm32", [10, 10, 10, 10]),  # uint32 map: cpes_update_step32
    "contig_unaligned": (300007, 3, [0, 1001, 150003, 300007], [5, 3, 4]),
    "contig_k1_std_es": (262147, 1, "equal", [8]),
    "contig_k8_empty": ((1 << 19) + 64, 8, "equal", [2, 0, 3, 1, 1, 0, 2, 2]),
    "contig_k32_n256_max": ((1 << 20) + 7, 32, "equal", [8] * 32),       # CPES_MAX_STEP_SUBSPACES, CPES_MAX_MEMBERS
    "chunk1024_k4": ((1 << 20) + 3, 4, "chunk1024", [6, 7, 8, 9]),      # a wave shares one chunk id
}


@pytest.mark.parametrize("case", list(STEP_CASES))
@pytest.mark.parametrize("dtype", [S.BF16, S.F32])
@pytest.mark.parametrize("scale", [S.SCALE_ALPHA_OVER_N, S.SCALE_ALPHA_OVER_N_SIGMA])
def test_update_step_matches_oracle(orc, T, case, dtype, scale):
    d, K, part, per = STEP_CASES[case]
    index = dindex = lengths = None
    chunk = 0
    if part in ("chunk", "chunk1024"):
        chunk = 256 if part == "chunk" else 1024
        offsets, lengths, chunks = orc.partition_chunks(d, chunk, K, 33)
        dindex = to_dev(chunks)
        # the oracle sees each chunked subspace through its element map, laid end to end
        maps = [orc.expand_chunks(chunks, int(offsets[k]), int(lengths[k]), chunk) for k in range(K)]
        index = np.concatenate(maps)
        host_offsets = np.concatenate([[0], np.cumsum(lengths)])
    elif part in ("perm", "perm32"):
        offsets, index = orc.partition(orc.PART_PERMUTATION, d, K, seed=33)
        dindex = to_dev(index if part == "perm" else index.astype(np.uint32).view(np.int32))
    elif part == "equal":
        offsets, _ = orc.partition(orc.PART_CONTIGUOUS, d, K)
    else:
        offsets = np.array(part, dtype=np.int64)
    offsets = [int(x) for x in offsets]
    if part not in ("chunk", "chunk1024"):
        host_offsets = offsets
    subs = [k for k in range(K) for _ in range(per[k])]
    n = len(subs)
    seeds = [1 + i for i in range(n)]
    signs = [1 if i % 3 else -1 for i in range(n)]
    rhat, _ = orc.normalize(S.rewards("uniform", n, 99), S.NORM_Z)        # joint standardisation (Eq. 12)
    sigmas = [float(np.float32(1e-3 * np.sqrt(d / max(1, host_offsets[k + 1] - host_offsets[k])))) for k in range(K)]
    w = S.host_weights(d, dtype, 70)
    dw = to_dev(w)
    cp.cpes_update_step(dw, offsets, seeds, signs, subs, to_dev(rhat), 5e-4, sigmas, scale, index=dindex, chunk=chunk,
                        lengths=lengths)
    orc.update_step(w, host_offsets, seeds, signs, subs, rhat, np.float32(5e-4), np.float32(sigmas), scale,
                    index=index)
    _sync(T)
    got = to_host(dw)
    if dtype == S.BF16:
        slack = _step_slack(orc, d, host_offsets, index, seeds, signs, subs, rhat, 5e-4, sigmas, scale)
        assert bf16_update_close(got, w, slack), describe_mismatch(bf16_value(got), bf16_value(w))
    else:
        assert f32_close(got, w), describe_mismatch(got, w)


def _step_slack(orc, d, offsets, index, seeds, signs, subs, rnorm, alpha, sigmas, scale):
    """update_slack for a whole-step update: parameter i of subspace k at noise
    position j gets the bound of k's members and step."""
    K = len(offsets) - 1
    sub_of = np.full(d, -1, dtype=np.int64)
    pos_of = np.full(d, -1, dtype=np.int64)
    for k in range(K):
        a, b = int(offsets[k]), int(offsets[k + 1])
        params = index[a:b] if index is not None else np.arange(a, b)
        sub_of[params] = k
        pos_of[params] = np.arange(b - a)

    def slack(ix):
        out = np.zeros(len(ix))
        for k in range(K):
            sel = np.nonzero(sub_of[ix] == k)[0]
            mem = [i for i in range(len(subs)) if subs[i] == k]
            if sel.size == 0 or not mem:
                continue
            step = update_step_size(alpha, sigmas[k], len(mem), scale)
            out[sel] = update_slack(orc, [seeds[i] for i in mem], [signs[i] for i in mem],
                                    [rnorm[i] for i in mem], step, pos_of[ix[sel]])
        return out
    return slack


def test_update_step_with_grouped_standardisation(orc, T):
    """The independent z-score ablation: each subspace standardised on its own."""
    d, K, Nk = (1 << 18) + 5, 4, 6
    offsets, index = orc.partition(orc.PART_PERMUTATION, d, K, seed=7)
    subs = np.repeat(np.arange(K), Nk).astype(np.int32)
    n = K * Nk
    r = S.rewards("uniform", n, 5)
    rn = T.empty(n, dtype=T.float32, device="cuda")
    cp.cpes_normalize_rewards(to_dev(r), rn, cp.NORM_Z, group=to_dev(subs), n_groups=K)
    rhat, _ = orc.normalize(r, S.NORM_Z, subs)
    w = S.host_weights(d, S.BF16, 71)
    dw = to_dev(w)
    sig = [2e-3] * K
    cp.cpes_update_step(dw, [int(x) for x in offsets], list(range(1, n + 1)), [1] * n, subs.tolist(), rn, 5e-4, sig,
                        S.SCALE_ALPHA_OVER_N, index=to_dev(index))
    orc.update_step(w, offsets, list(range(1, n + 1)), [1] * n, subs, rhat, np.float32(5e-4), np.float32(sig),
                    S.SCALE_ALPHA_OVER_N, index=index)
    _sync(T)
    assert zscore_close(to_host(rn), rhat, r, subs)
    slack = _step_slack(orc, d, offsets, index, list(range(1, n + 1)), [1] * n, subs.tolist(), rhat, 5e-4, sig,
                        S.SCALE_ALPHA_OVER_N)
    assert bf16_update_close(to_host(dw), w, slack)


@pytest.mark.parametrize("d,chunk,K", [(1000, 8, 3), ((1 << 20) + 5, 64, 8), (10000003, 4096, 16), (65536, 65536, 1)])
def test_chunk_partition_bit_exact(orc, T, d, chunk, K):
    n_chunks = -(-d // chunk)
    ws = T.empty(cp.cpes_partition_chunks_workspace_bytes(d, chunk, K), dtype=T.uint8, device="cuda")
    chunks = T.full((n_chunks,), -1, dtype=T.int64, device="cuda")
    st = T.full((1,), -7, dtype=T.int32, device="cuda")
    offs, lens = cp.cpes_partition_chunks(d, chunk, K, 33, chunks, ws, status=st)
    r_offs, r_lens, r_chunks = orc.partition_chunks(d, chunk, K, 33)
    _sync(T)
    assert int(st.item()) == 0
    assert offs == [int(x) for x in r_offs] and lens == [int(x) for x in r_lens]
    assert np.array_equal(to_host(chunks), r_chunks)
