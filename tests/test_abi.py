"""The C-ABI library loads without a GPU, exports every symbol include/cpes.h
declares, and rejects bad arguments on the host (status code + message, before
any HIP call).  No compute is launched here."""
import ctypes
import os
import re

import pytest

import paper_2608_02391_amd as cp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cpes.h")

FAKE = 0x10000  # a non-null, 16-byte aligned address that is never dereferenced on these paths


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(cp.LIB_PATH):
        pytest.fail("libcpes.so is not built (run __graft_entry__.build())")
    return cp.load()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^CPES_API\s+[\w\s\*]+?\b(cpes_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("cpes_partition", "cpes_perturb", "cpes_restore", "cpes_normalize_rewards", "cpes_update"):
        assert required in names
    assert sorted(cp.EXPORTED) == names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), name
    assert lib.cpes_abi_version() == 8


def _sub(offset=0, length=16, index=None, chunk=0, index32=None, noise_offset=0, flags=0):
    return cp.Subspace(offset, length, index, chunk, index32, noise_offset, flags)


def _rc_msg(lib, rc):
    return rc, lib.cpes_last_error().decode()


def test_perturb_rejects_bad_arguments(lib):
    s = _sub()
    cases = [
        (None, 64, cp.BF16, ctypes.byref(s), 1e-3, 1, 1, None, cp.AUX_NONE),        # null weights
        (FAKE, 64, 7, ctypes.byref(s), 1e-3, 1, 1, None, cp.AUX_NONE),              # bad dtype
        (FAKE, 64, cp.BF16, None, 1e-3, 1, 1, None, cp.AUX_NONE),                   # null subspace
        (FAKE, 64, cp.BF16, ctypes.byref(s), 1e-3, 1, 0, None, cp.AUX_NONE),        # sign 0
        (FAKE, 64, cp.BF16, ctypes.byref(s), -1e-3, 1, 1, None, cp.AUX_NONE),       # sigma < 0
        (FAKE, 64, cp.BF16, ctypes.byref(s), float("nan"), 1, 1, None, cp.AUX_NONE),
        (FAKE, 64, cp.BF16, ctypes.byref(s), 1e-3, 1, 1, None, cp.AUX_SNAPSHOT),    # snapshot missing
        (FAKE, 64, cp.BF16, ctypes.byref(s), 1e-3, 1, 1, FAKE, 9),                  # bad aux mode
        (FAKE, 64, cp.F32, ctypes.byref(s), 1e-3, 1, 1, FAKE, cp.AUX_MASTER),       # master on fp32
        (FAKE, 8, cp.BF16, ctypes.byref(s), 1e-3, 1, 1, None, cp.AUX_NONE),         # beyond numel
        (FAKE, 64, cp.BF16, ctypes.byref(_sub(0, -1)), 1e-3, 1, 1, None, cp.AUX_NONE),
        (FAKE, 64, cp.BF16, ctypes.byref(_sub(-4, 4)), 1e-3, 1, 1, None, cp.AUX_NONE),
        (FAKE, 64, cp.BF16, ctypes.byref(_sub(0, 16, noise_offset=-8)), 1e-3, 1, 1, None, cp.AUX_NONE),
        (FAKE, 64, cp.BF16, ctypes.byref(_sub(0, 16, noise_offset=12)), 1e-3, 1, 1, None, cp.AUX_NONE),  # not 8k
    ]
    for args in cases:
        rc, msg = _rc_msg(lib, lib.cpes_perturb(*args, None))
        assert rc == cp.ERR_INVALID_ARGUMENT, args
        assert msg.startswith("cpes_perturb:"), msg


def test_empty_subspace_is_a_no_op(lib):
    s = _sub(3, 0)
    assert lib.cpes_perturb(FAKE, 64, cp.BF16, ctypes.byref(s), 1e-3, 1, 1, None, cp.AUX_NONE, None) == cp.OK
    assert lib.cpes_restore(FAKE, 64, cp.BF16, ctypes.byref(s), 0.0, 0, 1, FAKE, cp.AUX_SNAPSHOT, None) == cp.OK
    assert lib.cpes_last_error() == b""


def test_restore_and_stage_reject_bad_arguments(lib):
    s = _sub()
    assert lib.cpes_restore(FAKE, 64, cp.BF16, ctypes.byref(s), 0.0, 0, 1, None, cp.AUX_SNAPSHOT, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_restore(FAKE, 64, cp.BF16, ctypes.byref(s), 1e-3, 0, 2, None, cp.AUX_NONE, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_restore(FAKE, 64, cp.F32, ctypes.byref(s), 0.0, 0, 1, FAKE, cp.AUX_MASTER, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_stage_master(FAKE, 64, cp.BF16, ctypes.byref(s), None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_stage_master(FAKE, 10, cp.BF16, ctypes.byref(s), FAKE, None) == cp.ERR_INVALID_ARGUMENT


def test_host_backup_rejects_bad_arguments(lib):
    s = _sub()
    for fn in (lib.cpes_backup, lib.cpes_backup_to_host, lib.cpes_restore_from_host):
        name = fn.__name__
        for args in [(None, 64, cp.BF16, ctypes.byref(s), FAKE),       # null weights
                     (FAKE, 64, 7, ctypes.byref(s), FAKE),             # bad dtype
                     (FAKE, 64, cp.BF16, None, FAKE),                  # null subspace
                     (FAKE, 8, cp.BF16, ctypes.byref(s), FAKE),        # beyond numel
                     (FAKE, 64, cp.BF16, ctypes.byref(s), None)]:      # null backup
            rc, msg = _rc_msg(lib, fn(*args, None))
            assert rc == cp.ERR_INVALID_ARGUMENT, (name, args)
            assert msg.startswith(name + ":"), msg
        assert fn(FAKE, 64, cp.BF16, ctypes.byref(_sub(3, 0)), FAKE, None) == cp.OK   # empty: no-op


def test_fill_normal_rejects_bad_arguments(lib):
    for args in [(FAKE, 16, 7, 1, 1, 0.02),               # bad dtype
                 (FAKE, -1, cp.BF16, 1, 1, 0.02),         # negative n
                 (FAKE, 16, cp.BF16, 1, 1, -0.02),        # negative stddev
                 (FAKE, 16, cp.F32, 1, 1, float("inf")),
                 (None, 16, cp.F32, 1, 1, 0.02)]:         # null weights
        rc, msg = _rc_msg(lib, lib.cpes_fill_normal(*args, None))
        assert rc == cp.ERR_INVALID_ARGUMENT, args
        assert msg.startswith("cpes_fill_normal:"), msg
    assert lib.cpes_fill_normal(None, 0, cp.BF16, 1, 1, 0.02, None) == cp.OK


def test_uint32_maps_are_validated(lib):
    both = _sub(0, 16, FAKE, 0, FAKE)                                   # int64 and uint32 map
    chunked32 = _sub(0, 16, None, 64, FAKE)                             # chunk lists are int64
    for s in (both, chunked32):
        rc, msg = _rc_msg(lib, lib.cpes_perturb(FAKE, 64, cp.BF16, ctypes.byref(s), 1e-3, 1, 1, None,
                                                cp.AUX_NONE, None))
        assert rc == cp.ERR_INVALID_ARGUMENT and msg.startswith("cpes_perturb:"), msg
    offs = (ctypes.c_int64 * 9)()
    assert lib.cpes_partition32((1 << 32) + 1, 8, 1, offs, FAKE, FAKE, 1 << 40, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition32(1000, 0, 1, offs, FAKE, FAKE, 1 << 20, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition32(1000, 8, 1, offs, None, FAKE, 1 << 20, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition32(1000, 8, 1, offs, FAKE, FAKE, 16, None, None) == cp.ERR_WORKSPACE
    assert lib.cpes_partition32(1000, 300, 1, offs, FAKE, FAKE, 1 << 20, None, None) == cp.ERR_UNSUPPORTED


def test_normalize_rejects_bad_arguments(lib):
    assert lib.cpes_normalize_rewards(None, 8, cp.NORM_Z, None, 1, FAKE, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_normalize_rewards(FAKE, 0, cp.NORM_Z, None, 1, FAKE, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_normalize_rewards(FAKE, 4097, cp.NORM_Z, None, 1, FAKE, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_normalize_rewards(FAKE, 8, 5, None, 1, FAKE, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_normalize_rewards(FAKE, 8, cp.NORM_Z, FAKE, 9, FAKE, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_normalize_rewards(FAKE, 2000, cp.NORM_Z, FAKE, 1500, FAKE, None, None) == cp.ERR_UNSUPPORTED


def test_update_rejects_bad_arguments(lib):
    s = _sub()
    seeds = (ctypes.c_uint64 * 4)(1, 2, 3, 4)
    signs = (ctypes.c_int8 * 4)(1, 1, -1, 1)
    bad_signs = (ctypes.c_int8 * 4)(1, 0, -1, 1)
    many = (ctypes.c_uint64 * 300)()
    many_s = (ctypes.c_int8 * 300)(*([1] * 300))
    args = lambda **kw: [kw.get("w", FAKE), 64, kw.get("dtype", cp.BF16), ctypes.byref(s), kw.get("master", None),
                         kw.get("n", 4), kw.get("seeds", seeds), kw.get("signs", signs), kw.get("r", FAKE),
                         kw.get("alpha", 5e-4), kw.get("sigma", 1e-3), kw.get("scale", 0), None]
    assert lib.cpes_update(*args(w=None)) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_update(*args(n=0)) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_update(*args(n=300, seeds=many, signs=many_s)) == cp.ERR_UNSUPPORTED
    assert lib.cpes_update(*args(signs=bad_signs)) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_update(*args(r=None)) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_update(*args(sigma=0.0)) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_update(*args(alpha=float("inf"))) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_update(*args(scale=3)) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_update(*args(dtype=cp.F32, master=FAKE)) == cp.ERR_INVALID_ARGUMENT
    assert "cpes_update" in lib.cpes_last_error().decode()


def test_partition_host_paths(lib):
    off = (ctypes.c_int64 * 4)()
    assert lib.cpes_partition(cp.PART_CONTIGUOUS, 10, 3, 0, None, off, None, None, 0, None, None) == cp.OK
    assert list(off) == [0, 3, 6, 10]
    b = (ctypes.c_int64 * 4)(0, 4, 4, 10)
    assert lib.cpes_partition(cp.PART_CONTIGUOUS, 10, 3, 0, b, off, None, None, 0, None, None) == cp.OK
    assert list(off) == [0, 4, 4, 10]
    bad = (ctypes.c_int64 * 4)(0, 5, 4, 10)
    assert lib.cpes_partition(cp.PART_CONTIGUOUS, 10, 3, 0, bad, off, None, None, 0, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition(cp.PART_CONTIGUOUS, 10, 11, 0, None, off, None, None, 0, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition(7, 10, 3, 0, None, off, None, None, 0, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition(cp.PART_PERMUTATION, 10, 300, 0, None, (ctypes.c_int64 * 301)(), FAKE, FAKE, 1 << 20,
                              None, None) == cp.ERR_INVALID_ARGUMENT  # K > d
    assert lib.cpes_partition(cp.PART_PERMUTATION, 1000, 300, 0, None, (ctypes.c_int64 * 301)(), FAKE, FAKE,
                              1 << 20, None, None) == cp.ERR_UNSUPPORTED
    need = lib.cpes_partition_workspace_bytes(cp.PART_PERMUTATION, 1000, 8)
    assert need >= 1000
    assert lib.cpes_partition(cp.PART_PERMUTATION, 1000, 8, 0, None, (ctypes.c_int64 * 9)(), FAKE, FAKE, need - 1,
                              None, None) == cp.ERR_WORKSPACE
    assert lib.cpes_partition(cp.PART_PERMUTATION, 1000, 8, 0, None, (ctypes.c_int64 * 9)(), None, FAKE, need,
                              None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition_workspace_bytes(cp.PART_CONTIGUOUS, 1000, 8) == 0
    assert lib.cpes_partition_workspace_bytes(cp.PART_PERMUTATION, 1000, 0) == 0


def test_debug_hooks_reject_bad_arguments(lib):
    assert lib.cpes_debug_philox(0, 0, 0, -1, FAKE, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_debug_normals(0, -1, 4, FAKE, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_debug_bm_grid(0, 4, None, None, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_debug_bm_grid(1 << 24, 2, None, None, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_debug_prp(0, 100, 8, 90, 20, None, None, None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_rng_probe(0, 8, None, None) == cp.ERR_INVALID_ARGUMENT


def test_binding_raises_without_fallback(tmp_path):
    """A missing library is an error, never a silent CPU path."""
    import importlib

    mod = importlib.import_module("paper_2608_02391_amd")
    saved = mod._lib
    try:
        mod._lib = None
        with pytest.raises(RuntimeError):
            mod.load(str(tmp_path / "missing.so"))
    finally:
        mod._lib = saved


def test_update_step_rejects_bad_arguments(lib):
    off = (ctypes.c_int64 * 3)(0, 32, 64)
    seeds = (ctypes.c_uint64 * 4)(1, 2, 3, 4)
    signs = (ctypes.c_int8 * 4)(1, 1, -1, 1)
    subs = (ctypes.c_int32 * 4)(0, 0, 1, 1)
    bad_subs = (ctypes.c_int32 * 4)(0, 0, 2, 1)
    sig = (ctypes.c_float * 2)(2e-3, 2e-3)
    zero_sig = (ctypes.c_float * 2)(2e-3, 0.0)
    dec = (ctypes.c_int64 * 3)(0, 40, 32)
    def call(**kw):
        return lib.cpes_update_step(kw.get("w", FAKE), kw.get("numel", 64), cp.BF16, kw.get("K", 2), kw.get("off", off),
                                    kw.get("index", None), kw.get("chunk", 0), kw.get("lens", None), 4, seeds, signs,
                                    kw.get("subs", subs), FAKE, 5e-4, kw.get("sig", sig), kw.get("scale", 0), None)
    assert call(w=None) == cp.ERR_INVALID_ARGUMENT
    assert call(K=0) == cp.ERR_INVALID_ARGUMENT
    assert call(K=40) == cp.ERR_UNSUPPORTED
    assert call(subs=bad_subs) == cp.ERR_INVALID_ARGUMENT
    assert call(sig=zero_sig) == cp.ERR_INVALID_ARGUMENT
    assert call(off=dec) == cp.ERR_INVALID_ARGUMENT
    assert call(numel=63) == cp.ERR_INVALID_ARGUMENT
    assert call(index=FAKE, chunk=64, lens=None) == cp.ERR_INVALID_ARGUMENT          # chunked needs lengths
    assert call(index=FAKE, chunk=24, lens=(ctypes.c_int64 * 2)(8, 8)) == cp.ERR_INVALID_ARGUMENT
    assert call(index=FAKE, chunk=8, lens=(ctypes.c_int64 * 2)(257, 8)) == cp.ERR_INVALID_ARGUMENT  # > 32 chunks x 8
    assert lib.cpes_last_error().decode().startswith("cpes_update_step")

    def call32(**kw):
        return lib.cpes_update_step32(kw.get("w", FAKE), kw.get("numel", 64), cp.BF16, kw.get("K", 2),
                                      kw.get("off", off), kw.get("index", FAKE), 4, seeds, signs,
                                      kw.get("subs", subs), FAKE, 5e-4, kw.get("sig", sig), 0, None)
    assert call32(index=None) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_last_error().decode().startswith("cpes_update_step32")
    assert call32(w=None) == cp.ERR_INVALID_ARGUMENT
    assert call32(K=40) == cp.ERR_UNSUPPORTED
    assert call32(subs=bad_subs) == cp.ERR_INVALID_ARGUMENT
    assert call32(off=dec) == cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_last_error().decode().startswith("cpes_update_step32")


def test_chunked_subspaces_are_validated(lib):
    for chunk, index in ((12, FAKE), (4, FAKE), (1 << 31, FAKE), (64, None)):
        s = cp.Subspace(0, 16, index, chunk)
        assert lib.cpes_perturb(FAKE, 64, cp.BF16, ctypes.byref(s), 1e-3, 1, 1, None, cp.AUX_NONE, None) == \
            cp.ERR_INVALID_ARGUMENT, chunk
    offs = (ctypes.c_int64 * 4)()
    lens = (ctypes.c_int64 * 3)()
    assert lib.cpes_partition_chunks(1000, 24, 3, 0, offs, lens, FAKE, FAKE, 1 << 20, None, None) == \
        cp.ERR_INVALID_ARGUMENT
    assert lib.cpes_partition_chunks(1000, 512, 3, 0, offs, lens, FAKE, FAKE, 1 << 20, None, None) == \
        cp.ERR_INVALID_ARGUMENT                                                       # 2 chunks < K
    need = lib.cpes_partition_chunks_workspace_bytes(1 << 20, 64, 3)
    assert need > 0 and lib.cpes_partition_chunks_workspace_bytes(1 << 20, 48, 3) == 0
    assert lib.cpes_partition_chunks(1 << 20, 64, 3, 0, offs, lens, FAKE, FAKE, need - 1, None, None) == \
        cp.ERR_WORKSPACE


def test_binding_checks_buffer_sizes_and_dtypes(lib):
    """The C ABI cannot see buffer sizes; the binding rejects undersized or
    mistyped tensors before any launch (CPU tensors suffice: the checks come
    before the device-pointer checks)."""
    torch = pytest.importorskip("torch")
    w = torch.zeros(64, dtype=torch.bfloat16)
    s = cp.subspace(0, 32)
    with pytest.raises(ValueError, match="aux holds 31"):
        cp.cpes_perturb(w, s, 1e-3, 1, 1, aux=torch.zeros(31, dtype=torch.bfloat16), aux_mode=cp.AUX_SNAPSHOT)
    with pytest.raises(TypeError, match="aux must have dtype torch.float32"):
        cp.cpes_perturb(w, s, 1e-3, 1, 1, aux=torch.zeros(32, dtype=torch.bfloat16), aux_mode=cp.AUX_MASTER)
    with pytest.raises(ValueError, match="aux holds 16"):
        cp.cpes_restore(w, s, aux=torch.zeros(16, dtype=torch.bfloat16), aux_mode=cp.AUX_SNAPSHOT)
    with pytest.raises(ValueError, match="master holds"):
        cp.cpes_stage_master(w, s, torch.zeros(8, dtype=torch.float32))
    with pytest.raises(ValueError, match="index map holds 40"):
        cp.subspace(10, 31, torch.zeros(40, dtype=torch.int64))
    with pytest.raises(ValueError, match="index map holds 3"):              # chunks: offset 1 + ceil(40 / 16)
        cp.subspace(1, 40, torch.zeros(3, dtype=torch.int64), chunk=16)
    with pytest.raises(ValueError, match="must be a GPU tensor"):            # size accepted; a host map is not
        cp.subspace(1, 40, torch.zeros(4, dtype=torch.int64), chunk=16)
    with pytest.raises(ValueError, match="rnorm holds 3"):
        cp.cpes_update(w, s, [1, 2, 3, 4], [1, 1, 1, 1], torch.zeros(3, dtype=torch.float32), 5e-4, 1e-3)
    with pytest.raises(TypeError, match="rnorm must have dtype"):
        cp.cpes_update(w, s, [1], [1], torch.zeros(1, dtype=torch.float64), 5e-4, 1e-3)
    with pytest.raises(ValueError, match="out holds 7"):
        cp.cpes_normalize_rewards(torch.zeros(8), torch.zeros(7), cp.NORM_Z)
    with pytest.raises(ValueError, match="index holds 99"):
        cp.cpes_partition(cp.PART_PERMUTATION, 100, 4, 0, index=torch.zeros(99, dtype=torch.int64),
                          workspace=torch.zeros(16, dtype=torch.uint8))
    with pytest.raises(ValueError, match="bounds needs K"):
        cp.cpes_partition(cp.PART_CONTIGUOUS, 100, 4, bounds=[0, 50, 100])


def test_probes_reject_bad_arguments(lib):
    s = _sub(length=16, index=FAKE)
    plain = _sub(length=16)
    chunked = _sub(length=16, index=FAKE, chunk=8)
    cases = [
        (FAKE, 64, cp.BF16, ctypes.byref(plain), FAKE, 0),     # no element map
        (FAKE, 64, cp.BF16, ctypes.byref(chunked), FAKE, 0),   # chunk lists are not element maps
        (FAKE, 64, cp.BF16, ctypes.byref(s), None, 1),         # null buffer
        (FAKE, 64, cp.BF16, ctypes.byref(s), FAKE, 2),         # direction
        (None, 64, cp.BF16, ctypes.byref(s), FAKE, 0),         # null weights
    ]
    for args in cases:
        rc, msg = _rc_msg(lib, lib.cpes_probe_map_copy(*args, None))
        assert rc == cp.ERR_INVALID_ARGUMENT, (args, msg)
    for src, dst, n in ((None, FAKE, 16), (FAKE, None, 16), (FAKE, FAKE, 15), (FAKE, FAKE, -16), (FAKE + 8, FAKE, 16)):
        rc, msg = _rc_msg(lib, lib.cpes_probe_copy(src, dst, n, 0, None))
        assert rc == cp.ERR_INVALID_ARGUMENT, (src, dst, n, msg)
    assert lib.cpes_probe_copy(FAKE, FAKE, 0, 1, None) == cp.OK


def test_static_chunk_partition_rejects_before_any_gpu_call(lib):
    offs = (ctypes.c_int64 * 9)()
    lens = (ctypes.c_int64 * 8)()
    call = lambda d, chunk, K, o=offs, l=lens: lib.cpes_partition_chunks_static(d, chunk, K, 1, o, l, FAKE, None, None)
    assert call(0, 8, 1) == cp.ERR_INVALID_ARGUMENT                  # d < 1
    assert call(1 << 20, 12, 4) == cp.ERR_INVALID_ARGUMENT           # chunk not a power of two
    assert call(64, 8, 9) == cp.ERR_INVALID_ARGUMENT                 # K above the chunk count
    assert call(64, 8, 4, None) == cp.ERR_INVALID_ARGUMENT           # null host outputs
    rc = call((1 << 23) + 8, 8, 4)                                   # 2^20 + 1 chunks: beyond the static array
    assert rc == cp.ERR_UNSUPPORTED
    assert "static workspace" in lib.cpes_last_error().decode()


def test_unknown_subspace_flags_are_rejected(lib):
    s = _sub(index=FAKE, flags=cp.SUB_ASCENDING | 2)
    rc, msg = _rc_msg(lib, lib.cpes_restore(FAKE, 64, cp.BF16, ctypes.byref(s), 0.0, 0, 1, FAKE, cp.AUX_SNAPSHOT, None))
    assert rc == cp.ERR_INVALID_ARGUMENT and "flags" in msg
