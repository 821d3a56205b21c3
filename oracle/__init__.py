"""CPU oracle for the CoPES parameter-space hot path -- test infrastructure only.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never does: it has
no CPU fallback.

The arithmetic lives in ``cpes_oracle.c`` (plain C, IEEE double, no fast-math,
no contraction); this module only builds it with gcc and marshals numpy arrays
through ctypes.  bf16 arrays are passed as ``numpy.uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cpes_oracle.c")
_LIB = os.path.join(_HERE, "libcpes_oracle.so")

BF16, F32 = 0, 1
AUX_NONE, AUX_SNAPSHOT, AUX_MASTER, AUX_BACKUP = 0, 1, 2, 3
NORM_Z, NORM_RANK = 0, 1
SCALE_ALPHA_OVER_N_SIGMA, SCALE_ALPHA_OVER_N = 0, 1
PART_CONTIGUOUS, PART_PERMUTATION = 0, 1
DOMAIN_NOISE, DOMAIN_PARTITION = 0, 3

_c_i64p = ctypes.POINTER(ctypes.c_int64)
_c_u32p = ctypes.POINTER(ctypes.c_uint32)
_c_f32p = ctypes.POINTER(ctypes.c_float)
_c_f64p = ctypes.POINTER(ctypes.c_double)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math, no FP contraction)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=gnu11", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True, cwd=_HERE)
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        vp, i64, u64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int, ctypes.c_float
        L.orc_philox4x32_10.argtypes = [_c_u32p, _c_u32p, _c_u32p]
        L.orc_block.argtypes = [u64, ctypes.c_uint32, u64, _c_u32p]
        L.orc_uniform_open0.argtypes = [ctypes.c_uint32]
        L.orc_uniform_open0.restype = ctypes.c_double
        L.orc_bm_radius.argtypes = [ctypes.c_uint32]
        L.orc_bm_radius.restype = ctypes.c_double
        L.orc_bm_angle.argtypes = [ctypes.c_uint32, _c_f64p, _c_f64p]
        L.orc_bm_radius_many.argtypes = [vp, i64, vp]
        L.orc_bm_angle_many.argtypes = [vp, i64, vp, vp]
        L.orc_blocks.argtypes = [u64, ctypes.c_uint32, u64, i64, vp]
        L.orc_normal.argtypes = [u64, i64]
        L.orc_normal.restype = ctypes.c_float
        L.orc_normals.argtypes = [u64, i64, i64, _c_f32p]
        L.orc_normal_domain.argtypes = [u64, ctypes.c_uint32, i64]
        L.orc_normal_domain.restype = ctypes.c_float
        L.orc_fill_normal.argtypes = [vp, ctypes.c_int, i64, u64, ctypes.c_uint32, ctypes.c_float]
        L.orc_f32_to_bf16.argtypes = [f32]
        L.orc_f32_to_bf16.restype = ctypes.c_uint16
        L.orc_perturb.argtypes = [vp, i32, i64, i64, vp, i64, f32, u64, i32, vp, i32]
        L.orc_restore.argtypes = [vp, i32, i64, i64, vp, i64, f32, u64, i32, vp, i32]
        L.orc_stage_master.argtypes = [vp, i32, i64, i64, vp, vp]
        L.orc_normalize.argtypes = [vp, i32, i32, vp, vp, ctypes.POINTER(ctypes.c_int)]
        L.orc_update.argtypes = [vp, i32, i64, i64, vp, i64, vp, i32, vp, vp, vp, f32, f32, i32]
        L.orc_update_step.argtypes = [vp, i32, i32, vp, vp, i32, vp, vp, vp, vp, f32, vp, i32]
        L.orc_prp.argtypes = [u64, i64, i64]
        L.orc_prp.restype = i64
        L.orc_bucket.argtypes = [u64, i64, ctypes.c_int32, i64]
        L.orc_bucket.restype = ctypes.c_int32
        L.orc_partition.argtypes = [i32, i64, ctypes.c_int32, u64, vp, vp, vp]
        L.orc_partition_chunks.argtypes = [i64, i64, ctypes.c_int32, u64, vp, vp, vp]
        L.orc_num_threads.restype = i32
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


def _dtype_code(w: np.ndarray) -> int:
    if w.dtype == np.uint16:
        return BF16
    if w.dtype == np.float32:
        return F32
    raise TypeError("weights must be uint16 (bf16 bits) or float32")


# ---------------------------------------------------------------- generator --

def philox4x32_10(ctr, key) -> np.ndarray:
    c = (ctypes.c_uint32 * 4)(*[int(x) & 0xFFFFFFFF for x in ctr])
    k = (ctypes.c_uint32 * 2)(*[int(x) & 0xFFFFFFFF for x in key])
    o = (ctypes.c_uint32 * 4)()
    lib().orc_philox4x32_10(c, k, o)
    return np.array(list(o), dtype=np.uint32)


def block(seed: int, domain: int, q: int) -> np.ndarray:
    o = (ctypes.c_uint32 * 4)()
    lib().orc_block(seed, domain, q, o)
    return np.array(list(o), dtype=np.uint32)


def blocks(seed: int, domain: int, q0: int, nblocks: int) -> np.ndarray:
    """Words of blocks q0 .. q0+nblocks-1, flattened (4 words per block)."""
    out = np.empty(4 * nblocks, dtype=np.uint32)
    lib().orc_blocks(seed, domain, q0, nblocks, _ptr(out))
    return out


def uniform_open0(x: int) -> float:
    return lib().orc_uniform_open0(x)


def bm_radius(a: int) -> float:
    return lib().orc_bm_radius(a)


def bm_angle(b: int):
    c, s = ctypes.c_double(), ctypes.c_double()
    lib().orc_bm_angle(b, ctypes.byref(c), ctypes.byref(s))
    return c.value, s.value


def bm_radius_many(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.uint32)
    out = np.empty(a.size, dtype=np.float64)
    lib().orc_bm_radius_many(_ptr(a), a.size, _ptr(out))
    return out


def bm_angle_many(b):
    b = np.ascontiguousarray(b, dtype=np.uint32)
    c = np.empty(b.size, dtype=np.float64)
    s = np.empty(b.size, dtype=np.float64)
    lib().orc_bm_angle_many(_ptr(b), b.size, _ptr(c), _ptr(s))
    return c, s


def normal(seed: int, j: int) -> float:
    return lib().orc_normal(seed, j)


def normals(seed: int, j0: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    lib().orc_normals(seed, j0, n, out.ctypes.data_as(_c_f32p))
    return out


def normal_domain(seed: int, domain: int, j: int) -> float:
    return lib().orc_normal_domain(seed, domain, j)


def fill_normal(n: int, dtype: int, seed: int, domain: int, stddev: float) -> np.ndarray:
    """Seeded weights: cast(stddev * z_j) for j < n from stream (seed, domain)."""
    w = np.empty(n, dtype=np.uint16 if dtype == BF16 else np.float32)
    _check(lib().orc_fill_normal(_ptr(w), dtype, n, seed, domain, stddev), "fill_normal")
    return w


def f32_to_bf16(x: float) -> int:
    return lib().orc_f32_to_bf16(x)


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------- path ops --

def perturb(w, offset, length, sigma, seed, sign, index=None, j0=0, aux=None, aux_mode=AUX_NONE):
    """In place on the host array ``w``; ``aux`` is the snapshot (out) or master (in)."""
    _check(lib().orc_perturb(_ptr(w), _dtype_code(w), offset, length, _ptr(index), j0,
                             sigma, seed, sign, _ptr(aux), aux_mode), "perturb")


def restore(w, offset, length, sigma, seed, sign, index=None, j0=0, aux=None, aux_mode=AUX_NONE):
    _check(lib().orc_restore(_ptr(w), _dtype_code(w), offset, length, _ptr(index), j0,
                             sigma, seed, sign, _ptr(aux), aux_mode), "restore")


def stage_master(w, offset, length, index=None) -> np.ndarray:
    m = np.empty(length, dtype=np.float32)
    _check(lib().orc_stage_master(_ptr(w), _dtype_code(w), offset, length, _ptr(index), _ptr(m)),
           "stage_master")
    return m


def normalize(r, mode=NORM_Z, group=None):
    r = np.ascontiguousarray(r, dtype=np.float32)
    g = None if group is None else np.ascontiguousarray(group, dtype=np.int32)
    out = np.empty_like(r)
    st = ctypes.c_int(0)
    _check(lib().orc_normalize(_ptr(r), r.size, mode, _ptr(g), _ptr(out), ctypes.byref(st)),
           "normalize")
    return out, st.value


def update(w, offset, length, seeds, signs, rnorm, alpha, sigma, scale_mode=SCALE_ALPHA_OVER_N_SIGMA,
           index=None, j0=0, master=None):
    seeds = np.ascontiguousarray(seeds, dtype=np.uint64)
    signs = np.ascontiguousarray(signs, dtype=np.int8)
    rnorm = np.ascontiguousarray(rnorm, dtype=np.float32)
    assert seeds.size == signs.size == rnorm.size
    _check(lib().orc_update(_ptr(w), _dtype_code(w), offset, length, _ptr(index), j0, _ptr(master),
                            seeds.size, _ptr(seeds), _ptr(signs), _ptr(rnorm), alpha, sigma,
                            scale_mode), "update")


def update_step(w, offsets, seeds, signs, subspaces, rnorm, alpha, sigmas, scale_mode=SCALE_ALPHA_OVER_N_SIGMA,
                index=None):
    offsets = np.ascontiguousarray(offsets, dtype=np.int64)
    K = offsets.size - 1
    seeds = np.ascontiguousarray(seeds, dtype=np.uint64)
    signs = np.ascontiguousarray(signs, dtype=np.int8)
    subspaces = np.ascontiguousarray(subspaces, dtype=np.int32)
    rnorm = np.ascontiguousarray(rnorm, dtype=np.float32)
    sigmas = np.ascontiguousarray(sigmas, dtype=np.float32)
    assert seeds.size == signs.size == subspaces.size == rnorm.size and sigmas.size == K
    _check(lib().orc_update_step(_ptr(w), _dtype_code(w), K, _ptr(offsets), _ptr(index), seeds.size, _ptr(seeds),
                                 _ptr(signs), _ptr(subspaces), _ptr(rnorm), alpha, _ptr(sigmas), scale_mode),
           "update_step")


def prp(seed: int, d: int, x: int) -> int:
    return lib().orc_prp(seed, d, x)


def bucket(seed: int, d: int, K: int, i: int) -> int:
    return lib().orc_bucket(seed, d, K, i)


def partition(mode, d, K, seed=0, bounds=None, with_index=True):
    offsets = np.empty(K + 1, dtype=np.int64)
    b = None if bounds is None else np.ascontiguousarray(bounds, dtype=np.int64)
    index = np.empty(d, dtype=np.int64) if (mode == PART_PERMUTATION and with_index) else None
    _check(lib().orc_partition(mode, d, K, seed, _ptr(b), _ptr(offsets), _ptr(index)), "partition")
    return offsets, index


def partition_chunks(d, chunk, K, seed):
    """Returns (list_offsets[K+1], lengths[K], chunk ids grouped by subspace)."""
    n_chunks = -(-d // chunk)
    offs = np.empty(K + 1, dtype=np.int64)
    lens = np.empty(K, dtype=np.int64)
    chunks = np.empty(n_chunks, dtype=np.int64)
    _check(lib().orc_partition_chunks(d, chunk, K, seed, _ptr(offs), _ptr(lens), _ptr(chunks)), "partition_chunks")
    return offs, lens, chunks


def expand_chunks(chunks, list_offset, length, chunk):
    """Element map of a chunked subspace: position j -> chunks[list_offset + j // chunk] * chunk + j % chunk."""
    j = np.arange(length, dtype=np.int64)
    return chunks[list_offset + j // chunk] * chunk + j % chunk


def num_threads() -> int:
    return lib().orc_num_threads()
