"""Python binding of ``libcpes`` -- the gfx950 C-ABI library of the CoPES
parameter-space hot path (see ``include/cpes.h``).

Argument marshalling only: every step runs in the library's HIP kernels.
Tensors must live on the GPU; streams default to torch's current stream.
There is no CPU fallback: if ``libcpes.so`` is missing or fails to load, every
call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcpes.so")

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, -1, -2, -3, -4
BF16, F32 = 0, 1
PART_CONTIGUOUS, PART_PERMUTATION = 0, 1
AUX_NONE, AUX_SNAPSHOT, AUX_MASTER, AUX_BACKUP = 0, 1, 2, 3
NORM_Z, NORM_RANK = 0, 1
SCALE_ALPHA_OVER_N_SIGMA, SCALE_ALPHA_OVER_N = 0, 1
SUB_ASCENDING = 1
MAX_MEMBERS, MAX_REWARDS, MAX_GROUPS, MAX_PERMUTATION_K, MAX_STEP_SUBSPACES = 256, 4096, 1024, 256, 32

EXPORTED = (
    "cpes_partition", "cpes_partition32", "cpes_partition_workspace_bytes", "cpes_partition_chunks",
    "cpes_partition_chunks_workspace_bytes", "cpes_partition_chunks_static", "cpes_perturb", "cpes_restore", "cpes_backup",
    "cpes_backup_to_host", "cpes_restore_from_host", "cpes_stage_master", "cpes_normalize_rewards",
    "cpes_update", "cpes_update_step", "cpes_update_step32", "cpes_debug_philox", "cpes_debug_normals", "cpes_debug_bm_grid",
    "cpes_debug_prp", "cpes_rng_probe", "cpes_probe_map_copy", "cpes_probe_copy", "cpes_fill_normal",
    "cpes_last_error", "cpes_abi_version",
)


class CpesError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{message} (status {code})")
        self.code = code


class Subspace(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_int64), ("length", ctypes.c_int64), ("index", ctypes.c_void_p),
                ("chunk", ctypes.c_int64), ("index32", ctypes.c_void_p), ("noise_offset", ctypes.c_int64),
                ("flags", ctypes.c_int64)]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load ``libcpes.so`` (built by ``paper_2608_02391_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2608_02391_amd.build`")
    L = ctypes.CDLL(path)
    vp, i64, u64, i32, u32, f32 = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int32,
                                   ctypes.c_uint32, ctypes.c_float)
    sp = ctypes.POINTER(Subspace)
    sig = {
        "cpes_partition": [i32, i64, i32, u64, vp, vp, vp, vp, ctypes.c_size_t, vp, vp],
        "cpes_partition32": [i64, i32, u64, vp, vp, vp, ctypes.c_size_t, vp, vp],
        "cpes_partition_workspace_bytes": [i32, i64, i32],
        "cpes_partition_chunks": [i64, i64, i32, u64, vp, vp, vp, vp, ctypes.c_size_t, vp, vp],
        "cpes_partition_chunks_workspace_bytes": [i64, i64, i32],
        "cpes_partition_chunks_static": [i64, i64, i32, u64, vp, vp, vp, vp, vp],
        "cpes_perturb": [vp, i64, i32, sp, f32, u64, i32, vp, i32, vp],
        "cpes_restore": [vp, i64, i32, sp, f32, u64, i32, vp, i32, vp],
        "cpes_backup": [vp, i64, i32, sp, vp, vp],
        "cpes_backup_to_host": [vp, i64, i32, sp, vp, vp],
        "cpes_restore_from_host": [vp, i64, i32, sp, vp, vp],
        "cpes_stage_master": [vp, i64, i32, sp, vp, vp],
        "cpes_normalize_rewards": [vp, i32, i32, vp, i32, vp, vp, vp],
        "cpes_update": [vp, i64, i32, sp, vp, i32, vp, vp, vp, f32, f32, i32, vp],
        "cpes_update_step": [vp, i64, i32, i32, vp, vp, i64, vp, i32, vp, vp, vp, vp, f32, vp, i32, vp],
        "cpes_update_step32": [vp, i64, i32, i32, vp, vp, i32, vp, vp, vp, vp, f32, vp, i32, vp],
        "cpes_debug_philox": [u64, u32, u64, i64, vp, vp],
        "cpes_debug_normals": [u64, i64, i64, vp, vp],
        "cpes_debug_bm_grid": [u32, i64, vp, vp, vp, vp],
        "cpes_debug_prp": [u64, i64, i32, i64, i64, vp, vp, vp],
        "cpes_rng_probe": [u64, i64, vp, vp],
        "cpes_probe_map_copy": [vp, i64, i32, sp, vp, i32, vp],
        "cpes_probe_copy": [vp, vp, i64, i32, vp],
        "cpes_fill_normal": [vp, i64, i32, u64, u32, f32, vp],
        "cpes_last_error": [],
        "cpes_abi_version": [],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    L.cpes_partition_workspace_bytes.restype = ctypes.c_size_t
    L.cpes_partition_chunks_workspace_bytes.restype = ctypes.c_size_t
    L.cpes_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def last_error() -> str:
    return load().cpes_last_error().decode()


def _check(rc: int) -> None:
    if rc != OK:
        raise CpesError(rc, last_error())


# ----------------------------------------------------------- marshalling --

def _torch():
    import torch

    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"weights must be bfloat16 or float32, not {t.dtype}")


def _dev_ptr(t, what: str) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return t.data_ptr()


def _need(t, what: str, numel: int, dtype=None) -> None:
    """A device buffer the kernels will address: it must hold ``numel``
    elements (of ``dtype`` when given).  The C ABI takes bare pointers and
    cannot see sizes, so the binding checks them before any launch."""
    if t is None:
        return
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} must have dtype {dtype}, not {t.dtype}")
    if t.numel() < numel:
        raise ValueError(f"{what} holds {t.numel()} elements, {numel} needed")


def _aux_need(w, s: "Subspace", aux, aux_mode: int, what: str = "aux") -> None:
    torch = _torch()
    if aux_mode == AUX_MASTER:
        _need(aux, what, s.length, torch.float32)
    elif aux_mode in (AUX_SNAPSHOT, AUX_BACKUP):
        _need(aux, what, s.length, w.dtype)


def _host_ptr(t, w, s: "Subspace", what: str) -> int:
    """A host backup: a CPU tensor of w's dtype holding at least s.length
    elements.  Whether it is pinned is checked by the library."""
    if t.is_cuda:
        raise ValueError(f"{what} must be a host tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if t.dtype != w.dtype:
        raise TypeError(f"{what} must have dtype {w.dtype}, not {t.dtype}")
    if t.numel() < s.length:
        raise ValueError(f"{what} holds {t.numel()} elements, {s.length} needed")
    return t.data_ptr()


def _current_stream() -> int:
    """torch's current stream on the current device, as a raw hipStream_t."""
    torch = _torch()
    raw, dev = getattr(torch._C, "_cuda_getCurrentRawStream", None), getattr(torch._C, "_cuda_getDevice", None)
    if raw is not None and dev is not None:
        return raw(dev())               # the same handle, without building a Stream object per call
    return torch.cuda.current_stream().cuda_stream


def _stream(stream) -> Optional[int]:
    if stream is None:
        return _current_stream()
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def subspace(offset: int, length: int, index=None, chunk: int = 0, noise_offset: int = 0,
             ascending: bool = False) -> Subspace:
    """Positions j < length at parameter offset + j, index[offset + j], or
    (chunk > 0) index[offset + j // chunk] * chunk + j % chunk; the map must
    hold the entries those positions read.  An int64 map
    goes to ``index``; a 32-bit map (torch.int32 or torch.uint32 holding the
    uint32 entries of cpes_partition32) goes to ``index32``.  Position j uses
    noise index noise_offset + j (a shard of a larger subspace).
    ascending=True sets CPES_SUB_ASCENDING: the element map is strictly
    ascending (a partition's own map), so bf16 perturbations and restores may
    rewrite whole 128-byte lines around its entries."""
    torch = _torch()
    idx64 = idx32 = None
    if index is not None:
        if length > 0:
            entries = offset + (-(-length // chunk) if chunk else length)
            _need(index, "index map", entries)
        if index.dtype == torch.int64:
            idx64 = _dev_ptr(index, "index map")
        elif index.dtype in (torch.int32, getattr(torch, "uint32", torch.int32)):
            idx32 = _dev_ptr(index, "index map")
        else:
            raise TypeError("index map must be int64, or 32-bit for a uint32 map")
    sub = Subspace(int(offset), int(length), idx64, int(chunk), idx32, int(noise_offset),
                   SUB_ASCENDING if ascending else 0)
    sub._index = index      # the descriptor holds a raw pointer: keep the map's storage alive with it
    return sub


# ------------------------------------------------------------- entry points --

def cpes_partition(mode: int, d: int, K: int, seed: int = 0, bounds: Optional[Sequence[int]] = None,
                   index=None, workspace=None, status=None, stream=None):
    """Returns the K+1 subspace offsets (host ints); PERMUTATION fills ``index``."""
    L = load()
    offsets = (ctypes.c_int64 * (K + 1))()
    b = None if bounds is None else (ctypes.c_int64 * (K + 1))(*[int(x) for x in bounds])
    if bounds is not None and len(bounds) != K + 1:
        raise ValueError(f"bounds needs K + 1 = {K + 1} entries, not {len(bounds)}")
    if mode == PART_PERMUTATION:
        _need(index, "index", d, _torch().int64)
    _need(status, "status", 1, _torch().int32)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(L.cpes_partition(mode, d, K, seed, b, offsets, _dev_ptr(index, "index"),
                            _dev_ptr(workspace, "workspace"), ws_bytes, _dev_ptr(status, "status"),
                            _stream(stream)))
    return [int(x) for x in offsets]


def cpes_partition32(d: int, K: int, seed: int, index, workspace, status=None, stream=None):
    """Permutation partition into a 32-bit map (d <= 2^32); returns the K+1 offsets."""
    L = load()
    offsets = (ctypes.c_int64 * (K + 1))()
    if index.element_size() != 4:
        raise TypeError("cpes_partition32 writes a 32-bit map")
    _need(index, "index", d)
    _need(status, "status", 1, _torch().int32)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(L.cpes_partition32(d, K, seed, offsets, _dev_ptr(index, "index"), _dev_ptr(workspace, "workspace"),
                              ws_bytes, _dev_ptr(status, "status"), _stream(stream)))
    return [int(x) for x in offsets]


def cpes_partition_workspace_bytes(mode: int, d: int, K: int) -> int:
    return int(load().cpes_partition_workspace_bytes(mode, d, K))


def cpes_partition_chunks(d: int, chunk: int, K: int, seed: int, chunks, workspace, status=None, stream=None):
    """Chunk-granular random partition; returns (list_offsets[K+1], lengths[K])."""
    L = load()
    offs = (ctypes.c_int64 * (K + 1))()
    lens = (ctypes.c_int64 * K)()
    _need(chunks, "chunks", -(-d // chunk) if chunk > 0 else 0, _torch().int64)
    _need(status, "status", 1, _torch().int32)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(L.cpes_partition_chunks(d, chunk, K, seed, offs, lens, _dev_ptr(chunks, "chunks"),
                                   _dev_ptr(workspace, "workspace"), ws_bytes, _dev_ptr(status, "status"),
                                   _stream(stream)))
    return [int(x) for x in offs], [int(x) for x in lens]


def cpes_partition_chunks_static(d: int, chunk: int, K: int, seed: int, chunks, status=None, stream=None):
    """cpes_partition_chunks on the library's own device scratch array (no
    workspace, no allocation); returns (list_offsets[K+1], lengths[K])."""
    L = load()
    offs = (ctypes.c_int64 * (K + 1))()
    lens = (ctypes.c_int64 * K)()
    _need(chunks, "chunks", -(-d // chunk) if chunk > 0 else 0, _torch().int64)
    _need(status, "status", 1, _torch().int32)
    _check(L.cpes_partition_chunks_static(d, chunk, K, seed, offs, lens, _dev_ptr(chunks, "chunks"),
                                          _dev_ptr(status, "status"), _stream(stream)))
    return [int(x) for x in offs], [int(x) for x in lens]


def cpes_partition_chunks_workspace_bytes(d: int, chunk: int, K: int) -> int:
    return int(load().cpes_partition_chunks_workspace_bytes(d, chunk, K))


def cpes_perturb(w, s: Subspace, sigma: float, seed: int, sign: int, aux=None, aux_mode: int = AUX_NONE,
                 stream=None) -> None:
    _aux_need(w, s, aux, aux_mode)
    _check(load().cpes_perturb(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s), sigma, seed, sign,
                               _dev_ptr(aux, "aux"), aux_mode, _stream(stream)))


def cpes_restore(w, s: Subspace, sigma: float = 0.0, seed: int = 0, sign: int = 1, aux=None,
                 aux_mode: int = AUX_SNAPSHOT, stream=None) -> None:
    _aux_need(w, s, aux, aux_mode)
    _check(load().cpes_restore(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s), sigma, seed, sign,
                               _dev_ptr(aux, "aux"), aux_mode, _stream(stream)))


def cpes_backup(w, s: Subspace, backup, stream=None) -> None:
    """backup[j] = w[p(j)] into a device tensor of w's dtype."""
    _need(backup, "backup", s.length, w.dtype)
    _check(load().cpes_backup(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s),
                              _dev_ptr(backup, "backup"), _stream(stream)))


def cpes_backup_to_host(w, s: Subspace, backup, stream=None) -> None:
    """backup[j] = w[p(j)] into a pinned host tensor (``pin_memory=True``)."""
    _check(load().cpes_backup_to_host(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s),
                                      _host_ptr(backup, w, s, "backup"), _stream(stream)))


def cpes_restore_from_host(w, s: Subspace, backup, stream=None) -> None:
    """w[p(j)] = backup[j] from a pinned host tensor."""
    _check(load().cpes_restore_from_host(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s),
                                         _host_ptr(backup, w, s, "backup"), _stream(stream)))


def cpes_fill_normal(w, seed: int, domain: int = 1, stddev: float = 0.02, stream=None) -> None:
    """Fill the device tensor w with cast(stddev * z_j) from stream (seed, domain)."""
    _check(load().cpes_fill_normal(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), seed, domain, stddev,
                                   _stream(stream)))


def cpes_stage_master(w, s: Subspace, master, stream=None) -> None:
    _need(master, "master", s.length, _torch().float32)
    _check(load().cpes_stage_master(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s),
                                    _dev_ptr(master, "master"), _stream(stream)))


def cpes_normalize_rewards(r, out, mode: int = NORM_Z, group=None, n_groups: int = 1, status=None,
                           stream=None) -> None:
    torch = _torch()
    _need(r, "rewards", 0, torch.float32)
    _need(out, "out", r.numel(), torch.float32)
    _need(group, "group", r.numel(), torch.int32)
    _need(status, "status", 1, torch.int32)
    _check(load().cpes_normalize_rewards(_dev_ptr(r, "rewards"), r.numel(), mode, _dev_ptr(group, "group"),
                                         n_groups, _dev_ptr(out, "out"), _dev_ptr(status, "status"),
                                         _stream(stream)))


def cpes_update(w, s: Subspace, seeds: Sequence[int], signs: Sequence[int], rnorm, alpha: float, sigma: float,
                scale_mode: int = SCALE_ALPHA_OVER_N_SIGMA, master=None, stream=None) -> None:
    n = len(seeds)
    if len(signs) != n:
        raise ValueError("seeds and signs differ in length")
    _need(rnorm, "rnorm", n, _torch().float32)
    _need(master, "master", s.length, _torch().float32)
    cs = (ctypes.c_uint64 * n)(*[int(x) & 0xFFFFFFFFFFFFFFFF for x in seeds])
    cg = (ctypes.c_int8 * n)(*[int(x) for x in signs])
    _check(load().cpes_update(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s),
                              _dev_ptr(master, "master"), n, cs, cg, _dev_ptr(rnorm, "rnorm"), alpha, sigma,
                              scale_mode, _stream(stream)))


def cpes_update_step(w, offsets: Sequence[int], seeds: Sequence[int], signs: Sequence[int],
                     subspaces: Sequence[int], rnorm, alpha: float, sigmas: Sequence[float],
                     scale_mode: int = SCALE_ALPHA_OVER_N_SIGMA, index=None, chunk: int = 0,
                     lengths: Optional[Sequence[int]] = None, stream=None) -> None:
    """Update every subspace of a partition with its own members (one launch).
    ``index``: None (contiguous), an int64 map or chunk list, or a 32-bit map
    (cpes_partition32) that goes to cpes_update_step32."""
    K = len(offsets) - 1
    n = len(seeds)
    if not (len(signs) == len(subspaces) == n) or len(sigmas) != K:
        raise ValueError("inconsistent member or subspace arrays")
    co = (ctypes.c_int64 * (K + 1))(*[int(x) for x in offsets])
    cs = (ctypes.c_uint64 * n)(*[int(x) & 0xFFFFFFFFFFFFFFFF for x in seeds])
    cg = (ctypes.c_int8 * n)(*[int(x) for x in signs])
    ck = (ctypes.c_int32 * n)(*[int(x) for x in subspaces])
    csg = (ctypes.c_float * K)(*[float(x) for x in sigmas])
    torch = _torch()
    idx32 = index is not None and index.dtype in (torch.int32, getattr(torch, "uint32", torch.int32))
    if index is not None and index.dtype != torch.int64 and not idx32:
        raise TypeError("index map must be int64, or 32-bit for a uint32 map")
    if idx32 and chunk:
        raise ValueError("chunk lists are int64 maps")
    if lengths is not None and len(lengths) != K:
        raise ValueError(f"lengths needs K = {K} entries, not {len(lengths)}")
    _need(index, "index map", int(offsets[-1]))
    _need(rnorm, "rnorm", n, torch.float32)
    if idx32:
        _check(load().cpes_update_step32(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), K, co, _dev_ptr(index, "index"),
                                         n, cs, cg, ck, _dev_ptr(rnorm, "rnorm"), alpha, csg, scale_mode,
                                         _stream(stream)))
        return
    cl = None if lengths is None else (ctypes.c_int64 * K)(*[int(x) for x in lengths])
    _check(load().cpes_update_step(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), K, co, _dev_ptr(index, "index"),
                                   int(chunk), cl, n, cs, cg, ck, _dev_ptr(rnorm, "rnorm"), alpha, csg, scale_mode,
                                   _stream(stream)))


def cpes_debug_philox(seed: int, domain: int, q0: int, nblocks: int, out, stream=None) -> None:
    if out is not None and out.numel() * out.element_size() < 16 * nblocks:
        raise ValueError(f"out holds {out.numel() * out.element_size()} bytes, {16 * nblocks} needed")
    _check(load().cpes_debug_philox(seed, domain, q0, nblocks, _dev_ptr(out, "out"), _stream(stream)))


def cpes_debug_normals(seed: int, j0: int, n: int, out, stream=None) -> None:
    _need(out, "out", n, _torch().float32)
    _check(load().cpes_debug_normals(seed, j0, n, _dev_ptr(out, "out"), _stream(stream)))


def cpes_debug_bm_grid(m0: int, n: int, rho=None, cos=None, sin=None, stream=None) -> None:
    for t, what in ((rho, "rho"), (cos, "cos"), (sin, "sin")):
        _need(t, what, n, _torch().float64)
    _check(load().cpes_debug_bm_grid(m0, n, _dev_ptr(rho, "rho"), _dev_ptr(cos, "cos"), _dev_ptr(sin, "sin"),
                                     _stream(stream)))


def cpes_debug_prp(seed: int, d: int, K: int, i0: int, n: int, perm=None, bucket=None, stream=None) -> None:
    _need(perm, "perm", n, _torch().int64)
    _need(bucket, "bucket", n, _torch().int32)
    _check(load().cpes_debug_prp(seed, d, K, i0, n, _dev_ptr(perm, "perm"), _dev_ptr(bucket, "bucket"),
                                 _stream(stream)))


def cpes_rng_probe(seed: int, n: int, sink, stream=None) -> None:
    if sink is not None and sink.numel() * sink.element_size() < 4:
        raise ValueError("sink needs at least 4 bytes")
    _check(load().cpes_rng_probe(seed, n, _dev_ptr(sink, "sink"), _stream(stream)))


def cpes_probe_map_copy(w, s: Subspace, buf, direction: int, stream=None) -> None:
    """Plain gather (direction 0: buf[j] = w[p(j)]) or scatter (1: w[p(j)] =
    buf[j]) through the subspace's element map: a measurement reference."""
    _need(buf, "buf", s.length, w.dtype)
    _check(load().cpes_probe_map_copy(_dev_ptr(w, "w"), w.numel(), _dtype_code(w), ctypes.byref(s),
                                      _dev_ptr(buf, "buf"), direction, _stream(stream)))


def cpes_probe_copy(src, dst, nbytes: int, nontemporal: bool = False, stream=None) -> None:
    """dst[:nbytes] = src[:nbytes], one 16-byte vector per thread (non-temporal
    accesses if asked): a measurement reference."""
    for t, what in ((src, "src"), (dst, "dst")):
        if t.numel() * t.element_size() < nbytes:
            raise ValueError(f"{what} holds fewer than {nbytes} bytes")
    _check(load().cpes_probe_copy(_dev_ptr(src, "src"), _dev_ptr(dst, "dst"), nbytes, int(bool(nontemporal)),
                                  _stream(stream)))


def cpes_abi_version() -> int:
    return int(load().cpes_abi_version())
