"""Shards of a subspace (cpes_subspace.noise_offset): the single-GPU part of
the sharded update across GPUs.  Each shard [a, b) of a subspace is passed as
its own subspace with noise_offset = a; updating the shards one by one must
give the same bits as updating the whole subspace, since every position keeps
its noise index and its own arithmetic.  The oracle's window start (j0) checks
a shard's perturbation directly."""
import numpy as np
import pytest

import paper_2608_02391_amd as cp
import synthetic as S
from tests.gpu_helpers import to_dev, to_host, torch, ulp_bf16

pytestmark = pytest.mark.gpu


def _bounds(length, G, align):
    cuts = [0] + [((length * g // G) // align) * align for g in range(1, G)] + [length]
    return list(zip(cuts[:-1], cuts[1:]))


@pytest.mark.parametrize("layout", ["contiguous", "chunked"])
def test_sharded_update_equals_whole_update(layout):
    T = torch()
    assert T.cuda.is_available(), "GPU tests need an MI355X"
    cp.load()
    d, G = (1 << 22) + 4096, 8
    w = S.device_weights(d, S.BF16, 21)
    seeds = list(range(1, 31))
    signs = [1] * 30
    rn = T.from_numpy(np.linspace(-1.5, 1.5, 30).astype(np.float32)).cuda()
    if layout == "contiguous":
        off, L = 40, (1 << 22) + 1000
        whole = cp.subspace(off, L)
        shards = [cp.subspace(off + a, b - a, noise_offset=a) for a, b in _bounds(L, G, 8)]
    else:
        chunk = 1 << 12
        chunks = T.empty(-(-d // chunk), dtype=T.int64, device="cuda")
        ws = T.empty(cp.cpes_partition_chunks_workspace_bytes(d, chunk, 2), dtype=T.uint8, device="cuda")
        lo, lens = cp.cpes_partition_chunks(d, chunk, 2, 7, chunks, ws)
        L = lens[1]
        whole = cp.subspace(lo[1], L, chunks, chunk)
        shards = [cp.subspace(lo[1] + a // chunk, b - a, chunks, chunk, noise_offset=a)
                  for a, b in _bounds(L, G, chunk)]
    ref = w.clone()
    cp.cpes_update(ref, whole, seeds, signs, rn, 5e-4, 2e-3)
    for s in shards:
        cp.cpes_update(w, s, seeds, signs, rn, 5e-4, 2e-3)
    T.cuda.synchronize()
    assert T.equal(w, ref)


def test_shard_perturbation_matches_oracle_window(orc):
    T = torch()
    assert T.cuda.is_available(), "GPU tests need an MI355X"
    cp.load()
    n, a, L = 300000, 65536, 100003
    w = S.host_weights(n, S.BF16, 4)
    dw = to_dev(w)
    cp.cpes_perturb(dw, cp.subspace(17, L, noise_offset=a), 3e-3, 77, -1)
    orc.perturb(w, 17, L, np.float32(3e-3), 77, -1, j0=a)
    T.cuda.synchronize()
    assert ulp_bf16(to_host(dw), w).max() <= 1
