"""The hot path under HIP graph capture.  Every entry point only enqueues
kernels (no allocation, no memset node, no host synchronisation), so a whole
member loop plus the update can be captured once and replayed.  Each replay
must equal the same calls run eagerly, bit for bit (the kernels are
deterministic), with eager work and synchronisations between replays."""
import numpy as np
import pytest

import paper_2608_02391_amd as cp
import synthetic as S
from tests.gpu_helpers import torch

pytestmark = pytest.mark.gpu


def _step(w, subs, backup, rewards, rnorm, sigmas, seeds, signs, alpha):
    for k, s in enumerate(subs):
        for m, (seed, sign) in enumerate(zip(seeds, signs)):
            mode = cp.AUX_SNAPSHOT if m == 0 else cp.AUX_NONE
            cp.cpes_perturb(w, s, sigmas[k], seed + 100 * k, sign, aux=backup[:s.length], aux_mode=mode)
            cp.cpes_restore(w, s, aux=backup[:s.length], aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_normalize_rewards(rewards[k], rnorm[k], cp.NORM_Z)
        cp.cpes_update(w, s, [x + 100 * k for x in seeds], signs, rnorm[k], alpha, sigmas[k])


@pytest.mark.parametrize("layout", ["contiguous", "chunked"])
def test_captured_step_replays_match_eager(layout):
    T = torch()
    assert T.cuda.is_available(), "GPU tests need an MI355X"
    cp.load()
    d, K, n = (1 << 22) + 37, 4, 6
    dev = T.device("cuda")
    w0 = S.device_weights(d, S.BF16, 3)
    if layout == "contiguous":
        offs = cp.cpes_partition(cp.PART_CONTIGUOUS, d, K)
        subs = [cp.subspace(offs[k], offs[k + 1] - offs[k]) for k in range(K)]
    else:
        chunk = 1 << 12
        chunks = T.empty(-(-d // chunk), dtype=T.int64, device=dev)
        ws = T.empty(cp.cpes_partition_chunks_workspace_bytes(d, chunk, K), dtype=T.uint8, device=dev)
        lo, lens = cp.cpes_partition_chunks(d, chunk, K, 5, chunks, ws)
        subs = [cp.subspace(lo[k], lens[k], chunks, chunk) for k in range(K)]
    backup = T.empty(max(s.length for s in subs), dtype=T.bfloat16, device=dev)
    rewards = T.from_numpy(np.stack([S.rewards("uniform", n, 50 + k) for k in range(K)])).to(dev)
    rnorm = T.empty_like(rewards)
    sigmas = [float(np.float32(2e-3 * np.sqrt(d / s.length))) for s in subs]
    args = (backup, rewards, rnorm, sigmas, list(range(1, n + 1)), [1, -1] * (n // 2), 5e-4)

    ref = w0.clone()                                   # eager reference: three steps
    refs = []
    for _ in range(3):
        _step(ref, subs, *args)
        T.cuda.synchronize()
        refs.append(ref.clone())

    w = w0.clone()
    g = T.cuda.CUDAGraph()
    side = T.cuda.Stream()
    side.wait_stream(T.cuda.current_stream())
    with T.cuda.stream(side):                          # warm-up outside the graph
        scratch = w0.clone()
        _step(scratch, subs, *args)
    T.cuda.current_stream().wait_stream(side)
    T.cuda.synchronize()
    with T.cuda.graph(g):
        _step(w, subs, *args)
    for r in range(3):
        g.replay()
        T.cuda.synchronize()
        assert T.equal(w, refs[r]), f"replay {r}"
        junk = T.randn(1 << 20, device=dev) * 2      # unrelated eager work between replays
        del junk
        T.cuda.synchronize()
