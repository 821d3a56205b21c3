"""cpes_partition_chunks_static, the allocation-free chunk partition: through
the C ABI, bit-identical to cpes_partition_chunks with a caller workspace, on
two calls in a row (the second smaller, so stale contents of the shared
device array would show)."""
import numpy as np
import pytest
import torch

import paper_2608_02391_amd as cp


@pytest.mark.gpu
def test_static_chunk_partition_matches_workspace_partition():
    cp.load()
    torch.cuda.set_device(0)
    cases = [((3 << 17) * 8 + 5, 8, 16, 77), (100_003, 16, 5, 78)]   # 393,217 then 6,251 chunks
    for d, chunk, K, seed in cases:
        print(f"static chunk partition d={d} chunk={chunk} K={K} seed={seed}", flush=True)
        n_chunks = -(-d // chunk)
        ref = torch.full((n_chunks,), -7, dtype=torch.int64, device="cuda")
        got = torch.full((n_chunks,), -9, dtype=torch.int64, device="cuda")
        ws = torch.empty(cp.cpes_partition_chunks_workspace_bytes(d, chunk, K), dtype=torch.uint8, device="cuda")
        st_ref = torch.full((1,), 5, dtype=torch.int32, device="cuda")
        st_got = torch.full((1,), 5, dtype=torch.int32, device="cuda")
        offs_ref, lens_ref = cp.cpes_partition_chunks(d, chunk, K, seed, ref, ws, status=st_ref)
        offs_got, lens_got = cp.cpes_partition_chunks_static(d, chunk, K, seed, got, status=st_got)
        torch.cuda.synchronize()
        assert offs_got == offs_ref and lens_got == lens_ref
        assert sum(lens_got) == d
        assert int(st_ref.item()) == 0 and int(st_got.item()) == 0
        a, b = ref.cpu().numpy(), got.cpu().numpy()
        assert np.array_equal(a, b)
        assert np.array_equal(np.sort(b), np.arange(n_chunks))      # every chunk exactly once
