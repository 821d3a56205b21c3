"""Pins of the oracle's partition (Eq. 7): disjoint subspaces that cover all d
indices with sizes d/K, resampled from a stored seed (Sec. 3.3, Supp. A.8
'Partition Replay').  The permutation itself is our reading (a keyed Feistel
permutation with cycle-walking), pinned by exhaustive bijectivity on small
domains, the structural properties of the maps, and uniformity statistics."""
import itertools
import math

import numpy as np
import pytest
from scipy import stats


@pytest.mark.parametrize("d", [1, 2, 3, 5, 16, 17, 255, 1000, 4096, 4097])
@pytest.mark.parametrize("seed", [0, 33, 2**64 - 1])
def test_prp_is_a_bijection(orc, d, seed):
    img = [orc.prp(seed, d, x) for x in range(d)]
    assert sorted(img) == list(range(d))


def test_prp_depends_on_seed(orc):
    d = 1000
    a = [orc.prp(1, d, x) for x in range(d)]
    b = [orc.prp(2, d, x) for x in range(d)]
    assert a != b
    assert a == [orc.prp(1, d, x) for x in range(d)]


@pytest.mark.parametrize("d,K", [(1, 1), (7, 7), (10, 3), (4096, 8), (100003, 8), (65536, 16), (1 << 16, 1)])
def test_permutation_maps_structure(orc, d, K):
    offsets, index = orc.partition(orc.PART_PERMUTATION, d, K, seed=33)
    # offsets are ceil(k d / K): sizes differ by at most one
    assert list(offsets) == [-(-k * d // K) for k in range(K + 1)]
    sizes = np.diff(offsets)
    assert sizes.max() - sizes.min() <= 1
    # disjoint and covering
    assert np.array_equal(np.sort(index), np.arange(d))
    for k in range(K):
        seg = index[offsets[k]:offsets[k + 1]]
        assert np.all(np.diff(seg) > 0)                      # ascending
        for i in seg[:: max(1, seg.size // 50)]:
            assert orc.bucket(33, d, K, int(i)) == k         # every entry is in its bucket


def test_permutation_is_replayable_and_seeded(orc):
    a = orc.partition(orc.PART_PERMUTATION, 5000, 4, seed=33)[1]
    b = orc.partition(orc.PART_PERMUTATION, 5000, 4, seed=33)[1]
    c = orc.partition(orc.PART_PERMUTATION, 5000, 4, seed=34)[1]
    assert np.array_equal(a, b) and not np.array_equal(a, c)


def test_bucket_counts_in_windows_are_binomial(orc):
    """Each index lands in each of K subspaces with probability 1/K, independent of
    its neighbours: counts in windows of W consecutive indices follow
    Binomial(W, 1/K) (chi-square test of the window-count histogram)."""
    d, K, W = 1 << 18, 8, 64
    offsets, index = orc.partition(orc.PART_PERMUTATION, d, K, seed=33)
    lab = np.empty(d, dtype=np.int64)
    for k in range(K):
        lab[index[offsets[k]:offsets[k + 1]]] = k
    counts = (lab.reshape(-1, W) == 0).sum(axis=1)
    obs = np.bincount(counts, minlength=W + 1)
    p = stats.binom.pmf(np.arange(W + 1), W, 1.0 / K)
    exp = p * counts.size
    keep = exp >= 5
    o = np.append(obs[keep], obs[~keep].sum())
    e = np.append(exp[keep], exp[~keep].sum())
    chi2 = ((o - e) ** 2 / e).sum()
    assert stats.chi2.sf(chi2, o.size - 1) > 1e-4


def test_partition_of_tiny_domain_is_near_uniform(orc):
    """Eq. (7) asks for a uniform random equal-size partition: over many seeds,
    each of the C(6,3) choices of the first half of 6 indices (and of the
    C(10,5) for 10 indices) appears about equally often.  (A four-round Feistel
    fails this: p ~ 1e-13.)"""
    for d in (6, 10):
        _tiny_uniformity(orc, d)


def _tiny_uniformity(orc, d):
    K, T = 2, 6000
    seen = {}
    for s in range(T):
        offsets, index = orc.partition(orc.PART_PERMUTATION, d, K, seed=1000 + s)
        key = tuple(index[: offsets[1]])
        seen[key] = seen.get(key, 0) + 1
    assert len(seen) == math.comb(d, d // 2)
    obs = np.array(list(seen.values()), dtype=np.float64)
    chi2 = ((obs - T / obs.size) ** 2 / (T / obs.size)).sum()
    assert stats.chi2.sf(chi2, obs.size - 1) > 1e-4


def test_contiguous_partition(orc):
    offsets, index = orc.partition(orc.PART_CONTIGUOUS, 10, 3)
    assert list(offsets) == [0, 3, 6, 10] and index is None
    b = [0, 4, 4, 10]
    assert list(orc.partition(orc.PART_CONTIGUOUS, 10, 3, bounds=b)[0]) == b
    with pytest.raises(ValueError):
        orc.partition(orc.PART_CONTIGUOUS, 10, 3, bounds=[0, 5, 4, 10])
    with pytest.raises(ValueError):
        orc.partition(orc.PART_CONTIGUOUS, 10, 3, bounds=[0, 5, 6, 9])
    with pytest.raises(ValueError):
        orc.partition(orc.PART_CONTIGUOUS, 10, 11)


@pytest.mark.parametrize("d,chunk,K", [(1000, 8, 3), ((1 << 16) + 5, 64, 4), (100003, 256, 8), (4096, 4096, 1)])
def test_chunk_partition_covers_every_parameter_once(orc, d, chunk, K):
    """Chunk-to-subspace assignment (partition replay at chunk granularity):
    the chunks of all subspaces cover [0, d) exactly once, the short last chunk
    counts only its real parameters, and chunk lists are ascending."""
    offs, lens, chunks = orc.partition_chunks(d, chunk, K, 33)
    n_chunks = -(-d // chunk)
    assert list(offs) == [-(-k * n_chunks // K) for k in range(K + 1)]
    assert lens.sum() == d
    seen = np.zeros(d, dtype=np.int64)
    for k in range(K):
        seg = chunks[offs[k]:offs[k + 1]]
        assert np.all(np.diff(seg) > 0)
        m = orc.expand_chunks(chunks, offs[k], lens[k], chunk)
        assert m.size == lens[k] and np.all(m < d)
        seen[m] += 1
    assert np.all(seen == 1)
    # the chunk assignment is the element partition of the chunk ids
    o2, idx = orc.partition(orc.PART_PERMUTATION, n_chunks, K, seed=33)
    assert np.array_equal(o2, offs) and np.array_equal(idx, chunks)
