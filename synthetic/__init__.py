"""Seeded synthetic inputs and workload shapes, shared by the tests, the smoke
check and the benchmark.

This module holds none of the method's arithmetic: it draws weights and rewards
(numpy's PCG64 on the host, torch's generator on the device), converts fp32 to
bf16 with torch's own rounding, and describes the five workloads.  The noise
that the method itself draws is never produced here; each side (oracle, GPU
library) generates it from its own Philox.

Workloads (weights N(0, 0.02); sigma = 1e-3; alpha = 5e-4 unless stated):

* ``c1`` -- fp32 vector of 1,048,576; 4 equal contiguous subspaces, active 0;
  8 members (seeds 1..8, all +); rewards U[0,1) -> z-score.
* ``c2`` -- bf16, 12 transformer layers (hidden 1024, intermediate 4096):
  150,994,944 params; 16 equal contiguous subspaces; 32 members = 16 seeds x
  (+, -); rewards Bernoulli(0.4) -> centred ranks.
* ``c3`` -- bf16, Qwen3-4B-like decoder (36 layers, hidden 2560, intermediate
  9728, 32 q / 8 kv heads of dim 128, vocab 151,936 tied embedding):
  4,022,468,096 params; 8 contiguous layer-group subspaces (embedding + layers
  0-3, then 4/4/4/5/5/5/5 layers, final norm in the last); 30 members (seeds
  1..30, all +); rewards U[0,1) -> z-score.
* ``c4`` -- the c3 buffer split into 8 subspaces by a seeded permutation
  (seed 33) with int64 index maps; members and rewards as c3.
* ``c5`` -- the c3 buffer with an fp32 master of the active subspace; 16 equal
  contiguous subspaces visited round-robin over 16 iterations; 128 members =
  64 seeds x (+, -) per iteration; rewards = mean of 8 Bernoulli(0.4) draws.
* ``c4c`` -- c4 with a chunk-granular permutation (chunks of 65,536
  parameters, seed 33) instead of an element-level one.
* ``p0`` -- one CoPES step as the paper runs it (Alg. 1, Table S2): the c3
  buffer, K = 4 chunk-granular random subspaces (chunks of 65,536), N = 40
  members split 10 per subspace, rewards U[0,1) standardised jointly (Eq. 12),
  update alpha / N_k (Eq. 13) over all subspaces in one call.
* ``c3h``, ``p0h`` -- c3 and p0 with the weight backup in pinned host memory
  (the backup of Sec. 3.3 kept off the GPU).
* ``c4u`` -- c4 with uint32 index maps (the model has fewer than 2^32
  parameters).

The effective perturbation scale passed to the library is
sigma_k = sigma * sqrt(d / d_k) (the dimension-aware scale of Eq. 11).
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

BF16, F32 = 0, 1
PART_CONTIGUOUS, PART_PERMUTATION, PART_CHUNKED = 0, 1, 2
NORM_Z, NORM_RANK = 0, 1
SCALE_ALPHA_OVER_N_SIGMA, SCALE_ALPHA_OVER_N = 0, 1

INIT_STD = 0.02


# ------------------------------------------------------------------ weights --

def host_weights(n: int, dtype: int, seed: int, std: float = INIT_STD) -> np.ndarray:
    """N(0, std^2) weights on the host: float32, or bf16 bit patterns (uint16)."""
    x = np.random.Generator(np.random.PCG64(seed)).standard_normal(n, dtype=np.float32)
    x *= np.float32(std)
    if dtype == F32:
        return x
    return f32_to_bf16_bits(x)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 through torch (library conversion)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def device_weights(n: int, dtype: int, seed: int, device="cuda", std: float = INIT_STD):
    """N(0, std^2) weights generated on the device by torch's generator, filled in
    chunks so no fp32 temporary of the whole buffer is needed."""
    import torch

    tdt = torch.bfloat16 if dtype == BF16 else torch.float32
    out = torch.empty(n, dtype=tdt, device=device)
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    chunk = 1 << 28
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        tmp = torch.randn(e - s, generator=g, device=device, dtype=torch.float32)
        tmp.mul_(std)
        out[s:e].copy_(tmp)
        del tmp
    return out


# ------------------------------------------------------------------ rewards --

def rewards(kind: str, n: int, seed: int) -> np.ndarray:
    """Synthetic per-member rewards (float32):
    'uniform'        U[0, 1)
    'bernoulli'      Bernoulli(0.4) in {0, 1}
    'mean_bernoulli' mean of 8 Bernoulli(0.4) draws (a batch-mean reward, Eq. 4)
    """
    g = np.random.Generator(np.random.PCG64(seed))
    if kind == "uniform":
        return g.random(n, dtype=np.float32)
    if kind == "bernoulli":
        return (g.random(n) < 0.4).astype(np.float32)
    if kind == "mean_bernoulli":
        return (g.random((n, 8)) < 0.4).mean(axis=1).astype(np.float32)
    raise ValueError(kind)


# ------------------------------------------------------------------ layouts --

def qwen3_4b_like_layers() -> Tuple[int, List[int], int]:
    """(embedding size, per-layer sizes, final-norm size) of the 4.02 G stand-in."""
    hidden, inter, vocab = 2560, 9728, 151936
    q, kv, head = 32, 8, 128
    per_layer = (q * head * hidden + 2 * kv * head * hidden + hidden * q * head
                 + 2 * head + 2 * hidden + 3 * inter * hidden)
    return vocab * hidden, [per_layer] * 36, hidden


def transformer_100m_size() -> int:
    hidden, inter, layers = 1024, 4096, 12
    return layers * (4 * hidden * hidden + 2 * hidden * inter)


def c3_bounds() -> List[int]:
    emb, layers, final = qwen3_4b_like_layers()
    groups = [4, 4, 4, 4, 5, 5, 5, 5]
    bounds, pos, li = [0], 0, 0
    for k, g in enumerate(groups):
        size = sum(layers[li:li + g]) + (emb if k == 0 else 0) + (final if k == len(groups) - 1 else 0)
        li += g
        pos += size
        bounds.append(pos)
    return bounds


def equal_bounds(d: int, K: int) -> List[int]:
    return [(d * k) // K for k in range(K + 1)]


# ---------------------------------------------------------------- workloads --

@dataclasses.dataclass
class Workload:
    name: str
    d: int
    dtype: int
    K: int
    partition_mode: int
    bounds: Optional[List[int]]          # contiguous bounds (None for a permutation)
    partition_seed: int
    seeds: List[int]                      # per member
    signs: List[int]                      # per member
    reward_kind: str
    reward_seed: int
    norm_mode: int
    sigma: float = 1e-3
    alpha: float = 5e-4
    scale_mode: int = SCALE_ALPHA_OVER_N_SIGMA
    master: bool = False
    weight_seed: int = 0
    active: Sequence[int] = (0,)          # subspaces visited, in order
    seed_stride: int = 0                  # member seeds of iteration t are seeds + t * seed_stride
    chunk: int = 0                        # chunk size of a chunk-granular partition
    copes_step: bool = False              # members split across all subspaces, one joint update
    host_backup: bool = False             # weight backup in pinned host memory instead of HBM
    map32: bool = False                   # permutation maps as uint32 (d <= 2^32)
    description: str = ""

    @property
    def n(self) -> int:
        return len(self.seeds)

    def sizes(self) -> List[int]:
        """Nominal subspace sizes (chunked partitions: K equal shares of d)."""
        if self.bounds is not None:
            return [self.bounds[k + 1] - self.bounds[k] for k in range(self.K)]
        return [-(-(k + 1) * self.d // self.K) - (-(-k * self.d // self.K)) for k in range(self.K)]

    def member_subspaces(self) -> List[int]:
        """Subspace of each member for a whole CoPES step (N / K per subspace)."""
        per = self.n // self.K
        return [i // per for i in range(self.n)]

    def sigma_k(self, k: int) -> float:
        """Dimension-aware scale sigma * sqrt(d / d_k) (Eq. 11)."""
        return float(np.float32(self.sigma * math.sqrt(self.d / self.sizes()[k])))

    def member_seeds(self, it: int = 0) -> List[int]:
        return [s + it * self.seed_stride for s in self.seeds]

    def rewards(self, it: int = 0) -> np.ndarray:
        return rewards(self.reward_kind, self.n, self.reward_seed + it)


def _antithetic(seeds: Sequence[int]) -> Tuple[List[int], List[int]]:
    s, g = [], []
    for x in seeds:
        s += [x, x]
        g += [1, -1]
    return s, g


def workload(name: str) -> Workload:
    name = name.lower()
    if name == "c1":
        d = 1 << 20
        return Workload("c1", d, F32, 4, PART_CONTIGUOUS, equal_bounds(d, 4), 0,
                        list(range(1, 9)), [1] * 8, "uniform", 99, NORM_Z,
                        description="fp32 1,048,576; K=4 contiguous; N=8")
    if name == "c2":
        d = transformer_100m_size()
        s, g = _antithetic(range(1, 17))
        return Workload("c2", d, BF16, 16, PART_CONTIGUOUS, equal_bounds(d, 16), 0, s, g,
                        "bernoulli", 99, NORM_RANK, active=tuple(range(16)),
                        description="bf16 150,994,944 (12 x h1024/i4096); K=16 contiguous; N=32 antithetic")
    emb, layers, final = qwen3_4b_like_layers()
    d4 = emb + sum(layers) + final
    if name == "c3":
        return Workload("c3", d4, BF16, 8, PART_CONTIGUOUS, c3_bounds(), 0,
                        list(range(1, 31)), [1] * 30, "uniform", 99, NORM_Z,
                        active=tuple(range(8)),
                        description="bf16 4,022,468,096 Qwen3-4B-like; 8 layer-group subspaces; N=30")
    if name == "c4":
        return Workload("c4", d4, BF16, 8, PART_PERMUTATION, None, 33,
                        list(range(1, 31)), [1] * 30, "uniform", 99, NORM_Z,
                        active=tuple(range(8)),
                        description="bf16 4,022,468,096; 8 permuted subspaces (seed 33); N=30")
    if name == "c5":
        s, g = _antithetic(range(1, 65))
        return Workload("c5", d4, BF16, 16, PART_CONTIGUOUS, equal_bounds(d4, 16), 0, s, g,
                        "mean_bernoulli", 99, NORM_Z, master=True, active=tuple(range(16)),
                        seed_stride=1000,
                        description="bf16 4,022,468,096 + fp32 master; K=16 round-robin; N=128 antithetic")
    if name == "c4c":
        return Workload("c4c", d4, BF16, 8, PART_CHUNKED, None, 33,
                        list(range(1, 31)), [1] * 30, "uniform", 99, NORM_Z,
                        active=tuple(range(8)), chunk=1 << 16,
                        description="bf16 4,022,468,096; 8 chunk-permuted subspaces (chunks of 65,536, seed 33); N=30")
    if name == "p0":
        return Workload("p0", d4, BF16, 4, PART_CHUNKED, None, 33,
                        list(range(1, 41)), [1] * 40, "uniform", 99, NORM_Z,
                        scale_mode=SCALE_ALPHA_OVER_N, active=tuple(range(4)), chunk=1 << 16, copes_step=True,
                        description="bf16 4,022,468,096; one CoPES step: K=4 chunk-permuted subspaces, "
                                    "N=40 (10 per subspace), joint z-score, alpha/N_k")
    if name == "c4u":
        return dataclasses.replace(workload("c4"), name=name, map32=True,
                                   description=workload("c4").description + "; uint32 maps")
    if name in ("c3h", "p0h"):
        base = workload(name[:-1])
        return dataclasses.replace(base, name=name, host_backup=True,
                                   description=base.description + "; weight backup in pinned host memory")
    raise ValueError(name)


WORKLOADS = ("c1", "c2", "c3", "c4", "c5", "c4c", "p0", "c3h", "p0h", "c4u")
