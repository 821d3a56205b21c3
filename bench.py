"""Benchmark of the CoPES parameter-space hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload c3]

One step = one pass of the hot path over every subspace of the workload:
for each active subspace: partition lookup, N x (perturb, restore from the
backup), reward normalisation, seed-replayed update.  The first member's
perturbation also writes the backup; the others perturb the restored weights
in place.  Inputs (weights, rewards) are
resident in HBM before the timed region.  Prints ONE JSON line.

Workloads (synthetic, see synthetic/__init__.py): c3 (default; 4,022,468,096
bf16 params, 8 layer-group subspaces, N = 30), c1, c2, c4 (index-map
subspaces), c5 (fp32 master, 16 iterations of N = 128).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GB/s and % HBM peak for perturb/restore + ES update (params/s) at 4B params"
HBM_PEAK_GBPS = 8000.0                 # MI355X HBM3E
VALU_LANE_OPS_PEAK = 256 * 64 * 2.4e9  # 256 CUs x 64 lanes x 2.4 GHz: one VALU lane-op per lane per clock
# Per-kernel figures measured with rocprofv3 on a 504,654,080-position bf16
# subspace (profiles/c3_subspace_counters.md): VALU instructions per generated
# normal (SQ_INSTS_VALU x 64 lanes / normals) and HBM bytes per position
# (FETCH_SIZE x 2.0 and WRITE_SIZE x 1.0, the factors a plain copy of known
# size reads).  Valid for the kernels as profiled; re-measure after a kernel
# change.
MEASURED = {
    "perturb": {"valu_per_normal": 33.8, "hbm_bytes_first": 6.0, "hbm_bytes_rest": 4.0},
    "perturb_master": {"valu_per_normal": 33.6, "hbm_bytes": 6.0},
    "update": {"valu_per_normal": 31.3, "hbm_bytes": 4.0},
    "update_master": {"valu_per_normal": 31.2, "hbm_bytes": 10.0},
    "restore": {"hbm_bytes": 4.0},
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--workload", default="c3", choices=["c1", "c2", "c3", "c4", "c5", "c4c", "p0", "c3h", "p0h", "c4u"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--fused-restore", action="store_true",
                   help="variant schedule, reported separately from the headline: members after the first perturb "
                        "from the backup (restore and perturbation in one pass) and one restore follows the last")
    p.add_argument("--no-graph", action="store_true",
                   help="skip the HIP-graph timing (by default one step is also captured in a graph and K replays "
                        "of it are timed: graph_ms_per_step)")
    p.add_argument("--kernels-once", action="store_true",
                   help="run each kernel once on one subspace (for counter passes) and exit: c3's 504,654,080-position "
                        "subspace 4, or subspace 0 of a partitioned workload (c4, c4u, c4c)")
    p.add_argument("--cpu-positions", type=int, default=None,
                   help="positions per subspace sample for the oracle baseline (default: 2^31 / members, "
                        "about 10-30 s of host work)")
    return p.parse_args()


class NoTimer:
    """Stands in for KernelTimer inside graph capture (no events)."""

    def run(self, name, fn, positions=0):
        fn()


class KernelTimer:
    """HIP-event timing of each launch of a kernel class on the working stream."""

    def __init__(self, torch):
        self.torch = torch
        self.pending = {}
        self.done = {}

    def run(self, name, fn, positions=0):
        ev0 = self.torch.cuda.Event(enable_timing=True)
        ev1 = self.torch.cuda.Event(enable_timing=True)
        ev0.record()
        fn()
        ev1.record()
        self.pending.setdefault(name, []).append((ev0, ev1, positions))

    def collect(self):
        for name, evs in self.pending.items():
            self.done.setdefault(name, []).extend((a.elapsed_time(b), n) for a, b, n in evs)
        self.pending = {}

    def stats(self, name):
        ts = [t for t, _ in self.done.get(name, [])]
        return (sum(ts) / len(ts) if ts else 0.0), len(ts), sum(ts)

    def rates(self, name):
        """Per-launch positions per second: min, median and 90th percentile."""
        r = sorted(n / (t * 1e-3) for t, n in self.done.get(name, []) if n and t > 0)
        if not r:
            return None
        pick = lambda q: r[min(len(r) - 1, int(q * (len(r) - 1) + 0.5))]
        return {"min": r[0], "p50": pick(0.5), "p90": pick(0.9)}


def build_plan(W, cp, torch):
    """Device buffers of workload W (weights, maps, backup, rewards)."""
    import numpy as np

    import synthetic as S

    dev = torch.device("cuda")
    w = S.device_weights(W.d, W.dtype, W.weight_seed)
    index = ws = None
    if W.partition_mode == S.PART_PERMUTATION:
        index = torch.empty(W.d, dtype=torch.int32 if W.map32 else torch.int64, device=dev)
        ws = torch.empty(cp.cpes_partition_workspace_bytes(cp.PART_PERMUTATION, W.d, W.K), dtype=torch.uint8,
                         device=dev)
    elif W.partition_mode == S.PART_CHUNKED:
        index = torch.empty(-(-W.d // W.chunk), dtype=torch.int64, device=dev)
        ws = torch.empty(cp.cpes_partition_chunks_workspace_bytes(W.d, W.chunk, W.K), dtype=torch.uint8, device=dev)
    maxk = max(W.sizes()) + 2 * W.chunk        # a chunked subspace exceeds d/K by under two chunks
    tdt = torch.bfloat16 if W.dtype == S.BF16 else torch.float32
    aux = torch.empty(maxk, dtype=torch.float32 if W.master else tdt, device=dev)
    n_iter = 1 if W.copes_step else len(W.active)
    rewards = torch.from_numpy(np.stack([W.rewards(t) for t in range(n_iter)])).to(dev)
    rnorm = torch.empty_like(rewards)
    host = torch.empty(maxk, dtype=tdt, pin_memory=True) if W.host_backup else None
    # master workloads restore from a copy of the weights taken at staging
    backup = torch.empty(maxk, dtype=tdt, device=dev) if W.master else None
    return dict(w=w, index=index, ws=ws, aux=aux, rewards=rewards, rnorm=rnorm, host=host, backup=backup)


def random_partition(W, cp, P):
    """Permutation or chunk partition into P (done once, timed on its own):
    list of (offset, length) per subspace."""
    import synthetic as S

    if W.partition_mode == S.PART_PERMUTATION:
        if W.map32:
            offs = cp.cpes_partition32(W.d, W.K, W.partition_seed, P["index"], P["ws"])
        else:
            offs = cp.cpes_partition(cp.PART_PERMUTATION, W.d, W.K, W.partition_seed, index=P["index"],
                                     workspace=P["ws"])
        return [(offs[k], offs[k + 1] - offs[k]) for k in range(W.K)]
    offs, lens = cp.cpes_partition_chunks(W.d, W.chunk, W.K, W.partition_seed, P["index"], P["ws"])
    P["chunk_offsets"], P["chunk_lengths"] = offs, lens
    return [(offs[k], lens[k]) for k in range(W.K)]


def run_step(W, cp, torch, P, timer, cache, fused=False):
    """One pass of the hot path over the workload."""
    import synthetic as S

    if W.partition_mode == S.PART_CONTIGUOUS:
        offs = cp.cpes_partition(cp.PART_CONTIGUOUS, W.d, W.K, bounds=W.bounds)
        parts = [(offs[k], offs[k + 1] - offs[k]) for k in range(W.K)]
    else:
        parts = cache["parts"]
    subs = [cp.subspace(o, n, P["index"], W.chunk) for o, n in parts]
    sigmas = [float(__import__("numpy").float32(W.sigma * (W.d / n) ** 0.5)) for _, n in parts]
    aux_mode = cp.AUX_MASTER if W.master else cp.AUX_SNAPSHOT

    later = cp.AUX_BACKUP if W.partition_mode == S.PART_PERMUTATION else cp.AUX_NONE

    def members(k, seeds, signs):
        s, aux = subs[k], P["aux"][:parts[k][1]]
        n_k = parts[k][1]
        if W.host_backup:
            # Sec. 3.3: the pre-perturbation weights go to host memory once, every
            # member is perturbed in place and restored from there
            host = P["host"][:parts[k][1]]
            timer.run("backup_host", lambda: cp.cpes_backup_to_host(P["w"], s, host), n_k)
            for seed, sign in zip(seeds, signs):
                timer.run("perturb", lambda: cp.cpes_perturb(P["w"], s, sigmas[k], seed, sign), n_k)
                timer.run("restore_host", lambda: cp.cpes_restore_from_host(P["w"], s, host), n_k)
            return
        restore_aux, restore_mode = aux, aux_mode
        if W.master:
            timer.run("stage_master", lambda: cp.cpes_stage_master(P["w"], s, aux), n_k)
            # w is the master rounded to bf16 now, so a bf16 copy of w restores the
            # same bits as the master does, reading 2 bytes per position instead of 4
            restore_aux, restore_mode = P["backup"][:n_k], cp.AUX_SNAPSHOT
            timer.run("backup", lambda: cp.cpes_backup(P["w"], s, restore_aux), n_k)
        for m, (seed, sign) in enumerate(zip(seeds, signs)):
            # the first member takes the backup of the subspace; the others perturb the
            # restored weights in place, or, on an index map, read the (contiguous)
            # backup instead of gathering w (a master source is read by every member)
            mode = aux_mode if (W.master or m == 0) else later
            if fused and m > 0 and not W.master:
                mode = cp.AUX_BACKUP                 # restore of the previous member + perturbation, one pass
            timer.run("perturb", lambda: cp.cpes_perturb(P["w"], s, sigmas[k], seed, sign, aux=aux, aux_mode=mode),
                      n_k)
            # (the perturbed model would be evaluated here)
            if not fused or m == len(seeds) - 1:
                timer.run("restore", lambda: cp.cpes_restore(P["w"], s, aux=restore_aux, aux_mode=restore_mode), n_k)

    if W.copes_step:
        # Alg. 1: every subspace gets N/K members, joint standardisation, one composed update
        seeds, ks = W.member_seeds(0), W.member_subspaces()
        for k in W.active:
            idx = [i for i in range(W.n) if ks[i] == k]
            members(k, [seeds[i] for i in idx], [W.signs[i] for i in idx])
        timer.run("normalize", lambda: cp.cpes_normalize_rewards(P["rewards"][0], P["rnorm"][0], W.norm_mode))
        offsets = [o for o, _ in parts] + [parts[-1][0] + (parts[-1][1] if not W.chunk else 0)]
        if W.chunk:
            offsets = P["chunk_offsets"]
        timer.run("update", lambda: cp.cpes_update_step(
            P["w"], offsets, seeds, W.signs, ks, P["rnorm"][0], W.alpha, sigmas, W.scale_mode,
            index=P["index"], chunk=W.chunk, lengths=[n for _, n in parts] if W.chunk else None),
            sum(n for _, n in parts))
        return
    for t, k in enumerate(W.active):
        seeds = W.member_seeds(t)
        members(k, seeds, W.signs)
        timer.run("normalize", lambda: cp.cpes_normalize_rewards(P["rewards"][t], P["rnorm"][t], W.norm_mode))
        timer.run("update", lambda: cp.cpes_update(P["w"], subs[k], seeds, W.signs, P["rnorm"][t], W.alpha,
                                                   sigmas[k], W.scale_mode,
                                                   master=P["aux"][:parts[k][1]] if W.master else None),
                  parts[k][1])


def bytes_per_position(W, op):
    """Algorithmic HBM bytes per subspace position."""
    import synthetic as S

    e = 2 if W.dtype == S.BF16 else 4
    ix = (4 if W.map32 else 8) if W.partition_mode == S.PART_PERMUTATION else 0
    m = W.n // W.K if W.copes_step else W.n          # members perturbing one subspace
    if op == "perturb" and W.host_backup:
        return 2 * e + ix
    if op in ("backup_host", "restore_host"):
        return e + ix                                  # HBM side; the same e bytes cross the host link
    if op == "perturb":
        # master: read master, write w; else the first member reads w and writes w and the
        # backup, the others read and write w (or, on an index map, read the backup and
        # write w: the same bytes, one map read)
        return (4 + e if W.master else (3 * e + (m - 1) * 2 * e) / m) + ix
    if op == "restore":
        return 2 * e + ix                              # a bit copy from the backup (taken at staging for a master)
    if op == "backup":
        return 2 * e + ix
    if op == "update":
        return (4 + 4 + e if W.master else 2 * e) + ix
    if op == "stage_master":
        return e + 4 + ix
    return 0


def graph_step_ms(W, cp, torch, P, cache, steps, fused=False):
    """One step captured in a HIP graph (torch.cuda.CUDAGraph), then `steps`
    replays timed between synchronisations: the step without per-launch host
    overhead.  The library only enqueues kernels, so the step captures whole."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run_step(W, cp, torch, P, NoTimer(), cache, fused)
    g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    del g
    return ms


def copy_reference(W, torch, P, sizes):
    """The achievable-HBM reference, in the same run: torch's device-to-device
    copy (hipMemcpy) of the largest subspace's weights, median of 5."""
    import statistics

    L = max(sizes[k] for k in W.active)
    src = P["w"][:L]
    dst = P["aux"].view(src.dtype)[:L]
    dst.copy_(src)
    ts = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    nbytes = 2 * L * src.element_size()
    ms = statistics.median(ts)
    return {"GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1), "bytes": nbytes, "ms": round(ms, 4),
            "kind": "torch copy_ (hipMemcpy D2D) of the largest subspace's weights"}


def cpu_baseline(W, positions):
    """The oracle on a bounded sample: the first `positions` positions of every
    active subspace, every member (perturb with backup, restore) and the
    update; extrapolated linearly to the full step."""
    import numpy as np

    import oracle as O
    import synthetic as S

    O.build(force=False)
    sizes = W.sizes()
    t_total, pos_total, full_total = 0.0, 0, 0
    for t, k in enumerate(W.active[:2]):
        n = min(positions, sizes[k])
        w = S.host_weights(n, W.dtype, 1 + k)
        seeds, signs = W.member_seeds(0 if W.copes_step else t), W.signs
        if W.copes_step:                                 # this subspace's members only
            ks = W.member_subspaces()
            seeds = [x for x, kk in zip(seeds, ks) if kk == k]
            signs = [x for x, kk in zip(signs, ks) if kk == k]
        aux = np.empty(n, dtype=np.float32 if W.master else w.dtype)
        mode = O.AUX_MASTER if W.master else O.AUX_SNAPSHOT
        rn, _ = O.normalize(W.rewards(0 if W.copes_step else t), W.norm_mode)
        if W.copes_step:
            rn = rn[[i for i, kk in enumerate(W.member_subspaces()) if kk == k]]
        t0 = time.perf_counter()
        raux, rmode = aux, mode
        if W.master:
            aux[:] = O.stage_master(w, 0, n)
            raux, rmode = w.copy(), O.AUX_SNAPSHOT          # the GPU schedule: restore from a copy of w
        for m, (seed, sign) in enumerate(zip(seeds, signs)):
            pmode = mode if (W.master or m == 0) else (O.AUX_BACKUP if W.partition_mode == S.PART_PERMUTATION
                                                       else O.AUX_NONE)
            O.perturb(w, 0, n, np.float32(W.sigma_k(k)), seed, sign, aux=aux, aux_mode=pmode)
            O.restore(w, 0, n, np.float32(W.sigma_k(k)), seed, sign, aux=raux, aux_mode=rmode)
        O.normalize(W.rewards(0 if W.copes_step else t), W.norm_mode)
        O.update(w, 0, n, seeds, signs, rn, np.float32(W.alpha), np.float32(W.sigma_k(k)), W.scale_mode,
                 master=aux if W.master else None)
        t_total += time.perf_counter() - t0
        pos_total += n
    full_total = sum(sizes[k] for k in W.active)
    step_s = t_total / pos_total * full_total
    return {"value": W.d / step_s, "unit": "params/s", "cores": O.num_threads(), "kind": "oracle",
            "sample": f"first {positions} positions of subspaces {list(W.active[:2])}, all their members "
                      f"(perturb+backup, restore) + normalise + update; {t_total:.1f} s, "
                      f"extrapolated per position to the full step"}


def kernels_once(cp, torch):
    """One warm-up and one measured launch of every kernel on the shape of the
    c3 layer-group subspace 4 (504,654,080 bf16 positions), plus torch's copy
    of the same bytes as the plain-copy reference for traffic counters."""
    import synthetic as S

    W = S.workload("c3")
    L = W.sizes()[4]
    dev = torch.device("cuda")
    w = S.device_weights(L + 64, S.BF16, 0)
    snap = torch.empty(L, dtype=torch.bfloat16, device=dev)
    master = torch.empty(L, dtype=torch.float32, device=dev)
    r = torch.from_numpy(W.rewards(0)).to(dev)
    rn = torch.empty_like(r)
    s = cp.subspace(0, L)
    sigma = W.sigma_k(4)
    seeds64 = [m + 1 for m in range(64) for _ in (0, 1)]
    signs64 = [1, -1] * 64
    r128 = torch.from_numpy(S.rewards("mean_bernoulli", 128, 99)).to(dev)
    rn128 = torch.empty_like(r128)
    for _ in range(2):
        cp.cpes_perturb(w, s, sigma, 3, 1, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_perturb(w, s, sigma, 4, -1)
        cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_normalize_rewards(r, rn, cp.NORM_Z)
        cp.cpes_update(w, s, W.member_seeds(0), W.signs, rn, W.alpha, sigma)
        cp.cpes_stage_master(w, s, master)
        cp.cpes_perturb(w, s, sigma, 3, 1, aux=master, aux_mode=cp.AUX_MASTER)
        cp.cpes_restore(w, s, aux=master, aux_mode=cp.AUX_MASTER)
        cp.cpes_normalize_rewards(r128, rn128, cp.NORM_Z)
        cp.cpes_update(w, s, seeds64, signs64, rn128, W.alpha, sigma, master=master)
        snap.copy_(w[:L])
    torch.cuda.synchronize()
    print(json.dumps({"kernels_once": "c3 subspace 4", "positions": L}), flush=True)


def kernels_once_mapped(W, cp, torch):
    """The same for a partitioned workload (c4, c4u, c4c): partition once, then
    one warm-up and one measured launch of each kernel of subspace 0 (perturb
    taking the backup, perturb from the backup or in place, restore, update),
    plus torch's copy of the subspace's bf16 bytes as the plain-copy reference."""
    import synthetic as S

    P = build_plan(W, cp, torch)
    parts = random_partition(W, cp, P)
    off, L = parts[0]
    s = cp.subspace(off, L, P["index"], W.chunk)
    sigma = float(__import__("numpy").float32(W.sigma * (W.d / L) ** 0.5))
    snap = P["aux"][:L]
    later = cp.AUX_BACKUP if W.partition_mode == S.PART_PERMUTATION else cp.AUX_NONE
    rn = P["rnorm"][0]
    dst = torch.empty(L, dtype=torch.bfloat16, device="cuda")
    for _ in range(2):
        cp.cpes_perturb(P["w"], s, sigma, 3, 1, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_restore(P["w"], s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_perturb(P["w"], s, sigma, 4, -1, aux=snap if later == cp.AUX_BACKUP else None, aux_mode=later)
        cp.cpes_restore(P["w"], s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_normalize_rewards(P["rewards"][0], rn, cp.NORM_Z)
        cp.cpes_update(P["w"], s, W.member_seeds(0), W.signs, rn, W.alpha, sigma)
        dst.copy_(P["w"][:L])
    torch.cuda.synchronize()
    print(json.dumps({"kernels_once": f"{W.name} subspace 0", "positions": L}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the library has no multi-GPU "
              "path: a population would shard across GPUs by member, with a reward all-gather.", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2608_02391_amd as cp
    import synthetic as S

    W = S.workload(args.workload)
    cp.load()
    torch.cuda.set_device(0)
    if args.kernels_once:
        if W.partition_mode == S.PART_CONTIGUOUS:
            kernels_once(cp, torch)
        else:
            kernels_once_mapped(W, cp, torch)
        return
    P = build_plan(W, cp, torch)
    torch.cuda.synchronize()
    cache = {}
    part_ms = None
    if W.partition_mode != S.PART_CONTIGUOUS:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        cache["parts"] = random_partition(W, cp, P)
        e1.record()
        torch.cuda.synchronize()
        part_ms = e0.elapsed_time(e1)
    warm = KernelTimer(torch)
    for _ in range(args.warmup):
        run_step(W, cp, torch, P, warm, cache, args.fused_restore)
    torch.cuda.synchronize()
    timer = KernelTimer(torch)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run_step(W, cp, torch, P, timer, cache, args.fused_restore)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    timer.collect()
    ms_step = elapsed * 1e3 / args.steps
    # host-backup steps query pointer attributes while enqueueing, which stream capture does not allow
    graph_ms = None if (args.no_graph or W.host_backup) else graph_step_ms(W, cp, torch, P, cache, args.steps, args.fused_restore)

    sizes = [n for _, n in cache["parts"]] if "parts" in cache else W.sizes()
    span = sum(sizes[k] for k in W.active)                # subspace positions visited per step
    per_sub_members = W.n // W.K if W.copes_step else W.n
    ops = {}
    for op in ("perturb", "restore", "update", "normalize", "stage_master", "backup", "backup_host", "restore_host"):
        avg_ms, count, tot_ms = timer.stats(op)
        if count == 0:
            continue
        reps = per_sub_members if op in ("perturb", "restore_host") or (op == "restore" and not args.fused_restore) else 1
        per_step = span * reps
        per_launch = per_step / (count / args.steps)     # average positions per launch
        entry = {"launches": count, "avg_ms": round(avg_ms, 4), "ms_per_step": round(tot_ms / args.steps, 3),
                 "positions_per_launch": round(per_launch)}
        b = bytes_per_position(W, op)
        if b:
            gbps = b * per_launch / (avg_ms * 1e-3) / 1e9
            entry["GB/s"] = round(gbps, 1)
            entry["frac_hbm"] = round(gbps / HBM_PEAK_GBPS, 4)
        if op in ("backup_host", "restore_host"):
            e = 2 if W.dtype == S.BF16 else 4
            entry["host_link_GB/s"] = round(e * per_launch / (avg_ms * 1e-3) / 1e9, 1)
        if op in ("perturb", "update"):
            streams = 1
            if op == "update":
                streams = len(set(W.member_seeds(0))) // (W.K if W.copes_step else 1)
            entry["params/s"] = round(per_launch / (avg_ms * 1e-3), 1)
            entry["Gnormal/s"] = round(streams * per_launch / (avg_ms * 1e-3) / 1e9, 2)
        rr = timer.rates(op)
        if rr:                                       # spread over launches, in G positions/s
            entry["per_launch_Gpos/s"] = {q: round(v / 1e9, 2) for q, v in rr.items()}
        ops[op] = entry
    # the dominant GPU kernel; host-link transfers are reported in ops
    dominant = max((o for o in ops if o not in ("normalize", "backup_host", "restore_host")),
                   key=lambda o: ops[o]["ms_per_step"])
    d_entry = ops[dominant]
    gather = W.partition_mode != S.PART_CONTIGUOUS
    key = dominant + ("_master" if W.master and dominant in ("perturb", "update") else "")
    meas = None if (gather or W.dtype != S.BF16 or W.host_backup) else MEASURED.get(key)
    traffic = None
    if meas is not None:
        per_pos = meas.get("hbm_bytes")
        if per_pos is None:                          # first member takes the backup, the rest read it
            per_pos = (meas["hbm_bytes_first"] + (W.n - 1) * meas["hbm_bytes_rest"]) / W.n
        traffic = round(per_pos * d_entry["positions_per_launch"])
    if dominant in ("restore", "stage_master", "backup"):
        roof = {"bound": "hbm", "achieved": d_entry["GB/s"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(d_entry["GB/s"] / HBM_PEAK_GBPS, 4), "traffic": traffic, "kernel": dominant}
    else:
        valu = (meas or {}).get("valu_per_normal", MEASURED["perturb"]["valu_per_normal"])
        peak_gn = VALU_LANE_OPS_PEAK / valu / 1e9
        roof = {"bound": "alu", "achieved": d_entry["Gnormal/s"], "peak": round(peak_gn, 1), "unit": "Gnormal/s",
                "frac": round(d_entry["Gnormal/s"] / peak_gn, 4), "traffic": traffic, "kernel": dominant,
                "valu_insts_per_normal": valu,
                "note": "peak = VALU issue rate (256 CUs x 64 lanes x 2.4 GHz) / VALU instructions per normal"}
    line = {
        "metric": METRIC,
        "value": round(W.d / (ms_step * 1e-3), 1),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{W.name}: {W.description}", "d": W.d, "K": W.K, "members": W.n,
                   "active_subspaces": len(W.active), "weights": "bf16" if W.dtype == S.BF16 else "f32",
                   "noise": "Philox4x32-10 + fp64 Box-Muller, fp32 FMA",
                   "schedule": ("fused restore (variant): one pass restores and perturbs each later member"
                                if args.fused_restore else "perturb and restore per member")},
        "roofline": roof,
        "ops": ops,
    }
    if part_ms is not None:
        line["partition_ms"] = round(part_ms, 3)
    line["copy_reference"] = copy_reference(W, torch, P, sizes)
    if graph_ms is not None:
        line["graph_ms_per_step"] = round(graph_ms, 3)
    if not args.no_cpu_baseline:
        positions = args.cpu_positions or (1 << 31) // W.n
        line["cpu_baseline"] = cpu_baseline(W, positions)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
