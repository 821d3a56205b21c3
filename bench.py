"""Benchmark of the CoPES parameter-space hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload c3] [--extras c1,c2,c4,c5 | --no-extras]

One step = one pass of the hot path over every subspace of the workload:
for each active subspace: partition lookup, N x (perturb, restore from the
backup), reward normalisation, seed-replayed update.  The first member's
perturbation also writes the backup; the others perturb the restored weights
in place (or, on an index map or from an fp32 master, read the backup).
Inputs (weights, rewards) are resident in HBM before the timed region.
Prints ONE JSON line.

The headline (`value`, `config`, `roofline`, `cpu_baseline`) is the
--workload (default c3: 4,022,468,096 bf16 params, 8 layer-group subspaces,
N = 30).  With the default workload the same line also carries short timed
passes of the other four benchmark workloads (`workloads`: c1, c2, c4, c5),
and `ceilings`: reference kernels measured in the same run -- the generator
alone (RNG-only probe), a plain copy and hipMemcpy, and, for index maps, the
plainest gather and scatter through the same map.

Workloads (synthetic, see synthetic/__init__.py): c1, c2, c3, c4 (index-map
subspaces), c5 (fp32 master, 16 iterations of N = 128), and the variants c4c,
p0, c3h, p0h, c4u.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GB/s and % HBM peak for perturb/restore + ES update (params/s) at 4B params"
HBM_PEAK_GBPS = 8000.0                 # MI355X HBM3E
CLOCK_GHZ = 2.4                        # MI355X peak engine clock
VALU_LANE_OPS_PEAK = 256 * 64 * CLOCK_GHZ * 1e9   # 256 CUs x 4 SIMDs x 16 lanes: 64 VALU lane-ops per CU per clock
KERNEL_SOURCES = ("cpes_kernels.hip", "cpes_device.hpp", "cpes_bm_tables.hpp", "cpes_launch.hpp")

# Counter figures of the kernels on a 504,654,080-position bf16 subspace
# (profiles/c3_subspace_counters.md): VALU instructions per generated normal
# (SQ_INSTS_VALU x 64 lanes / normals), HBM bytes per position (FETCH_SIZE x
# 2.0 + WRITE_SIZE x 1.0, the factors a plain copy of known size reads) and
# the engine clock while the kernel ran (GRBM_GUI_ACTIVE / duration).  They
# hold for the kernel sources whose SHA-256 is `sources_sha256`; with other
# sources they are reported as stale and not used.
MEASURED = {
    "sources_sha256": "ae0681dd0564eb9fcb51e3492868b875f1f1a0d3d73926326e37ada394b90709",
    "perturb": {"valu_per_normal": 33.82, "hbm_bytes_first": 6.0, "hbm_bytes_rest": 4.0, "clock_ghz": 2.30},
    "perturb_master": {"valu_per_normal": 34.07, "hbm_bytes": 4.0, "clock_ghz": 2.39},
    "update": {"valu_per_normal": 31.29, "hbm_bytes": 4.0, "clock_ghz": 2.33},
    "update_master": {"valu_per_normal": 31.20, "hbm_bytes": 10.0, "clock_ghz": 2.34},
    "restore": {"hbm_bytes": 4.0},
}

DEFAULT_EXTRAS = ("c1", "c2", "c4", "c5")
# (timed steps at most, warm-up steps, time a HIP graph) of each extra workload
EXTRA_PLAN = {"c1": (20, 2, True), "c2": (5, 1, True), "c3": (3, 1, False), "c4": (2, 1, False),
              "c5": (2, 1, False), "c4c": (2, 1, False), "p0": (3, 1, False), "c4u": (2, 1, False)}


def parse(argv=None):
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--workload", default="c3", choices=["c1", "c2", "c3", "c4", "c5", "c4c", "p0", "c3h", "p0h", "c4u"])
    p.add_argument("--extras", default=None,
                   help="comma-separated workloads timed after the headline (default: c1,c2,c4,c5 with the "
                        "default workload c3, none otherwise)")
    p.add_argument("--no-extras", action="store_true")
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
    a = p.parse_args(argv)
    if a.no_extras:
        a.extras = []
    elif a.extras is None:
        a.extras = list(DEFAULT_EXTRAS) if a.workload == "c3" else []
    else:
        a.extras = [x for x in a.extras.split(",") if x]
    return a


def sources_sha256() -> str:
    """SHA-256 of the kernel sources the counter figures in MEASURED belong to."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_02391_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


class NoTimer:
    """Stands in for KernelTimer inside graph capture (no events)."""

    def run(self, name, fn, positions=0):
        fn()


class KernelTimer:
    """HIP-event timing of each launch of a kernel class on the working stream
    (torch's current stream, which the library launches on)."""

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


def event_ms(torch, fn, reps=5):
    """Median duration of `reps` launches of fn between HIP events, after one warm-up."""
    fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return statistics.median(ts)


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
    # master workloads perturb and restore from a bf16 copy of the weights taken at staging
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
    import numpy as np

    import synthetic as S

    if W.partition_mode == S.PART_CONTIGUOUS:
        offs = cp.cpes_partition(cp.PART_CONTIGUOUS, W.d, W.K, bounds=W.bounds)
        parts = [(offs[k], offs[k + 1] - offs[k]) for k in range(W.K)]
    else:
        parts = cache["parts"]
    # a permutation partition's maps are ascending: bf16 perturbations and
    # restores may then rewrite whole 128-byte lines around the entries
    asc = W.partition_mode == S.PART_PERMUTATION
    subs = [cp.subspace(o, n, P["index"], W.chunk, ascending=asc) for o, n in parts]
    sigmas = [float(np.float32(W.sigma * (W.d / n) ** 0.5)) for _, n in parts]
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
        if W.master:
            # the fp32 master of the active subspace, and a bf16 copy of the weights taken
            # right after staging: w is the master rounded to bf16 then, so the copy's fp32
            # value is the master bit for bit.  Members perturb from the copy (2 bytes per
            # position instead of 4) and restore from it: the same bits as perturbing from
            # and restoring from the master.
            backup = P["backup"][:n_k]
            timer.run("stage_master", lambda: cp.cpes_stage_master(P["w"], s, aux), n_k)
            timer.run("backup", lambda: cp.cpes_backup(P["w"], s, backup), n_k)
            for m, (seed, sign) in enumerate(zip(seeds, signs)):
                timer.run("perturb", lambda: cp.cpes_perturb(P["w"], s, sigmas[k], seed, sign, aux=backup,
                                                             aux_mode=cp.AUX_BACKUP), n_k)
                if not fused or m == len(seeds) - 1:
                    timer.run("restore", lambda: cp.cpes_restore(P["w"], s, aux=backup, aux_mode=cp.AUX_SNAPSHOT),
                              n_k)
            return
        for m, (seed, sign) in enumerate(zip(seeds, signs)):
            # the first member takes the backup of the subspace; the others perturb the
            # restored weights in place, or, on an index map, read the (contiguous)
            # backup instead of gathering w
            mode = cp.AUX_SNAPSHOT if m == 0 else later
            if fused and m > 0:
                mode = cp.AUX_BACKUP                 # restore of the previous member + perturbation, one pass
            timer.run("perturb", lambda: cp.cpes_perturb(P["w"], s, sigmas[k], seed, sign, aux=aux, aux_mode=mode),
                      n_k)
            # (the perturbed model would be evaluated here)
            if not fused or m == len(seeds) - 1:
                timer.run("restore", lambda: cp.cpes_restore(P["w"], s, aux=aux, aux_mode=cp.AUX_SNAPSHOT), n_k)

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
        # master workloads read the bf16 copy and write w; otherwise the first member reads
        # w and writes w and the backup, the others read and write w (or, on an index map,
        # read the backup and write w: the same bytes, one map read)
        return (2 * e if W.master else (3 * e + (m - 1) * 2 * e) / m) + ix
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


# ---------------------------------------------------------- same-run ceilings --

def rng_ceiling(cp, torch):
    """The generator alone (cpes_rng_probe): 2^32 normals, 16 streams per
    position as the update generates them, folded into one word with no other
    memory traffic; median of 9 launches."""
    n = 1 << 32
    sink = torch.empty(1, dtype=torch.int32, device="cuda")
    ms = event_ms(torch, lambda: cp.cpes_rng_probe(7, n, sink), reps=9)
    return {"Gnormal/s": round(n / (ms * 1e-3) / 1e9, 1), "normals": n, "ms": round(ms, 4),
            "kind": "cpes_rng_probe: Philox4x32-10 + Box-Muller, 16 streams per position, no memory traffic"}


def copy_ceilings(cp, torch, src, dst):
    """Achievable HBM copy rates on the given buffers (read + write bytes):
    a plain copy kernel (one 16-byte vector per thread), the same with
    non-temporal accesses, and torch's copy_ (hipMemcpy device to device),
    median of 5 each; the best of them is the copy ceiling."""
    nbytes = src.numel() * src.element_size()
    nbytes -= nbytes % 16
    out = {}
    rate = lambda ms: round(2 * nbytes / (ms * 1e-3) / 1e9, 1)
    for name, nt in (("copy_kernel", False), ("copy_kernel_nt", True)):
        ms = event_ms(torch, lambda: cp.cpes_probe_copy(src, dst, nbytes, nontemporal=nt))
        out[name] = {"GB/s": rate(ms), "ms": round(ms, 4),
                     "kind": "cpes_probe_copy: one 16-byte vector per thread" + (", non-temporal" if nt else "")}
    d = dst.view(src.dtype)[:src.numel()]
    ms = event_ms(torch, lambda: d.copy_(src))
    out["hip_memcpy"] = {"GB/s": rate(ms), "ms": round(ms, 4), "kind": "torch copy_ (hipMemcpy device to device)"}
    out["bytes"] = 2 * nbytes
    out["best_GB/s"] = max(v["GB/s"] for v in out.values() if isinstance(v, dict))
    return out


def map_ceilings(W, cp, torch, P, parts):
    """The plainest gather and scatter of the workload's weights through
    subspace 0's map (one position per thread, nothing else), and torch's own
    index_select / index_copy_ through the same int64 map; median of 3 each,
    in algorithmic GB/s (map entry + weight read + weight written)."""
    import synthetic as S

    off, L = parts[0]
    s = cp.subspace(off, L, P["index"], W.chunk)
    buf = P["aux"][:L]
    e = 2 if W.dtype == S.BF16 else 4
    ix = 4 if W.map32 else 8
    rate = lambda ms: round((2 * e + ix) * L / (ms * 1e-3) / 1e9, 1)
    out = {"positions": L, "bytes_per_position": 2 * e + ix}
    backup = torch.empty_like(buf)
    cp.cpes_backup(P["w"], s, backup)                  # scatters below write back the same values
    ms = event_ms(torch, lambda: cp.cpes_probe_map_copy(P["w"], s, buf, 0), reps=3)
    out["plain_gather"] = {"GB/s": rate(ms), "ms": round(ms, 4)}
    ms = event_ms(torch, lambda: cp.cpes_probe_map_copy(P["w"], s, backup, 1), reps=3)
    out["plain_scatter"] = {"GB/s": rate(ms), "ms": round(ms, 4)}
    if not W.map32:
        idx = P["index"][off:off + L]
        ms = event_ms(torch, lambda: torch.index_select(P["w"], 0, idx, out=buf), reps=3)
        out["torch_index_select"] = {"GB/s": rate(ms), "ms": round(ms, 4)}
        ms = event_ms(torch, lambda: P["w"].index_copy_(0, idx, backup), reps=3)
        out["torch_index_copy"] = {"GB/s": rate(ms), "ms": round(ms, 4)}
    torch.cuda.synchronize()
    del backup
    return out


# ------------------------------------------------------------------ measure --

def measure(W, cp, torch, steps, warmup, graph, fused=False):
    """Build W's buffers, partition, warm up, time `steps` steps; returns the
    per-kernel timings and the buffers."""
    import synthetic as S

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
    for _ in range(warmup):
        run_step(W, cp, torch, P, warm, cache, fused)
    torch.cuda.synchronize()
    timer = KernelTimer(torch)
    t0 = time.perf_counter()
    for _ in range(steps):
        run_step(W, cp, torch, P, timer, cache, fused)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    timer.collect()
    # host-backup steps query pointer attributes while enqueueing, which stream capture does not allow
    graph_ms = graph_step_ms(W, cp, torch, P, cache, steps, fused) if (graph and not W.host_backup) else None
    sizes = [n for _, n in cache["parts"]] if "parts" in cache else W.sizes()
    parts = cache.get("parts") or [(W.bounds[k], sizes[k]) for k in range(W.K)]
    return dict(P=P, timer=timer, ms_step=elapsed * 1e3 / steps, part_ms=part_ms, graph_ms=graph_ms,
                sizes=sizes, parts=parts, steps=steps, warmup=warmup)


def op_table(W, M, fused, ceil):
    """Per kernel class: launches, average ms, algorithmic GB/s and fractions."""
    import synthetic as S

    timer, steps = M["timer"], M["steps"]
    span = sum(M["sizes"][k] for k in W.active)             # subspace positions visited per step
    per_sub_members = W.n // W.K if W.copes_step else W.n
    rng = (ceil or {}).get("rng_probe", {}).get("Gnormal/s")
    copy_best = (ceil or {}).get("copy", {}).get("best_GB/s")
    ops = {}
    for op in ("perturb", "restore", "update", "normalize", "stage_master", "backup", "backup_host", "restore_host"):
        avg_ms, count, tot_ms = timer.stats(op)
        if count == 0:
            continue
        reps = per_sub_members if op in ("perturb", "restore_host") or (op == "restore" and not fused) else 1
        per_launch = span * reps / (count / steps)           # average positions per launch
        entry = {"launches": count, "avg_ms": round(avg_ms, 4), "ms_per_step": round(tot_ms / steps, 3),
                 "positions_per_launch": round(per_launch)}
        b = bytes_per_position(W, op)
        if b:
            gbps = b * per_launch / (avg_ms * 1e-3) / 1e9
            entry["GB/s"] = round(gbps, 1)
            entry["frac_hbm"] = round(gbps / HBM_PEAK_GBPS, 4)
            if copy_best and op in ("restore", "backup", "stage_master") and W.partition_mode != S.PART_PERMUTATION:
                entry["frac_copy_ceiling"] = round(gbps / copy_best, 4)
        if op in ("backup_host", "restore_host"):
            e = 2 if W.dtype == S.BF16 else 4
            entry["host_link_GB/s"] = round(e * per_launch / (avg_ms * 1e-3) / 1e9, 1)
        if op in ("perturb", "update"):
            streams = 1
            if op == "update":
                streams = len(set(W.member_seeds(0))) // (W.K if W.copes_step else 1)
            gn = streams * per_launch / (avg_ms * 1e-3) / 1e9
            entry["params/s"] = round(per_launch / (avg_ms * 1e-3), 1)
            entry["Gnormal/s"] = round(gn, 2)
            if rng:
                entry["frac_rng_probe"] = round(gn / rng, 4)
        rr = timer.rates(op)
        if rr:                                       # spread over launches, in G positions/s
            entry["per_launch_Gpos/s"] = {q: round(v / 1e9, 2) for q, v in rr.items()}
        ops[op] = entry
    return ops


def roofline(W, ops, ceil, sha_ok):
    """The bench line's roofline object for the workload's dominant kernel."""
    import synthetic as S

    dominant = max((o for o in ops if o not in ("normalize", "backup_host", "restore_host")),
                   key=lambda o: ops[o]["ms_per_step"])
    d = ops[dominant]
    mapped = W.partition_mode == S.PART_PERMUTATION
    key = dominant + ("_master" if W.master and dominant in ("perturb", "update") else "")
    meas = MEASURED.get(key) if (sha_ok and W.dtype == S.BF16 and not mapped and not W.host_backup
                                 and W.partition_mode == S.PART_CONTIGUOUS) else None
    traffic = None
    if meas is not None and (meas.get("hbm_bytes") or meas.get("hbm_bytes_first")):
        per_pos = meas.get("hbm_bytes")
        if per_pos is None:                          # first member takes the backup, the rest read it
            per_pos = (meas["hbm_bytes_first"] + (W.n - 1) * meas["hbm_bytes_rest"]) / W.n
        traffic = round(per_pos * d["positions_per_launch"])
    rng = (ceil or {}).get("rng_probe", {}).get("Gnormal/s")
    if dominant in ("perturb", "update") and not mapped:
        roof = {"bound": "alu", "achieved": d["Gnormal/s"], "unit": "Gnormal/s", "traffic": traffic,
                "kernel": dominant, "frac_hbm": d.get("frac_hbm")}
        if meas and meas.get("valu_per_normal"):
            valu = meas["valu_per_normal"]
            peak = VALU_LANE_OPS_PEAK / valu / 1e9
            roof.update(peak=round(peak, 1), frac=round(d["Gnormal/s"] / peak, 4), valu_insts_per_normal=valu,
                        peak_kind="VALU issue rate (256 CUs x 64 lanes x 2.4 GHz) / VALU instructions per normal "
                                  "of this build (counters)")
            if meas.get("clock_ghz"):
                roof["counter_clock_ghz"] = meas["clock_ghz"]
                roof["frac_at_counter_clock"] = round(d["Gnormal/s"] / (peak * meas["clock_ghz"] / CLOCK_GHZ), 4)
        elif rng:
            roof.update(peak=rng, frac=round(d["Gnormal/s"] / rng, 4),
                        peak_kind="RNG-only probe of this run (counter figures stale for these kernel sources)")
        if rng:
            roof["rng_probe_Gnormal/s"] = rng
            roof["frac_rng_probe"] = round(d["Gnormal/s"] / rng, 4)
        return roof
    roof = {"bound": "hbm", "achieved": d["GB/s"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(d["GB/s"] / HBM_PEAK_GBPS, 4), "traffic": traffic, "kernel": dominant}
    copy_best = (ceil or {}).get("copy", {}).get("best_GB/s")
    if copy_best and not mapped:
        roof["copy_ceiling_GB/s"] = copy_best
        roof["frac_copy_ceiling"] = round(d["GB/s"] / copy_best, 4)
    return roof


def summary(W, M, ops, roof, map_ceil=None):
    """The compact record of one extra workload."""
    out = {"workload": f"{W.name}: {W.description}", "ms_per_step": round(M["ms_step"], 3),
           "params/s": round(W.d / (M["ms_step"] * 1e-3), 1), "steps": M["steps"], "warmup": M["warmup"],
           "roofline": roof, "ops": ops}
    if M["part_ms"] is not None:
        out["partition_ms"] = round(M["part_ms"], 3)
    if M["graph_ms"] is not None:
        out["graph_ms_per_step"] = round(M["graph_ms"], 3)
    if map_ceil:
        out["map_ceilings"] = map_ceil
        for op, probe in (("perturb", "plain_scatter"), ("restore", "plain_scatter"), ("update", "plain_scatter")):
            if op in ops and "GB/s" in ops[op]:
                ops[op]["frac_plain_scatter"] = round(ops[op]["GB/s"] / map_ceil[probe]["GB/s"], 4)
    return out


def cpu_baseline(W, positions):
    """The oracle on a bounded sample: the first `positions` positions of every
    active subspace, every member (perturb with backup, restore) and the
    update; extrapolated linearly to the full step."""
    import numpy as np

    import oracle as O
    import synthetic as S

    O.build(force=False)
    sizes = W.sizes()
    t_total, pos_total = 0.0, 0
    for t, k in enumerate(W.active[:2]):
        n = min(positions, sizes[k])
        w = S.host_weights(n, W.dtype, 1 + k)
        seeds, signs = W.member_seeds(0 if W.copes_step else t), W.signs
        if W.copes_step:                                 # this subspace's members only
            ks = W.member_subspaces()
            seeds = [x for x, kk in zip(seeds, ks) if kk == k]
            signs = [x for x, kk in zip(signs, ks) if kk == k]
        aux = np.empty(n, dtype=np.float32 if W.master else w.dtype)
        rn, _ = O.normalize(W.rewards(0 if W.copes_step else t), W.norm_mode)
        if W.copes_step:
            rn = rn[[i for i, kk in enumerate(W.member_subspaces()) if kk == k]]
        t0 = time.perf_counter()
        if W.master:
            aux[:] = O.stage_master(w, 0, n)
            backup = w.copy()                            # the GPU schedule: perturb and restore from a copy of w
        for m, (seed, sign) in enumerate(zip(seeds, signs)):
            if W.master:
                O.perturb(w, 0, n, np.float32(W.sigma_k(k)), seed, sign, aux=backup, aux_mode=O.AUX_BACKUP)
                O.restore(w, 0, n, np.float32(W.sigma_k(k)), seed, sign, aux=backup, aux_mode=O.AUX_SNAPSHOT)
                continue
            pmode = O.AUX_SNAPSHOT if m == 0 else (O.AUX_BACKUP if W.partition_mode == S.PART_PERMUTATION
                                                   else O.AUX_NONE)
            O.perturb(w, 0, n, np.float32(W.sigma_k(k)), seed, sign, aux=aux, aux_mode=pmode)
            O.restore(w, 0, n, np.float32(W.sigma_k(k)), seed, sign, aux=aux, aux_mode=O.AUX_SNAPSHOT)
        O.normalize(W.rewards(0 if W.copes_step else t), W.norm_mode)
        O.update(w, 0, n, seeds, signs, rn, np.float32(W.alpha), np.float32(W.sigma_k(k)), W.scale_mode,
                 master=aux if W.master else None)
        t_total += time.perf_counter() - t0
        pos_total += n
    full_total = sum(sizes[k] for k in W.active)
    step_s = t_total / pos_total * full_total
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": W.d / step_s, "unit": "params/s", "cores": O.num_threads(), "kind": "oracle",
            "host_cpus": len(os.sched_getaffinity(0)), "cpu_model": model,
            "sample": f"first {positions} positions of subspaces {list(W.active[:2])}, all their members "
                      f"(perturb+backup, restore) + normalise + update; {t_total:.1f} s on {O.num_threads()} "
                      f"OpenMP threads, extrapolated per position to the full step"}


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
    sink = torch.empty(1, dtype=torch.int32, device=dev)
    for _ in range(2):
        cp.cpes_perturb(w, s, sigma, 3, 1, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_perturb(w, s, sigma, 4, -1)
        cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_normalize_rewards(r, rn, cp.NORM_Z)
        cp.cpes_update(w, s, W.member_seeds(0), W.signs, rn, W.alpha, sigma)
        cp.cpes_stage_master(w, s, master)
        cp.cpes_backup(w, s, snap)
        cp.cpes_perturb(w, s, sigma, 3, 1, aux=snap, aux_mode=cp.AUX_BACKUP)
        cp.cpes_restore(w, s, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        cp.cpes_normalize_rewards(r128, rn128, cp.NORM_Z)
        cp.cpes_update(w, s, seeds64, signs64, rn128, W.alpha, sigma, master=master)
        cp.cpes_rng_probe(7, L, sink)
        cp.cpes_probe_copy(w, snap, 2 * L)
        snap.copy_(w[:L])
    torch.cuda.synchronize()
    print(json.dumps({"kernels_once": "c3 subspace 4", "positions": L}), flush=True)


def kernels_once_mapped(W, cp, torch):
    """The same for a partitioned workload (c4, c4u, c4c): partition once, then
    one warm-up and one measured launch of each kernel of subspace 0 (perturb
    taking the backup, perturb from the backup or in place, restore, update,
    and for element maps the plain gather and scatter probes and, through the
    map left unflagged, the entry-by-entry perturbation from the backup and
    restore), plus torch's copy of the subspace's bf16 bytes as the plain-copy
    reference."""
    import synthetic as S

    P = build_plan(W, cp, torch)
    parts = random_partition(W, cp, P)
    off, L = parts[0]
    s = cp.subspace(off, L, P["index"], W.chunk, ascending=W.partition_mode == S.PART_PERMUTATION)
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
        if W.partition_mode == S.PART_PERMUTATION:
            cp.cpes_probe_map_copy(P["w"], s, dst, 0)
            cp.cpes_probe_map_copy(P["w"], s, dst, 1)
            entries = cp.subspace(off, L, P["index"], W.chunk)
            cp.cpes_perturb(P["w"], entries, sigma, 4, -1, aux=snap, aux_mode=cp.AUX_BACKUP)
            cp.cpes_restore(P["w"], entries, aux=snap, aux_mode=cp.AUX_SNAPSHOT)
        dst.copy_(P["w"][:L])
    torch.cuda.synchronize()
    print(json.dumps({"kernels_once": f"{W.name} subspace 0", "positions": L}), flush=True)


def release(torch, M):
    M["P"].clear()
    M.clear()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


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
    sha = sources_sha256()
    sha_ok = sha == MEASURED["sources_sha256"]

    M = measure(W, cp, torch, args.steps, args.warmup, not args.no_graph, args.fused_restore)
    # the ceilings are measured right after the timed steps, with the GPU as warm as it was for them
    ceil = {"rng_probe": rng_ceiling(cp, torch)}
    L = max(M["sizes"][k] for k in W.active)
    ceil["copy"] = copy_ceilings(cp, torch, M["P"]["w"][:L], M["P"]["aux"])
    ops = op_table(W, M, args.fused_restore, ceil)
    roof = roofline(W, ops, ceil, sha_ok)
    map_ceil = map_ceilings(W, cp, torch, M["P"], M["parts"]) if W.partition_mode == S.PART_PERMUTATION else None
    line = {
        "metric": METRIC,
        "value": round(W.d / (M["ms_step"] * 1e-3), 1),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(M["ms_step"], 3),
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
        "counter_figures": {"sources_sha256": sha[:16], "current": sha_ok},
    }
    if M["part_ms"] is not None:
        line["partition_ms"] = round(M["part_ms"], 3)
    if M["graph_ms"] is not None:
        line["graph_ms_per_step"] = round(M["graph_ms"], 3)
    if map_ceil:
        line["map_ceilings"] = map_ceil
    release(torch, M)

    extras = {}
    for name in args.extras:
        if name == W.name:
            continue
        X = S.workload(name)
        max_steps, warm, graph = EXTRA_PLAN.get(name, (2, 1, False))
        MX = measure(X, cp, torch, min(args.steps, max_steps), warm, graph and not args.no_graph, args.fused_restore)
        ox = op_table(X, MX, args.fused_restore, ceil)
        rx = roofline(X, ox, ceil, sha_ok)
        mc = map_ceilings(X, cp, torch, MX["P"], MX["parts"]) if X.partition_mode == S.PART_PERMUTATION else None
        extras[name] = summary(X, MX, ox, rx, mc)
        release(torch, MX)
    line["ceilings"] = ceil
    if extras:
        line["workloads"] = extras
    if not args.no_cpu_baseline:
        positions = args.cpu_positions or (1 << 31) // W.n
        line["cpu_baseline"] = cpu_baseline(W, positions)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
