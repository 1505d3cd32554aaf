"""Benchmark: batched KV-tier configuration evaluation on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload full]

One step is the whole hot path over one synthetic trace resident in HBM:
kv_trace_load (canonicalise), kv_eval_configs (every configuration of the
workload: stack-distance pass + closed-form LRU records, FIFO/LFU replays,
objectives) and kv_pareto (one front over all configurations, then one per
policy segment).  The metric is block accesses x configurations per second
of that step.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "config-evaluations/sec (block accesses × configs / s) + % HBM peak"
HBM_PEAK_GBS = 8000.0

WORKLOAD_TEXT = {
    "full": "full-scale sweep: 1M requests (chat 40% / tenant 30% / long-context 30%) over "
            "2 h, 128 KiB granules with 64-token blocks weighing 4; 10,000 LRU grid configs "
            "(25x20x20) + 1,000 FIFO/LFU replay configs",
    "chat": "multi-turn chat: 20,000 sessions over 2 h; 512 LRU configs (8x8x8 grid)",
    "tenant": "mixed tenant: 8 groups, 100,000 requests; 1,000 partitioned configs with "
              "per-group LRU/FIFO/LFU",
    "longctx": "long-context: 100,000 requests over 2,000 documents, 512 KiB blocks; 2,048 "
               "LRU write-back-demotion configs",
    "tiny": "tiny: 2,000 requests, Poisson 20/s; 64 LRU configs",
}

# Algorithmic bytes per unit of work of each stage (what the method must move
# at minimum; see the design notes): per access for trace-wide passes, per
# (job, access) for the replay.
ALGO_BYTES = {
    "load_sort": 18.0,        # read hash 8 + weight 1 + group 1, write prev 4 + next 4
    "stack_local": 5.0,       # read key 4 + weight 1 once for every LRU capacity
    "replay_lfu": 5.0,        # read block id 4 + weight 1 per LFU job-access
    "replay_fifo": 5.0,       # read block id 4 + weight 1 per FIFO job-access
    "ttl_curves": 14.0,       # read link 4 + request 4 + weight 1 + group 1, gather the
                              # previous access's request 4
}
# TTL curves of the disk tier: t = 0 and 63 values from 0.25 s to the 2 h span
TTL_GRID = [0.0] + [float(x) for x in np.geomspace(0.25, 7200.0, 63)]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="full", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--cpu-baseline-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the TTL-curve, adaptive-search, group-TTL and prefix-reuse "
                         "measurements and the other workloads' lines that follow the "
                         "timed steps")
    ap.add_argument("--ttl-extra-only", action="store_true",
                    help="of the measurements after the timed steps, only the TTL curves")
    ap.add_argument("--exclusive-extra-only", action="store_true",
                    help="of the measurements after the timed steps, only the exclusive "
                         "hierarchies replayed access by access")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="first run one plain device-to-device copy of BYTES (a reference "
                         "for hardware byte counters)")
    return ap.parse_args()


# Groups of library stages reported together, with the method's minimum bytes
# per access (A1: read hash 8 + weight 1 + group 1, write both links 8; A3:
# read each key 4 and weight 1 once for every LRU capacity).
STAGE_GROUPS = {
    "load": (("load_validate", "load_sort", "load_links"), 18.0),
    "stack_pass": (("stack_matrix", "stack_local", "stack_assemble", "stack_final"), 5.0),
}


def stage_table(workload, timing, steps, n, jobs_accesses, jobs_count):
    """Per hot stage: average launch time and algorithmic bytes per launch
    against the HBM peak (the dominant stage is reported on its own)."""
    out = {}

    def put(name, ms_step, calls_step, algo_launch, extra=None):
        if not calls_step or ms_step <= 0:
            return
        avg = ms_step / calls_step
        ach = algo_launch / (avg / 1000.0) / 1e9
        rec = {"avg_launch_ms": round(avg, 3), "launches_per_step": calls_step,
               "algorithmic_bytes_per_launch": algo_launch, "achieved": ach,
               "unit": "GB/s", "frac": ach / HBM_PEAK_GBS, "traffic": traffic_for(workload, name)}
        rec.update(extra or {})
        out[name] = rec

    for g, (names, per) in STAGE_GROUPS.items():
        ms = sum(timing[k][1] for k in names if k in timing) / steps
        # one launch of the group per step (the load and the stack pass run once)
        put(g, ms, 1, per * n, {"stages": list(names)})
    for k in ("stack_local", "replay_fifo", "replay_lfu"):
        if k in timing and timing[k][0]:
            calls = timing[k][0] / steps
            put(k, timing[k][1] / steps, calls,
                ALGO_BYTES[k] * stage_units(k, n, jobs_accesses) / calls,
                {"workgroups": jobs_count.get(k[7:])} if k.startswith("replay_") else None)
    if "replay_combine" in timing and timing["replay_combine"][0]:
        calls = timing["replay_combine"][0] / steps
        # each launch reads the hit bits of its jobs and 8 weight bit-planes once
        jobs = sum(jobs_count.values())
        put("replay_combine", timing["replay_combine"][1] / steps, calls,
            (jobs + 8 * calls) * n / 8.0 / calls)
    return out


def stage_units(stage, n, jobs_accesses):
    if stage.startswith("replay_") and stage[7:] in jobs_accesses:
        return jobs_accesses[stage[7:]]
    return n


def replay_job_accesses(cfgs, stats, n):
    """Accesses walked by replay jobs per step (closed-form jobs excluded),
    per policy: {"fifo": ..., "lfu": ...}, and the number of such jobs (one
    workgroup each) per policy."""
    import tracegen as tg
    G = stats.n_groups
    jobs = set()
    for c in range(cfgs.n):
        part = bool(cfgs.partitioned[c]) and G > 1
        for g in range(G if cfgs.partitioned[c] else 1):
            pol = int(cfgs.policy[c, g])
            if pol in (tg.POLICY_LRU, tg.POLICY_LEAF):
                continue
            for k in range(3):
                x = int(cfgs.cap_group[c, k, g] if cfgs.partitioned[c] else cfgs.cap[c, k])
                dw = stats.u_w_g[g] if part else stats.distinct_w
                if x and x < dw:
                    jobs.add((part, g if part else -1, pol, x))
    total, count = {"fifo": 0, "lfu": 0}, {"fifo": 0, "lfu": 0}
    for (part, g, pol, _) in jobs:
        key = "lfu" if pol == tg.POLICY_LFU else "fifo"
        total[key] += stats.n_g[g] if part else n
        count[key] += 1
    return total, count


def dominant_kernel(timing, steps):
    """Stage that takes the most device time; per-launch average in ms."""
    best, best_ms = None, -1.0
    for name, (calls, ms) in timing.items():
        if calls and ms > best_ms:
            best, best_ms = name, ms
    calls = timing[best][0]
    return best, best_ms / max(calls, 1), calls


def traffic_for(workload, stage):
    """HBM bytes per launch of a stage on a workload, from committed
    rocprofv3 counter runs, while the kernel sources are unchanged."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(workload, {}).get(stage)
    if not rec or source_sha(rec["source"]) != rec.get("source_sha"):
        return None
    return rec["bytes_per_launch"]


def source_sha(files):
    """Hash of the kernel sources a counter record was taken with (one file
    or a list of files, concatenated)."""
    h = hashlib.sha256()
    for f in [files] if isinstance(files, str) else files:
        h.update(open(os.path.join(ROOT, "paper_2603_08739_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


# What bounds a kernel that is not bound by HBM: its VALU instruction count
# per launch (from the committed rocprofv3 SQ counter run, valid while the
# kernel source is unchanged) against the issue rate of the compute units it
# occupies (one wave64 VALU instruction per cycle per compute unit: 4 SIMDs,
# 4 cycles each, at 2.4 GHz).
CU_COUNT, CLOCK_HZ = 256, 2.4e9


def limiter_for(workload, kernel, avg_ms, workgroups):
    path = os.path.join(ROOT, "profiles", "valu.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(workload, {}).get(kernel)
    if not rec:
        return None
    if source_sha(rec["source"]) != rec.get("source_sha"):
        return None
    rate = rec["valu_insts_per_launch"] / (avg_ms / 1000.0)
    cus = min(workgroups or CU_COUNT, CU_COUNT)
    return {"bound": "valu issue and dependent latency of one workgroup per job",
            "valu_wave_insts_per_launch": rec["valu_insts_per_launch"],
            "achieved": rate, "unit": "wave64 VALU instructions/s",
            "peak_occupied_cus": cus * CLOCK_HZ, "frac_occupied_cus": rate / (cus * CLOCK_HZ),
            "peak_chip": CU_COUNT * CLOCK_HZ, "frac_chip": rate / (CU_COUNT * CLOCK_HZ),
            "occupied_cus": cus}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(rec, cfgs, budget_s):
    """The oracle on a bounded sample: a prefix of the trace x a config sample."""
    from oracle import oracle as O
    O.build(force=False)
    rng = np.random.default_rng(11)
    pick = np.sort(rng.choice(cfgs.n, size=min(16, cfgs.n), replace=False))
    sample = cfgs.subset(pick)
    threads = O.default_threads()
    n_req = 2000
    t = rec.to_trace(max_requests=n_req)
    t0 = time.time()
    O.replay(t, sample, threads)
    dt = time.time() - t0
    # grow the prefix (aiming at the budget) until one run takes at least
    # half of it
    while dt < budget_s / 2 and n_req < rec.len0.shape[0]:
        n_req = min(rec.len0.shape[0], int(n_req * min(8.0, max(1.5, budget_s / max(dt, 1e-3)))))
        t = rec.to_trace(max_requests=n_req)
        t0 = time.time()
        O.replay(t, sample, threads)
        dt = time.time() - t0
    value = t.n * sample.n / dt
    # one core on the same configurations over a shorter prefix (a quarter
    # of the budget at the all-core rate's per-core share)
    n1 = max(200, int(n_req * min(1.0, 0.25 * budget_s / max(dt * threads, 1e-3))))
    t1s = rec.to_trace(max_requests=n1)
    t0 = time.time()
    O.replay(t1s, sample, 1)
    dt1 = time.time() - t0
    return {"value": value, "unit": "block-accesses×configs/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "value_one_core": t1s.n * sample.n / dt1,
            "sample": f"first {n_req} requests ({t.n} accesses) x {sample.n} configs sampled "
                      f"from the workload's batch (seed 11), literal replay, {dt:.1f} s on "
                      f"{threads} threads; one core: first {n1} requests ({t1s.n} accesses), "
                      f"{dt1:.1f} s"}


def _search_vs_grid(h, rec, G, model, P, hbm, second, d_rng, t_rng, res, grid_d, grid_t,
                    ttl_unit=1.0):
    """One Alg. 1 run against the full grid: evaluations, rounds, wall time,
    fronts and the hypervolume ratio under one reference point strictly
    worse than every configuration either evaluated."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ex = P.Explorer(h, G, model, hbm=hbm, second=second, ttl_unit=ttl_unit)
    rounds = ex.run(d_rng, t_rng, 0.02, 0.05, 0.02, res=res)
    flags = ex.front()
    wall = time.perf_counter() - t0
    grid_pts = [(d, t) for d in grid_d for t in grid_t]
    gx = P.Explorer(h, G, model, hbm=hbm, second=second, ttl_unit=ttl_unit)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    gx.obj = gx.evaluate(grid_pts)
    gflags = gx.front()
    gwall = time.perf_counter() - t1
    a, b = P.minimised(ex.obj), P.minimised(gx.obj)
    ref = np.maximum(a.max(axis=0), b.max(axis=0))
    ref = ref + 0.01 * np.abs(ref) + 1e-12
    hv_s, hv_g = P.hypervolume(a[flags], ref), P.hypervolume(b[gflags], ref)
    return {"evaluations": len(ex.points), "rounds": rounds, "wall_s": wall,
            "front": int(flags.sum()), "grid_points": len(grid_pts),
            "grid_front": int(gflags.sum()), "grid_wall_s": gwall,
            "hypervolume_vs_grid": hv_s / hv_g if hv_g > 0 else None}


def adaptive_search(h, rec, G, model, torch, K):
    """Alg. 1 (Section 4.2) at 40 GiB HBM, LRU inclusive, against full grids
    of 17 x 31 = 527 configurations:
    * the paper's ablation (Section 5.3.1): DRAM x disk capacity, grid DRAM
      0-4096 GiB step 256 x disk 0-3600 GiB step 120; the search starts from
      DRAM 0-2048 step 512 x disk 0-2400 step 600 and refines down to the
      grid's steps;
    * the planner's dimensions (Section 4.1): DRAM x disk TTL (an unbounded
      TTL tier), grid TTL 0-3600 s step 120, start 0-2400 s step 600."""
    from paper_2603_08739_amd import search as P
    gran = lambda nbytes: int(nbytes // rec.granule_bytes)
    gib = 1 << 30
    hbm = gran(40 * gib)
    d_rng = (0, gran(2048 * gib), gran(512 * gib))
    grid_d = [gran(256 * gib) * i for i in range(17)]
    out = {}
    cap = _search_vs_grid(h, rec, G, model, P, hbm, "disk", d_rng,
                          (0, gran(2400 * gib), gran(600 * gib)),
                          (gran(256 * gib), gran(120 * gib)), grid_d,
                          [gran(120 * gib) * j for j in range(31)])
    cap["algorithm"] = "Alg. 1 over (DRAM, disk capacity) at 40 GiB HBM, LRU inclusive"
    out["dram_x_disk"] = cap
    ttl = _search_vs_grid(h, rec, G, model, P, hbm, "ttl", d_rng, (0, 20, 5),
                          (gran(256 * gib), 1), grid_d, list(range(31)), ttl_unit=120.0)
    ttl["algorithm"] = ("Alg. 1 over (DRAM, disk TTL) at 40 GiB HBM, LRU inclusive, "
                        "unbounded TTL disk tier, TTL step 120 s")
    out["dram_x_ttl"] = ttl
    for k, v in out.items():
        print(f"[bench] adaptive search {k}: {v['evaluations']} evaluations in {v['rounds']} "
              f"rounds ({v['wall_s']:.2f} s) against {v['grid_points']}; hypervolume "
              f"{v['hypervolume_vs_grid']:.4f} of the grid's", file=sys.stderr, flush=True)
    return out


def group_ttl(dev, rec, torch, K, k=7, budget_fracs=(0.02, 0.05, 0.25)):
    """Alg. 2 on the workload: requests grouped by the k most frequent prefix
    subtrees plus a residual group, TTL curves on the device, allocation on
    the host; hits against the best single TTL under the same budget."""
    from paper_2603_08739_amd import group_ttl as P
    req = dev["req"]
    first = torch.cat([torch.zeros(1, dtype=torch.int64, device="cuda"),
                       torch.nonzero(req[1:] != req[:-1]).flatten() + 1])
    counts = torch.diff(torch.cat([first, torch.tensor([req.numel()], device="cuda")]))
    first_hash = dev["hash"][first].cpu().numpy().view(np.uint64)
    t0 = time.perf_counter()
    g_req, _ = P.subtree_groups(first_hash, k)
    groups = torch.repeat_interleave(torch.from_numpy(g_req).to("cuda"), counts)
    h = K.kv_trace_load(dev["hash"], dev["req"], dev["req_time"], group=groups,
                        weight=dev["weight"], n_groups=k + 1,
                        tokens_per_granule=rec.tokens_per_granule,
                        granule_bytes=rec.granule_bytes)
    hits = torch.zeros((k + 1, len(TTL_GRID)), dtype=torch.int64, device="cuda")
    hitw = torch.zeros_like(hits)
    store = torch.zeros((k + 1, len(TTL_GRID)), dtype=torch.float64, device="cuda")
    K.kv_ttl_curves(h, TTL_GRID, hits, hitw, store)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    H, C = hits.cpu().numpy().astype(np.float64), store.cpu().numpy()
    runs, chosen = [], []
    for frac in budget_fracs:
        budget = frac * float(C[:, -1].sum())
        a = P.allocate(H, C, TTL_GRID, budget)
        t_u, h_u = P.uniform_ttl(H, C, TTL_GRID, budget)
        runs.append({"budget_frac": frac, "hits": a["hits"], "uniform_ttl": t_u,
                     "uniform_hits": h_u, "gain": a["hits"] / h_u - 1.0 if h_u > 0 else None,
                     "ttl": [round(float(x), 3) for x in a["t"]]})
        chosen.append((list(a["t"]), t_u))
        print(f"[bench] group TTL at {frac} of the storage: {a['hits']:.0f} hits against "
              f"{h_u:.0f} with one TTL", file=sys.stderr, flush=True)
    t2 = time.perf_counter()
    # the chosen TTLs evaluated exactly: an unbounded disk TTL tier with the
    # group TTLs (and the single TTL), no HBM or DRAM, through kv_eval_configs
    import tracegen as tg
    from paper_2603_08739_amd import host
    items = []
    for t_g, t_u in chosen:
        items += [{"cap": (0, 0, 0), "ttl": [float(x) for x in t_g]},
                  {"cap": (0, 0, 0), "ttl": float(t_u)}]
    cnt, _ = host.evaluate(h, tg.from_list(items), tg.DEFAULT_COST, k + 1)
    disk_hits = cnt[:, :, 2, 0].sum(axis=1)
    for i, r in enumerate(runs):
        r["evaluated_hits"] = int(disk_hits[2 * i])
        r["evaluated_uniform_hits"] = int(disk_hits[2 * i + 1])
        r["evaluated_gain"] = (r["evaluated_hits"] / r["evaluated_uniform_hits"] - 1.0
                               if r["evaluated_uniform_hits"] else None)
    h.free()
    del groups
    return {"algorithm": f"Alg. 2 over the top {k} prefix subtrees + residual; budgets as "
                         "fractions of the storage at the largest TTL; hits from the "
                         "interpolated curves and, exactly, from kv_eval_configs with the "
                         "chosen TTLs on an unbounded disk TTL tier",
            "groups": k + 1, "n_ttl": len(TTL_GRID), "runs": runs,
            "grouping_and_curves_s": t1 - t0, "optimise_s": t2 - t1}


def prefix_reuse(h, cfgs, G, model, torch, K):
    """The workload's 10,000 LRU configurations with radix-tree prefix reuse
    against the plain inclusive mode: device time of one evaluation each and
    the share of accesses the tiers serve."""
    import tracegen as tg
    from paper_2603_08739_amd import host
    lru = cfgs.subset(np.nonzero(cfgs.policy[:, 0] == tg.POLICY_LRU)[0])
    out = {}
    for name, mode in (("plain", tg.MODE_INCLUSIVE), ("prefix", tg.MODE_INCLUSIVE_PREFIX)):
        b = lru.subset(np.arange(lru.n))
        b.mode[:] = mode
        arr, n_cfg = host.config_array(b)
        counts = torch.zeros((n_cfg, G, 3, 8), dtype=torch.int64, device="cuda")
        K.kv_eval_configs(h, arr, n_cfg, model, counts, None)
        torch.cuda.synchronize()
        K.kv_timing_read(reset=True)
        K.kv_timing_enable(True)
        K.kv_eval_configs(h, arr, n_cfg, model, counts, None)
        torch.cuda.synchronize()
        K.kv_timing_enable(False)
        tm = K.kv_timing_read(reset=True)
        served = counts[..., 0].sum(dim=(1, 2)).double().mean().item()
        out[name] = {"device_ms": round(sum(v[1] for v in tm.values()), 3),
                     "mean_served_accesses": served}
    print(f"[bench] prefix reuse: {out['prefix']['device_ms']} ms against "
          f"{out['plain']['device_ms']} ms", file=sys.stderr, flush=True)
    out["configs"] = lru.n
    return out


def copy_bandwidth(torch, nbytes=2 << 30, reps=5):
    """Rate of a plain device-to-device copy (GB/s, bytes read plus written):
    the achievable HBM bandwidth that the HBM fractions are also quoted
    against, beside the published peak."""
    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    b.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    torch.cuda.empty_cache()
    return 2 * nbytes / (ms / 1000.0) / 1e9


def device_info(torch, copy_gbs):
    p = torch.cuda.get_device_properties(0)
    return {"name": p.name, "arch": getattr(p, "gcnArchName", None),
            "compute_units": p.multi_processor_count, "memory_bytes": int(p.total_memory),
            "copy_GBs": copy_gbs}


def exclusive_replay(torch, tg, host, K):
    """Exclusive (write-back demotion) hierarchies that are no split stack,
    replayed access by access: the tiny workload's 64 configurations as FIFO
    and as LFU hierarchies, one wavefront walking the trace per
    configuration.  Bound by the dependent memory accesses of that walk, so
    the figure is the time per access of one configuration's walk."""
    rec = tg.recipe("tiny")
    base = tg.configs_for("tiny", rec)
    parts = []
    for p in (tg.POLICY_FIFO, tg.POLICY_LFU):
        c = base.subset(np.arange(base.n))
        c.mode[:] = tg.MODE_EXCLUSIVE_DEMOTE
        c.policy[:, :] = p
        parts.append(c)
    cfgs = tg.ConfigBatch.concat(parts)
    dev = rec.expand("cuda")
    n = int(dev["hash"].numel())
    G = rec.n_groups
    h = K.kv_trace_load(dev["hash"], dev["req"], dev["req_time"], group=dev["group"],
                        weight=dev["weight"], n_groups=G,
                        tokens_per_granule=rec.tokens_per_granule,
                        granule_bytes=rec.granule_bytes)
    arr, n_cfg = host.config_array(cfgs)
    model = host.cost_model(tg.DEFAULT_COST)
    counts = torch.zeros((n_cfg, G, 3, 8), dtype=torch.int64, device="cuda")
    K.kv_eval_configs(h, arr, n_cfg, model, counts, None)
    torch.cuda.synchronize()
    K.kv_timing_read(reset=True)
    K.kv_timing_enable(True)
    for _ in range(3):
        K.kv_eval_configs(h, arr, n_cfg, model, counts, None)
    torch.cuda.synchronize()
    K.kv_timing_enable(False)
    calls, ms = K.kv_timing_read(reset=True)["replay_excl"]
    h.free()
    per = ms / max(calls, 1)
    print(f"[bench] exclusive replay: {per:.1f} ms for {n_cfg} configurations",
          file=sys.stderr, flush=True)
    return {"workload": "tiny", "n_accesses": n, "configs": n_cfg,
            "policies": "FIFO and LFU, write-back demotion", "avg_launch_ms": per,
            "launches": calls, "value": n * n_cfg / (per / 1000.0),
            "unit": "block-accesses×configs/s", "ns_per_access": per * 1e6 / n,
            "bound": "dependent memory latency of one lane's walk per configuration"}


def extras(dev, rec, cfgs, G, model, n, torch, K, ttl_only=False):
    """Measurements outside the timed step: TTL curves, Alg. 1, prefix reuse,
    Alg. 2."""
    # TTL curves (disk-tier retention for the group TTL) over the same trace,
    # outside the step: one call per measured launch, timed by the library
    h = K.kv_trace_load(dev["hash"], dev["req"], dev["req_time"], group=dev["group"],
                        weight=dev["weight"], n_groups=G,
                        tokens_per_granule=rec.tokens_per_granule,
                        granule_bytes=rec.granule_bytes)
    t_hits = torch.zeros((G, len(TTL_GRID)), dtype=torch.int64, device="cuda")
    t_hitw = torch.zeros_like(t_hits)
    t_store = torch.zeros((G, len(TTL_GRID)), dtype=torch.float64, device="cuda")
    K.kv_ttl_curves(h, TTL_GRID, t_hits, t_hitw, t_store)
    torch.cuda.synchronize()
    K.kv_timing_enable(True)
    for _ in range(5):
        K.kv_ttl_curves(h, TTL_GRID, t_hits, t_hitw, t_store)
    torch.cuda.synchronize()
    K.kv_timing_enable(False)
    t_calls, t_ms = K.kv_timing_read(reset=True)["ttl_curves"]
    search = prefix = gttl = None
    if not ttl_only:
        search = adaptive_search(h, rec, G, model, torch, K)
        prefix = prefix_reuse(h, cfgs, G, model, torch, K)
    h.free()
    if not ttl_only:
        gttl = group_ttl(dev, rec, torch, K)
    ttl_ms = t_ms / max(t_calls, 1)
    ttl_ach = ALGO_BYTES["ttl_curves"] * n / (ttl_ms / 1000.0) / 1e9
    ttl = {"n_ttl": len(TTL_GRID), "avg_launch_ms": ttl_ms, "launches": t_calls,
           "bound": "hbm", "achieved": ttl_ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": ttl_ach / HBM_PEAK_GBS, "traffic": traffic_for(rec.name, "ttl_curves")}
    print(f"[bench] TTL curves {ttl_ms:.3f} ms", file=sys.stderr, flush=True)
    return ttl, search, prefix, gttl


def measure(name, steps, warmup, torch, tg, host, K, keep=False):
    """Times `steps` whole steps (load + eval + two Pareto passes) of one
    workload on the device; returns the figures, and with `keep` also the
    device inputs for the measurements that follow."""
    print(f"[bench] generating workload {name}", file=sys.stderr, flush=True)
    rec = tg.recipe(name)
    cfgs = tg.configs_for(name, rec)
    dev = rec.expand("cuda")
    torch.cuda.synchronize()
    n = int(dev["hash"].numel())
    arr, n_cfg = host.config_array(cfgs)
    model = host.cost_model(tg.DEFAULT_COST)
    G = rec.n_groups
    counts = torch.zeros((n_cfg, G, 3, 8), dtype=torch.int64, device="cuda")
    obj = torch.zeros((n_cfg, 3), dtype=torch.float64, device="cuda")
    front = torch.zeros(n_cfg, dtype=torch.uint8, device="cuda")
    front_seg = torch.zeros(n_cfg, dtype=torch.uint8, device="cuda")
    seg = torch.from_numpy(cfgs.segment.astype(np.int32)).to("cuda")
    print(f"[bench] {name}: {n} accesses, {n_cfg} configs", file=sys.stderr, flush=True)
    h0 = K.kv_trace_load(dev["hash"], dev["req"], dev["req_time"], group=dev["group"],
                         weight=dev["weight"], n_groups=G,
                         tokens_per_granule=rec.tokens_per_granule,
                         granule_bytes=rec.granule_bytes)
    stats = h0.info()
    h0.free()

    # events on the caller's stream between the three calls (the library's
    # forked streams join it again before each call returns)
    phases = []

    def step():
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record()
        h = K.kv_trace_load(dev["hash"], dev["req"], dev["req_time"], group=dev["group"],
                            weight=dev["weight"], n_groups=G,
                            tokens_per_granule=rec.tokens_per_granule,
                            granule_bytes=rec.granule_bytes)
        ev[1].record()
        K.kv_eval_configs(h, arr, n_cfg, model, counts, obj)
        ev[2].record()
        K.kv_pareto(obj, front, want_count=False)
        K.kv_pareto(obj, front_seg, segment=seg, want_count=False)
        ev[3].record()
        torch.cuda.synchronize()
        h.free()
        phases.append([ev[i].elapsed_time(ev[i + 1]) for i in range(3)])

    for w in range(warmup):
        t0 = time.time()
        step()
        print(f"[bench] {name} warmup {w} {time.time() - t0:.3f} s", file=sys.stderr, flush=True)
    K.kv_timing_read(reset=True)
    K.kv_timing_enable(True)
    phases.clear()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        step()
        print(f"[bench] {name} step {k} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    K.kv_timing_enable(False)
    timing = K.kv_timing_read(reset=True)
    ms_per_step = (t1 - t0) * 1000.0 / steps
    value = n * n_cfg / (ms_per_step / 1000.0)
    # replay work: distinct (order, group, policy, capacity) jobs that are replayed
    jobs_accesses, jobs_count = replay_job_accesses(cfgs, stats, n)
    kern, avg_ms, calls = dominant_kernel(timing, steps)
    units = stage_units(kern, n, jobs_accesses)
    algo = ALGO_BYTES.get(kern, 5.0) * units
    achieved = algo / (avg_ms / 1000.0) / 1e9
    roof = {"bound": "hbm", "kernel": kern, "achieved": achieved, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic_for(name, kern),
            "avg_launch_ms": avg_ms, "launches": calls,
            "algorithmic_bytes_per_launch": algo,
            # a replay launch runs one workgroup (on one compute unit) per job
            "workgroups": jobs_count.get(kern[7:]) if kern.startswith("replay_") else None,
            "stage_ms_per_step": {k: round(v[1] / steps, 3) for k, v in timing.items()
                                  if v[0]}}
    lim = limiter_for(name, kern, avg_ms, roof["workgroups"])
    if lim:
        # the replay is bound by instruction issue and latency, not by HBM:
        # the roofline is the chip's VALU issue rate, the HBM figures stay
        # beside it
        roof["hbm"] = {"achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                       "frac": achieved / HBM_PEAK_GBS}
        roof.update({"bound": "alu", "achieved": lim["achieved"], "peak": lim["peak_chip"],
                     "unit": lim["unit"], "frac": lim["frac_chip"], "limiter": lim})
    roof["stages"] = stage_table(name, timing, steps, n, jobs_accesses, jobs_count)
    med = np.median(np.asarray(phases), axis=0)
    st = roof["stage_ms_per_step"]
    lru_ms = sum(st.get(k, 0.0) for k in ("partition", "stack_matrix", "stack_local",
                                           "stack_assemble", "stack_final", "lru_counts"))
    rep_ms = {k: st[k] for k in ("replay_init", "replay_fifo", "replay_lfu", "replay_combine")
              if k in st}
    calls_ms = {"kv_trace_load": float(med[0]), "kv_eval_configs": float(med[1]),
                "kv_pareto_x2": float(med[2]), "median_of_steps": steps,
                # the metric over kv_eval_configs alone (the load amortised away)
                "value_eval_only": n * n_cfg / (float(med[1]) / 1000.0),
                # device time of the LRU stages and of the replay stages (the two
                # run concurrently on forked streams)
                "lru_part_device_ms": round(lru_ms, 3), "replay_part_device_ms": rep_ms}
    res = {"name": name, "workload": WORKLOAD_TEXT[name], "value": value,
           "ms_per_step": ms_per_step, "steps": steps, "warmup": warmup, "n_accesses": n,
           "n_configs": n_cfg, "n_requests": int(rec.len0.shape[0]), "calls_ms": calls_ms,
           "roofline": roof}
    if keep:
        return res, (rec, cfgs, dev, G, model, n)
    del dev, counts, obj
    return res, None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); multi-GPU sharding "
              "is described in the design notes but not built.", file=sys.stderr)
        sys.exit(2)
    import torch
    import tracegen as tg
    from paper_2603_08739_amd import host, kvcfg as K

    if args.copy_calibration:
        src = torch.ones(args.copy_calibration // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copy calibration: {src.numel() * 4} bytes", file=sys.stderr, flush=True)
        del src, dst
    copy_gbs = copy_bandwidth(torch)
    print(f"[bench] device copy: {copy_gbs:.0f} GB/s", file=sys.stderr, flush=True)
    head, ctx = measure(args.workload, args.steps, args.warmup, torch, tg, host, K, keep=True)
    rec, cfgs, dev, G, model, n = ctx
    def against_copy(res):
        # the HBM figures against the measured copy rate too
        roof = res["roofline"]
        hb = roof.get("hbm", roof if roof["bound"] == "hbm" else None)
        if hb is not None:
            hb["frac_of_copy"] = hb["achieved"] / copy_gbs
        for rec in roof.get("stages", {}).values():
            rec["frac_of_copy"] = rec["achieved"] / copy_gbs

    against_copy(head)
    ttl = search = prefix = gttl = None
    workloads = None
    if not args.no_extras and not args.exclusive_extra_only:
        ttl, search, prefix, gttl = extras(dev, rec, cfgs, G, model, n, torch, K,
                                           ttl_only=args.ttl_extra_only)
        del dev
        torch.cuda.empty_cache()
    excl = None
    if not args.no_extras and not args.ttl_extra_only:
        excl = exclusive_replay(torch, tg, host, K)
    if not args.no_extras and not args.ttl_extra_only and not args.exclusive_extra_only:
        workloads = {}
        for w in ("tiny", "chat", "tenant", "longctx", "full"):
            if w == args.workload:
                continue
            r, _ = measure(w, 5, 1, torch, tg, host, K)
            against_copy(r)
            if not args.no_cpu_baseline:
                # the oracle on a short sample of this workload too (5 s budget)
                wrec = tg.recipe(w)
                r["cpu_baseline"] = cpu_baseline(wrec, tg.configs_for(w, wrec), 5.0)
            workloads[w] = r
    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(rec, cfgs, args.cpu_baseline_seconds)
    out = {
        "metric": METRIC, "value": head["value"], "unit": "block-accesses×configs/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u32",
        "data": "synthetic (seeded generators shaped like the paper's traces)",
        "config": {"workload": head["workload"], "name": args.workload,
                   "n_accesses": head["n_accesses"], "n_configs": head["n_configs"],
                   "n_requests": head["n_requests"]},
        "calls_ms": head["calls_ms"],
        "roofline": head["roofline"], "cpu_baseline": cpu, "workloads": workloads,
        "ttl_curves": ttl, "adaptive_search": search, "group_ttl": gttl,
        "prefix_reuse": prefix, "exclusive_replay": excl,
        "device": device_info(torch, copy_gbs),
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
