"""Benchmark: op-evaluations/s of the timeline composer on one MI355X.

One step = one echo_compose_batch call over the whole scenario batch of the
workload: CC costs, composer pass 1, overlap detection, composer pass 2 (one
refinement) with step time, on inputs already resident in HBM.  The graph is
loaded once before timing (the simulator's initialisation, excluded as in
Table 8 of the paper).

Prints one JSON line with the metric, a roofline entry for the composer
(walk) kernel, and the CPU oracle timed on a bounded sample of the same work.

--replica times the data-parallel symmetry reduction instead (Sec. 8.5, DDP
mode): one DP replica of a graph whose replicas share their durations,
composed alone, against the sweep over every replica; the value counts the
whole job's ops.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "walk_traffic.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2412_12487_amd", "csrc", "echo_kernels.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def merged_pred_counts(g):
    """|preds(v)|: previous op of v's stream plus explicit dependencies, without repeats."""
    n = len(g["op_rank"])
    key = g["op_rank"].astype(np.int64) * 8 + g["op_stream"]
    order = np.lexsort((np.arange(n), key))
    sp = np.full(n, -1, np.int64)
    same = key[order][1:] == key[order][:-1]
    sp[order[1:][same]] = order[:-1][same]
    src = np.repeat(np.arange(n), np.diff(g["pred_off"]))
    pairs = np.unique(np.stack([src, g["pred_idx"].astype(np.int64)], 1), axis=0) if len(src) else \
        np.zeros((0, 2), np.int64)
    explicit = np.bincount(pairs[:, 0], minlength=n)
    dup = np.bincount(pairs[pairs[:, 1] == sp[pairs[:, 0]], 0], minlength=n)
    return explicit + (sp >= 0) - dup


def walk_bytes(g, n_scen, n_refine):
    """Algorithmic bytes of the composer passes (edge-relaxation model):
    per pass and scenario, 16 B written per op (start, finish), 8 B read per
    merged predecessor, 8 B per collective cost; a refined pass also reads a
    1 B overlap mask per compute op."""
    preds = merged_pred_counts(g)
    per_pass = (16 * len(preds) + 8 * int(preds.sum()) + 8 * len(g["coll_type"])) * n_scen
    n_compute = int((g["op_kind"] == 0).sum())
    passes = [per_pass] + [per_pass + 1 * n_compute * n_scen] * n_refine
    return passes


def source_hash():
    """sha256[:16] of the kernels' code: the source with comments removed and whitespace
    collapsed, so that recorded byte counters stay matched to kernels whose text changed
    only in comments."""
    src = open(KERNEL_SRC).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return hashlib.sha256(" ".join(src.split()).encode()).hexdigest()[:16]


def cpu_baseline(g, sc, n_refine, n_sample, variant, ops_counted=None):
    """The oracle on the first n_sample scenarios, with the same validator, CC tables
    and ensemble as the GPU run; op-evals counted as the GPU line counts them."""
    import oracle
    from workloads import scenarios
    sub = scenarios.take(sc, slice(0, n_sample))
    # at most 16 threads: the host cores one GPU's share of the machine comes with
    threads = max(1, min(n_sample, 16, len(os.sched_getaffinity(0))))
    t = time.perf_counter()
    oracle.run(g, sub, n_refine, threads=threads, timelines=False, **variant)
    dt = time.perf_counter() - t
    ops = len(g["op_rank"]) if ops_counted is None else ops_counted
    return {"value": ops * n_sample / dt, "unit": "op-evals/s", "cores": threads,
            "kind": "oracle", "wall_s": round(dt, 3), "nproc": os.cpu_count(),
            "per_core": ops * n_sample / dt / threads,
            "sample": f"scenarios 0..{n_sample - 1} of the same graph, {n_refine} refinement(s), "
                      f"{threads} thread(s)"}


def oracle_variant(args, extras):
    """oracle.run keyword arguments matching the GPU run's options."""
    v = {"until_stable": args.until_stable, "prorate": args.prorate}
    if extras.get("forest") is not None:
        v["forest"] = extras["forest"]
    if extras.get("cc_tables") is not None:
        v["cc_tables"] = extras["cc_tables"]
    return v


def extras_for(args):
    """The CC tables and the slowdown ensemble the options ask for."""
    from workloads import scenarios
    ex = {}
    if args.cc == "tables":
        ex["cc_tables"] = scenarios.draw_cc_tables(CC_TABLES, np.random.default_rng(99))
    if args.forest:
        from workloads import slowdown_forest
        ex["forest"] = slowdown_forest.synthetic_forest(0)
    return ex


def write_probe(torch, nbytes):
    """HBM write rate of torch's own fill kernels on an int64 array of nbytes, viewed as
    rows of 256 values (2 KB, one op's row of 256 scenarios): the whole array, and the
    array written as four launches of one 512-byte quarter of every row (one 64-scenario
    tile's segment, the unit the composer's timeline stores write).  Median of 3 runs."""
    rows = nbytes // 2048
    a = torch.empty((rows, 4, 64), dtype=torch.int64, device="cuda:0")
    def timed(fn):
        ts = []
        for _ in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return sorted(ts[1:])[1]
    whole = timed(lambda: a.fill_(1))
    def quarters():
        for t in range(4):
            a[:, t, :].fill_(t)
    quarter = timed(quarters)
    b = rows * 2048
    return {"write_probe_bytes": b, "whole_ms": round(whole, 3), "whole_TBps": round(b / whole / 1e9, 3),
            "quarter_rows_ms": round(quarter, 3), "quarter_rows_TBps": round(b / quarter / 1e9, 3)}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=3, help="workload 1-5 (see workloads/configs.py)")
    ap.add_argument("--index", type=int, default=0, help="graph of config 5 (0-15)")
    ap.add_argument("--scenarios", type=int, default=0,
                    help="batch size drawn with the config's recipe (0 = the config's own)")
    ap.add_argument("--forest", action="store_true",
                    help="validator variant: slowdown factors predicted by a seeded 64-tree ensemble")
    ap.add_argument("--cc", choices=["echo", "tables", "alpha-beta"], default="echo",
                    help="collective cost model of every scenario: Eq. 2-5 from bandwidths, Eq. 2-5 from "
                         "seeded CC parameter tables, or the alpha-beta baseline")
    ap.add_argument("--replica", action="store_true",
                    help="time one DP replica composed alone against the sweep over every replica")
    ap.add_argument("--refine", type=int, default=1, help="refinements (the most, with --until-stable)")
    ap.add_argument("--until-stable", action="store_true",
                    help="validator variant: refine until no duration changes (at most --refine times)")
    ap.add_argument("--prorate", action="store_true",
                    help="validator variant: inflate only the overlapped part of a compute op")
    ap.add_argument("--all", action="store_true",
                    help="config 5 as one batch: its 16 graphs composed back to back in every step")
    ap.add_argument("--no-floor", dest="floor", action="store_false",
                    help="skip the walk latency microbenchmarks (no latency floor per pass)")
    ap.add_argument("--cpu-sample", type=int, default=48, help="scenarios the CPU oracle composes (0 = skip)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device-to-device once (calibrates HBM byte counters) and exit")
    ap.add_argument("--write-probe", type=int, default=0, metavar="GIB",
                    help="only time HBM writes of a GIB GiB int64 array, whole and as 512-byte quarters of "
                         "2 KB rows (the timeline rows' pattern), and exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU: the composer evaluates every scenario on a single MI355X "
              f"(asked for {max(args.gpus, world)}); sharding the scenarios across GPUs is not built.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n}), flush=True)
        return
    if args.write_probe:
        print(json.dumps(write_probe(torch, args.write_probe << 30)), flush=True)
        return

    import paper_2412_12487_amd as E
    from workloads import configs, gpt1f1b

    E.lib()
    if args.replica:
        return replica_mode(args, E, configs, gpt1f1b)
    if args.all:
        return batch_mode(args, E, configs)
    t = time.perf_counter()
    g = configs.graph(args.config, args.index)
    sc = cc_variant(configs.scenario_batch(args.config, args.index, args.scenarios or None), args)
    log(f"graph: config {args.config} {configs.NAMES[args.config]}: {len(g['op_rank'])} ops, "
        f"{len(g['coll_type'])} collectives, {g['n_ranks']} ranks ({time.perf_counter() - t:.1f} s)")
    extras = extras_for(args)
    latency = None
    if args.floor:
        latency = latency_model(E, int(np.max(sc["jitter_amp_q16"])))
        log(f"walk latencies: {latency}")
    r = time_compose(E, g, sc, args, extras, latency)
    line = {
        "metric": "op-evaluations/sec (ops x scenarios composed), 1 GPU",
        "value": round(r["value"], 1),
        "unit": "op-evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 4),
        "gpu_ms_per_step": round(r["gpu_ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": f"config {args.config}: {configs.NAMES[args.config]}, "
                               f"{r['n_ops']} ops x {r['n_scen']} scenarios, " + validator_name(args),
                   "n_ops": r["n_ops"], "n_scenarios": r["n_scen"], "n_refine": args.refine,
                   "ranks": int(g["n_ranks"]), "levels": r["levels"], "load_s": round(r["load_s"], 2),
                   "cc_model": args.cc, "cc_cost_all_collectives_ms": r["cc_cost_all_ms"]},
        "kernels_ms": r["kernels_ms"],
        "walk_pass_ms": r["walk_pass_ms"],
        "roofline": roofline(g, r, args, args.config if not (args.until_stable or args.prorate or args.forest
                                                             or args.cc != "echo") else None),
    }
    if latency is not None:
        line["latency_model"] = latency
    if "refinements" in r:
        line["config"]["refinements"] = r["refinements"]
    if args.cpu_sample > 0:
        log(f"cpu baseline: oracle on {args.cpu_sample} scenario(s) ...")
        line["cpu_baseline"] = cpu_baseline(g, sc, args.refine, args.cpu_sample, oracle_variant(args, extras))
    print(json.dumps(line), flush=True)


def validator_name(args):
    if not (args.until_stable or args.prorate or args.forest):
        return f"{args.refine} refinement(s)"
    kind = " + ".join(x for x, on in (("until stable", args.until_stable), ("prorated", args.prorate),
                                      ("ensemble factors", args.forest)) if on)
    return f"validator {kind}, at most {args.refine} refinement(s)"


CC_TABLES = 8       # seeded tables for --cc tables


def cc_variant(sc, args):
    """Scenarios with the cost model --cc asks for."""
    from workloads import scenarios
    n = scenarios.count(sc)
    sc = dict(sc)
    if args.cc == "alpha-beta":
        sc["cc_model"] = np.ones(n, np.uint8)
    elif args.cc == "tables":
        sc["cc_table"] = (np.arange(n) % CC_TABLES + 1).astype(np.int32)
    return sc


# A final mask pass whose launches average at least this many 64-scenario tiles runs the walk
# variant that fetches only flagged mask rows (the library's kFlagRowTiles).
FLAG_ROW_TILES = 2


def walk_kernel_name(refined, final, digest, ext, n_tiles, launches=1):
    """The walk kernel a pass launches, as rocprofv3 names it: k_walk<input, final, digest>
    with input 0 = none (first pass), 1 = whole mask rows, 2 = flagged mask rows (a final
    pass of n_tiles >= FLAG_ROW_TILES x launches), 3 = flagged extra-time rows."""
    b = lambda x: "true" if x else "false"
    flagged = final and n_tiles >= FLAG_ROW_TILES * launches
    inp = 0 if not refined else 3 if ext else 2 if flagged else 1
    return f"k_walk<{inp}, {b(final)}, {b(digest)}>"


def time_compose(E, g, sc, args, extras, latency=None):
    """Load g, compose the batch warmup + steps times; wall and per-kernel timings.
    latency: the walk's measured per-item and per-barrier latencies (latency_model),
    turned into a latency floor per pass with the graph's longest walk chain."""
    t = time.perf_counter()
    G = E.Graph(g, 0)
    try:
        return _time_compose(E, G, sc, args, extras, latency, time.perf_counter() - t)
    finally:
        G.close()


def _time_compose(E, G, sc, args, extras, latency, load_s):
    import torch
    if extras.get("cc_tables") is not None:
        G.set_cc_tables(extras["cc_tables"])
    if extras.get("forest") is not None:
        G.set_forest(extras["forest"])
    log(f"loaded: {G.n_levels} levels in {load_s:.1f} s")
    d_scen, n_scen = E.scenarios_to_device(sc, "cuda:0")
    dev = torch.device("cuda:0")
    out = {"step": torch.empty(n_scen, dtype=torch.int64, device=dev),
           "start": torch.empty((G.n_ops, n_scen), dtype=torch.int64, device=dev),
           "finish": torch.empty((G.n_ops, n_scen), dtype=torch.int64, device=dev)}
    G.set_timing(True)
    variant = dict(until_stable=args.until_stable, prorate=args.prorate, forest=args.forest,
                   refinements=args.until_stable or args.prorate or args.forest)
    for i in range(args.warmup):
        G.compose(d_scen, n_scen, args.refine, out=out, **variant)
        log(f"warmup {i}: {G.kernel_times()}")
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    step_ms, kernels, pass_runs = [], {}, []
    last = {}
    t0 = time.perf_counter()
    for i in range(args.steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        last = G.compose(d_scen, n_scen, args.refine, out=out, check=False, **variant)
        e1.record(stream)
        torch.cuda.synchronize()
        step_ms.append(e0.elapsed_time(e1))
        kt = G.kernel_times()
        pass_runs.append(walk_passes(kt))
        for k, ms in kt:
            kernels.setdefault(k, []).append(ms)
        log(f"step {i}: {step_ms[-1]:.3f} ms  walk passes {[round(sum(p), 3) for p in pass_runs[-1]]} ms")
    wall = time.perf_counter() - t0
    G.sync_status()
    ms_per_step = wall * 1000.0 / max(args.steps, 1)
    res = {"n_ops": G.n_ops, "n_scen": n_scen, "levels": G.n_levels, "load_s": load_s,
           "ms_per_step": ms_per_step, "gpu_ms": float(np.median(step_ms)) if step_ms else 0.0,
           "value": G.n_ops * n_scen / (ms_per_step / 1000.0),
           "kernels_ms": {k: round(float(np.mean(v)), 4) for k, v in kernels.items()},
           # the last step's walk launches, pass by pass (a split pass lists each launch)
           "walk_pass_ms": [[round(ms, 4) for ms in p] for p in pass_runs[-1] if p] if pass_runs else []}
    res.update(pass_summary(pass_runs, args.prorate or args.forest, (n_scen + 63) // 64))
    if latency is not None:
        n_pass = max(res["pass_index"]) + 1 if res["pass_index"] else 1
        res["floors"] = [walk_floor(G, latency, k, n_pass) for k in res["pass_index"]]
    if "refinements" in last:
        rf = last["refinements"].cpu().numpy()
        res["refinements"] = {"min": int(rf.min()), "mean": round(float(rf.mean()), 3), "max": int(rf.max())}
    # the CC estimator alone over every collective (echo_cc_cost), per call
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    G.cc_cost(d_scen, n_scen)
    e0.record(stream)
    for _ in range(3):
        costs = G.cc_cost(d_scen, n_scen, check=False)
    e1.record(stream)
    torch.cuda.synchronize()
    res["cc_cost_all_ms"] = round(e0.elapsed_time(e1) / 3, 4)
    del costs
    del out
    return res


def pass_summary(pass_runs, ext, n_tiles):
    """Walk passes of the timed steps: mean time per pass (a pass split over several
    launches counts all of them), launches per pass and the kernel variant; passes that
    returned at once (every scenario already at its fixed point) are left out."""
    n_pass = max((len(p) for p in pass_runs), default=0)
    pass_ms = [float(np.mean([sum(p[k]) for p in pass_runs if k < len(p)])) for k in range(n_pass)]
    launches = [max(len(p[k]) for p in pass_runs if k < len(p)) for k in range(n_pass)]
    top = max(pass_ms, default=0.0)
    ran = [k for k in range(n_pass) if pass_ms[k] > 0.02 * top]
    names = [walk_kernel_name(k > 0, k == n_pass - 1, False, ext, n_tiles, launches[k]) for k in range(n_pass)]
    return {"pass_ms": [pass_ms[k] for k in ran], "pass_launches": [launches[k] for k in ran],
            "pass_kernels": [names[k] for k in ran], "pass_index": ran}


def walk_passes(kernel_times):
    """One compose call's walk launch times grouped by pass: every pass after the
    first begins with its overlap detection launch."""
    passes = [[]]
    for kind, ms in kernel_times:
        if kind == "overlap":
            passes.append([])
        elif kind == "walk":
            passes[-1].append(ms)
    return passes


# ---------------------------------------------------------------- latency floor of the walk
def latency_model(E, jitter_amp, n_scen=64):
    """The walk's latencies measured on the device with small graphs whose longest
    chain is known (workloads.microbench): ns per walk item (a chain of 40,000
    compute ops on one rank), and per barrier met in LDS (eight ranks joining an
    all-reduce after every eight ops) or in device memory (send/recv between ranks
    of two workgroups), for the first pass (stores only what later kernels read)
    and the final, refined pass (stores every start and finish).  Each graph
    composes one 64-scenario tile with the workload's jitter amplitude and one
    refinement; median of three calls after a warm-up.  A barrier's latency is
    what its chain takes beyond its items."""
    import torch
    from workloads import microbench, scenarios
    sc = scenarios.default_scenarios(n_scen)
    if jitter_amp:
        sc["jitter_amp_q16"][:] = jitter_amp
        sc["jitter_seed"][:] = 1
    d, n = E.scenarios_to_device(sc, "cuda:0")
    graphs = {"chain": microbench.chain(40_000), "lds": microbench.allreduce_rounds(8, 2_000, 8),
              "global": microbench.p2p_pingpong(1_000, 8)}
    meas = {}
    for name, g in graphs.items():
        G = E.Graph(g, 0)
        try:
            G.set_timing(True)
            chain = G.walk_chain(1, 0, 0)
            runs = []
            for _ in range(4):
                G.compose(d, n, 1, timelines=True)
                torch.cuda.synchronize()
                runs.append([sum(p) for p in walk_passes(G.kernel_times())])
        finally:
            G.close()
        meas[name] = ([float(np.median([r[k] for r in runs[1:]])) for k in (0, 1)], chain)
    return latency_from(meas, jitter_amp)


def latency_from(meas, jitter_amp):
    """Per-item and per-barrier latencies (ns) from the microbenchmark walk times
    {name: ([first-pass ms, final-pass ms], its walk chain with unit item weights)}."""
    out = {}
    (mc, cc), (ml, cl), (mg, cg) = meas["chain"], meas["lds"], meas["global"]
    for k, key in ((0, "first"), (1, "final")):
        item = mc[k] * 1e6 / cc["items"]
        lds = max(0.0, (ml[k] * 1e6 - cl["items"] * item) / max(cl["lds_barriers"], 1))
        glob = max(0.0, (mg[k] * 1e6 - cg["items"] * item - cg["lds_barriers"] * lds) /
                   max(cg["global_barriers"], 1))
        out[key] = {"item_ns": round(item, 2), "lds_barrier_ns": round(lds, 1), "global_barrier_ns": round(glob, 1)}
    out["jitter_amp_q16"] = int(jitter_amp)
    out["walk_ms"] = {name: [round(x, 4) for x in m[0]] for name, m in meas.items()}
    return out


def walk_floor(G, latency, k, n_pass):
    """Latency floor of walk pass k: the graph's longest walk chain with the measured
    per-item and per-barrier latencies of that kind of pass (a refined pass that is
    not the last takes the smaller of the two kinds' latencies, so it stays a floor)."""
    first, final = latency["first"], latency["final"]
    if k == 0:
        w = first
    elif k == n_pass - 1:
        w = final
    else:
        w = {key: min(first[key], final[key]) for key in first}
    ps = [int(w["item_ns"] * 1000), int(w["lds_barrier_ns"] * 1000), int(w["global_barrier_ns"] * 1000)]
    ch = G.walk_chain(*ps)
    return {"floor_ms": round(ch["ps"] / 1e9, 4), "chain_items": ch["items"], "lds_barriers": ch["lds_barriers"],
            "global_barriers": ch["global_barriers"]}


def roofline(g, r, args, traffic_config):
    """Per walk pass: algorithmic bytes (edge-relaxation model) and their fraction of
    the HBM peak at the pass's measured time, the byte counters' bytes when recorded
    for these very kernels, and the latency floor; the headline is the final,
    timeline-producing pass."""
    n_pass = max(r["pass_index"]) + 1 if r["pass_index"] else 1
    alg = walk_bytes(g, r["n_scen"], n_pass - 1)
    traffic = {}
    if traffic_config is not None and os.path.exists(TRAFFIC_FILE):
        tr = json.load(open(TRAFFIC_FILE))
        if tr.get("kernel_source_sha") == source_hash() and tr.get("config") == traffic_config:
            traffic = tr.get("pass_bytes", {})
    passes = []
    for j, k in enumerate(r["pass_index"]):
        ms = r["pass_ms"][j]
        e = {"pass": k + 1, "kernel": r["pass_kernels"][j], "launches": r["pass_launches"][j], "ms": round(ms, 4),
             "alg_bytes": int(alg[k]), "alg_frac": round(alg[k] / (ms / 1000.0) / 1e9 / HBM_PEAK_GBS, 4)}
        cb = traffic.get(r["pass_kernels"][j])
        e["counter_bytes"] = int(cb) if cb is not None else None
        e["counter_frac"] = round(cb / (ms / 1000.0) / 1e9 / HBM_PEAK_GBS, 4) if cb is not None else None
        if r.get("floors"):
            f = r["floors"][j]
            e.update(f)
            e["over_floor"] = round(ms / f["floor_ms"], 3) if f["floor_ms"] > 0 else None
        passes.append(e)
    head = passes[-1] if passes else {"kernel": "k_walk", "launches": 1, "ms": 0.0, "alg_bytes": 0,
                                      "counter_bytes": None, "counter_frac": None}
    per_launch = head["alg_bytes"] / max(head["launches"], 1)
    launch_ms = head["ms"] / max(head["launches"], 1)
    achieved = per_launch / (launch_ms / 1000.0) / 1e9 if launch_ms > 0 else 0.0
    out = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": round(achieved / HBM_PEAK_GBS, 4),
           "traffic": int(head["counter_bytes"] / max(head["launches"], 1))
           if head["counter_bytes"] is not None else None,
           "kernel": head["kernel"], "role": "final walk pass, the one that writes the caller's timelines",
           "avg_launch_ms": round(launch_ms, 4), "algorithmic_bytes_per_launch": int(per_launch)}
    if out["traffic"] is not None:
        out["traffic_frac"] = head["counter_frac"]
    out["passes"] = passes
    return out


def batch_mode(args, E, configs):
    """Config 5 as the batch it is: all 16 extrapolation graphs resident at once, every
    step composing each of them (its own 32 scenarios, one refinement, timelines out)
    back to back on one stream.  One pair of timeline buffers, sized for the largest
    graph, serves every call (the calls run one after the other)."""
    import torch
    if args.config != 5:
        raise SystemExit("--all is for config 5 (the 16-graph extrapolation batch)")
    n_graphs = len(configs.EXTRAP_GRAPHS)
    graphs, alg, pred_counts = [], [], []
    t = time.perf_counter()
    for i in range(n_graphs):
        g = configs.graph(5, i)
        sc = cc_variant(configs.scenario_batch(5, i, args.scenarios or None), args)
        G = E.Graph(g, 0)
        G.set_timing(True)
        d, n = E.scenarios_to_device(sc, "cuda:0")
        graphs.append({"G": G, "d": d, "n": n, "ops": G.n_ops, "ranks": int(g["n_ranks"]), "levels": G.n_levels})
        alg.append(walk_bytes(g, n, args.refine))
        log(f"graph {i + 1}/{n_graphs}: {G.n_ops} ops, {g['n_ranks']} ranks, loaded "
            f"({time.perf_counter() - t:.1f} s so far)")
        del g
    try:
        dev = torch.device("cuda:0")
        rows = max(x["ops"] * x["n"] for x in graphs)
        out = {"step": torch.empty(max(x["n"] for x in graphs), dtype=torch.int64, device=dev),
               "start": torch.empty(rows, dtype=torch.int64, device=dev),
               "finish": torch.empty(rows, dtype=torch.int64, device=dev)}

        def one_step():
            for x in graphs:
                x["G"].compose(x["d"], x["n"], args.refine, out=out, check=False)

        for i in range(args.warmup):
            one_step()
            torch.cuda.synchronize()
            log(f"warmup {i} done")
        stream = torch.cuda.current_stream(dev)
        step_ms, per_graph = [], [[] for _ in graphs]
        t0 = time.perf_counter()
        for i in range(args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for x in graphs:
                x["G"].compose(x["d"], x["n"], args.refine, out=out, check=False)
            e1.record(stream)
            torch.cuda.synchronize()
            step_ms.append(e0.elapsed_time(e1))
            for j, x in enumerate(graphs):       # each graph records its own kernels' events
                per_graph[j].append(x["G"].kernel_times())
            log(f"step {i}: {step_ms[-1]:.3f} ms")
        wall = time.perf_counter() - t0
        for x in graphs:
            x["G"].sync_status()
    finally:
        for x in graphs:
            x["G"].close()
    ms_per_step = wall * 1000.0 / max(args.steps, 1)
    total = sum(x["ops"] * x["n"] for x in graphs)
    rows = []
    for j, x in enumerate(graphs):
        runs = [walk_passes(kt) for kt in per_graph[j]]
        ps = pass_summary(runs, False, (x["n"] + 63) // 64)
        compose_ms = float(np.mean([sum(ms for _, ms in kt) for kt in per_graph[j]]))
        final = ps["pass_index"][-1] if ps["pass_index"] else 0
        fms = ps["pass_ms"][-1] if ps["pass_ms"] else 0.0
        model, tp, pp, dp, m, distopt = configs.EXTRAP_GRAPHS[j]
        rows.append({"graph": j + 1, "model": model, "tp": tp, "pp": pp, "dp": dp, "microbatches": m,
                     "distributed_optimizer": distopt, "ops": x["ops"], "ranks": x["ranks"], "levels": x["levels"],
                     "kernels_ms": round(compose_ms, 4), "walk_pass_ms": [round(v, 4) for v in ps["pass_ms"]],
                     "final_pass_alg_frac": round(alg[j][final] / (fms / 1000.0) / 1e9 / HBM_PEAK_GBS, 4)
                     if fms > 0 else None})
    line = {
        "metric": "op-evaluations/sec (ops x scenarios composed), 1 GPU",
        "value": round(total / (ms_per_step / 1000.0), 1),
        "unit": "op-evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "gpu_ms_per_step": round(float(np.median(step_ms)), 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": f"config 5: {configs.NAMES[5]}, all {n_graphs} graphs composed back to back, "
                               f"{sum(x['ops'] for x in graphs)} ops, {graphs[0]['n']} scenarios each, "
                               f"{args.refine} refinement(s)",
                   "n_ops": sum(x["ops"] for x in graphs), "n_scenarios_each": graphs[0]["n"],
                   "n_refine": args.refine, "load_s": round(time.perf_counter() - t - wall, 1)},
        "note": "32 scenarios fill half of each 64-lane wavefront: every walk item costs a whole "
                "wavefront for half its lanes",
        "graphs": rows,
    }
    print(json.dumps(line), flush=True)


def replica_mode(args, E, configs, gpt1f1b):
    """Symmetry reduction (one DP replica composed alone) against the sweep over
    every replica, on a graph whose replicas share their durations."""
    params = configs.graph_params(args.config, args.index)
    t = time.perf_counter()
    g = gpt1f1b.gpt_graph(**params, replica_invariant=True)
    rg, _ = gpt1f1b.dp_replica(g, params["tp"], params["dp"])
    sc = cc_variant(configs.scenario_batch(args.config, args.index, args.scenarios or None), args)
    name = f"config {args.config}" + (f" graph {args.index + 1}" if args.config == 5 else "") + \
        f" (TP{params['tp']} x PP{params['pp']} x DP{params['dp']}, replica-invariant durations)"
    log(f"graphs: {name}: {len(g['op_rank'])} ops, replica {len(rg['op_rank'])} ops "
        f"({time.perf_counter() - t:.1f} s)")
    n_scen = len(sc["alpha_ns"])
    # the sweep over every replica needs start + finish + masks for all of the job's ops
    full_fits = len(g["op_rank"]) * n_scen * 17 < 200 * 10**9
    extras = extras_for(args)
    full = time_compose(E, g, sc, args, extras) if full_fits else None
    red = time_compose(E, rg, sc, args, extras)
    line = {
        "metric": "op-evaluations/sec (ops x scenarios of the whole job, composed through one DP replica), 1 GPU",
        "value": round(len(g["op_rank"]) * red["n_scen"] / (red["ms_per_step"] / 1000.0), 1),
        "unit": "op-evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(red["ms_per_step"], 4),
        "gpu_ms_per_step": round(red["gpu_ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": f"{name}, DP-replica mode: {red['n_ops']} of {len(g['op_rank'])} ops x "
                               f"{red['n_scen']} scenarios, {args.refine} refinement(s)",
                   "n_ops_job": len(g["op_rank"]), "n_ops_replica": red["n_ops"], "n_scenarios": red["n_scen"],
                   "n_refine": args.refine,
                   "full_sweep_ms_per_step": round(full["ms_per_step"], 4) if full else None,
                   "speedup_vs_full_sweep": round(full["ms_per_step"] / red["ms_per_step"], 2) if full else None},
        "kernels_ms": red["kernels_ms"],
        "walk_pass_ms": red["walk_pass_ms"],
        "roofline": roofline(rg, red, args, None),
    }
    if args.cpu_sample > 0:
        log(f"cpu baseline: oracle on {args.cpu_sample} scenario(s) of the replica ...")
        line["cpu_baseline"] = cpu_baseline(rg, sc, args.refine, args.cpu_sample, oracle_variant(args, extras),
                                            ops_counted=len(g["op_rank"]))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
