"""Host-side accounting of bench.py (no GPU): predecessor counts of the
algorithmic byte model and the grouping of walk launches into passes."""
from __future__ import annotations

import pathlib

import numpy as np

import bench
from tests.tinygraph import AR, Builder

ROOT = pathlib.Path(__file__).resolve().parent.parent


def _graph():
    b = Builder(2)
    c = b.collective(AR, 1 << 20)
    a0 = b.compute(0, 10)
    x0 = b.comm(0, c, preds=[a0])
    b.compute(0, 20, preds=[x0, a0])           # a0 is also the stream predecessor
    b.compute(0, 5, stream=5, preds=[a0])
    a1 = b.compute(1, 7)
    x1 = b.comm(1, c, preds=[a1, a1])          # a repeated explicit dependency
    b.compute(1, 3, preds=[x1])
    return b.graph()


def test_merged_pred_counts_by_enumeration():
    g = _graph()
    n = len(g["op_rank"])
    want = []
    for v in range(n):
        preds = {int(u) for u in g["pred_idx"][g["pred_off"][v]:g["pred_off"][v + 1]]}
        same = [u for u in range(v) if g["op_rank"][u] == g["op_rank"][v] and g["op_stream"][u] == g["op_stream"][v]]
        if same:
            preds.add(same[-1])
        want.append(len(preds))
    assert bench.merged_pred_counts(g).tolist() == want


def test_walk_bytes_per_pass():
    g = _graph()
    preds = int(bench.merged_pred_counts(g).sum())
    n, n_colls, n_compute = len(g["op_rank"]), len(g["coll_type"]), int((g["op_kind"] == 0).sum())
    p = bench.walk_bytes(g, 3, 2)
    first = (16 * n + 8 * preds + 8 * n_colls) * 3
    assert p == [first, first + n_compute * 3, first + n_compute * 3]


def test_walk_passes_split_launches():
    kt = [("init", 0.1), ("cc_cost", 0.2), ("walk", 5.0), ("walk", 4.0),
          ("overlap", 1.0), ("clear", 0.1), ("walk", 6.0), ("walk", 6.5),
          ("overlap", 1.0), ("clear", 0.1), ("walk", 0.01), ("walk", 0.01)]
    assert bench.walk_passes(kt) == [[5.0, 4.0], [6.0, 6.5], [0.01, 0.01]]
    assert bench.walk_passes([("init", 0.1)]) == [[]]


def _timed(pass_ms, launches):
    return {"n_scen": 128, "pass_ms": pass_ms, "pass_launches": launches,
            "pass_kernels": [bench.walk_kernel_name(k > 0, k == len(pass_ms) - 1, False, False, 1)
                             for k in range(len(pass_ms))],
            "pass_index": list(range(len(pass_ms)))}


def test_roofline_headline_is_the_final_pass():
    """Two passes of two launches each: the headline is the final (timeline-writing)
    pass, per launch; every pass is listed with its own algorithmic fraction."""
    g = _graph()
    rf = bench.roofline(g, _timed([4.0, 6.0], [2, 2]), None, None)
    alg = bench.walk_bytes(g, 128, 1)
    assert rf["algorithmic_bytes_per_launch"] == int(alg[1] / 2)
    assert np.isclose(rf["achieved"], round(alg[1] / 2 / 3e-3 / 1e9, 1))
    assert rf["kernel"] == "k_walk<1, true, false>" and rf["traffic"] is None
    assert [p["kernel"] for p in rf["passes"]] == ["k_walk<0, false, false>", "k_walk<1, true, false>"]
    assert rf["passes"][0]["alg_frac"] == round(alg[0] / 4e-3 / 1e9 / bench.HBM_PEAK_GBS, 4)


def test_pass_summary_groups_and_drops_skipped_passes():
    runs = [[[5.0, 4.0], [6.0, 6.5], [0.01]], [[5.2, 4.0], [6.2, 6.5], [0.01]]]
    ps = bench.pass_summary(runs, False, 4)
    assert ps["pass_index"] == [0, 1] and ps["pass_launches"] == [2, 2]
    assert np.allclose(ps["pass_ms"], [9.1, 12.6])
    assert ps["pass_kernels"] == ["k_walk<0, false, false>", "k_walk<1, false, false>"]


def test_walk_kernel_names_follow_the_library_variants():
    """Pass 1 has no per-item input; refined non-final passes fetch whole mask rows; a final
    mask pass fetches flagged rows when its launches average the library's tile threshold
    or more; extra-time passes always fetch flagged rows.  The threshold is the one the
    library compiles in."""
    import re
    tiles = bench.FLAG_ROW_TILES
    assert bench.walk_kernel_name(False, False, False, False, 8) == "k_walk<0, false, false>"
    assert bench.walk_kernel_name(False, True, True, False, 8) == "k_walk<0, true, true>"
    assert bench.walk_kernel_name(True, False, False, False, 8) == "k_walk<1, false, false>"
    assert bench.walk_kernel_name(True, True, False, False, tiles - 1) == "k_walk<1, true, false>"
    assert bench.walk_kernel_name(True, True, False, False, tiles) == "k_walk<2, true, false>"
    assert bench.walk_kernel_name(True, True, False, False, 2 * tiles, 2) == "k_walk<2, true, false>"
    assert bench.walk_kernel_name(True, True, False, False, 2 * tiles - 1, 2) == "k_walk<1, true, false>"
    assert bench.walk_kernel_name(True, True, False, False, tiles, tiles) == "k_walk<1, true, false>"
    assert bench.walk_kernel_name(True, False, False, True, 1) == "k_walk<3, false, false>"
    assert bench.walk_kernel_name(True, True, False, True, 1) == "k_walk<3, true, false>"
    hdr = (ROOT / "paper_2412_12487_amd" / "csrc" / "echo_internal.h").read_text()
    assert int(re.search(r"constexpr int kFlagRowTiles = (\d+);", hdr).group(1)) == tiles


def test_latency_model_arithmetic():
    """Item latency from the chain; a barrier's latency is what its chain takes
    beyond its items."""
    meas = {"chain": ([4.0, 8.0], {"items": 40_000, "lds_barriers": 0, "global_barriers": 0}),
            "lds": ([3.0, 5.0], {"items": 20_000, "lds_barriers": 2_000, "global_barriers": 0}),
            "global": ([6.0, 9.0], {"items": 24_000, "lds_barriers": 0, "global_barriers": 2_000})}
    lat = bench.latency_from(meas, 6554)
    assert lat["first"] == {"item_ns": 100.0, "lds_barrier_ns": 500.0, "global_barrier_ns": 1800.0}
    assert lat["final"] == {"item_ns": 200.0, "lds_barrier_ns": 500.0, "global_barrier_ns": 2100.0}


def test_cpu_baseline_runs_the_gpu_run_options():
    """The oracle leg gets the same validator, CC tables and ensemble as the GPU
    run (a scenario naming a CC table the oracle lacks would be an error)."""
    import argparse

    import oracle
    from workloads import configs, scenarios

    g = configs.graph(1)
    for opts in ({"cc": "tables"}, {"forest": True}, {"until_stable": True, "prorate": True}):
        args = argparse.Namespace(**{"cc": "echo", "forest": False, "until_stable": False, "prorate": False,
                                     **opts})
        sc = bench.cc_variant(configs.scenario_batch(4, 0, 8), args)
        extras = bench.extras_for(args)
        variant = bench.oracle_variant(args, extras)
        cb = bench.cpu_baseline(g, sc, 2, 4, variant)
        assert cb["value"] > 0 and cb["kind"] == "oracle"
        # the options reach the oracle: the ensemble and prorating change its result
        ref = oracle.run(g, scenarios.take(sc, slice(0, 4)), 2, timelines=False, **variant)
        plain = oracle.run(g, scenarios.take(sc, slice(0, 4)), 2, timelines=False,
                           **({"cc_tables": extras["cc_tables"]} if "cc_tables" in extras else {}))
        if opts.get("forest") or opts.get("prorate"):
            assert not np.array_equal(ref["digest"], plain["digest"])
    assert bench.cpu_baseline(g, configs.scenario_batch(1), 1, 1, {}, ops_counted=10)["value"] > 0


def test_roofline_reports_measured_traffic_fraction(tmp_path, monkeypatch):
    """With a byte-counter record for the built kernels, each pass carries its measured
    bytes and their fraction of the peak beside the algorithmic ones."""
    import json
    g = _graph()
    rec = {"config": 3, "kernel_source_sha": bench.source_hash(),
           "pass_bytes": {"k_walk<0, false, false>": 1_000_000_000,
                          "k_walk<1, true, false>": 4_000_000_000}}
    f = tmp_path / "walk_traffic.json"
    f.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    rf = bench.roofline(g, _timed([0.5, 1.0], [1, 1]), None, 3)
    assert rf["traffic"] == 4_000_000_000
    assert rf["traffic_frac"] == round(4e9 / 1e-3 / 1e9 / bench.HBM_PEAK_GBS, 4)
    assert rf["passes"][0]["counter_bytes"] == 1_000_000_000
    assert rf["passes"][0]["counter_frac"] == round(1e9 / 0.5e-3 / 1e9 / bench.HBM_PEAK_GBS, 4)
    rf = bench.roofline(g, _timed([0.5, 1.0], [1, 1]), None, 2)
    assert rf["traffic"] is None and "traffic_frac" not in rf
