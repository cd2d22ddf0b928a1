"""Parity of the HIP composer with the CPU oracle, bit for bit (int64 ns, Q16).

All calls go through the C ABI (libecho.so via the ctypes binding).  Small
configurations compare every start/finish/step/digest; the full-size GPT-175B
graphs compare sampled scenarios' timelines in full against the oracle run in
the test, in the launch configuration the benchmark times (timelines out, no
digest), and every scenario's step time and digest against the oracle's values
stored by tests/golden/make_full_digests.py.
"""
from __future__ import annotations

import os

import numpy as np
import pytest

import oracle
from tests import tinygraph
from tests.test_oracle_pins import _tiny_cases
from tests.tinygraph import AG, AR, P2P, RS, Builder
from workloads import configs, gpt1f1b, scenarios

pytestmark = pytest.mark.gpu

THREADS = max(1, min(16, os.cpu_count() or 1))


@pytest.fixture(scope="module")
def E():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2412_12487_amd as E
    E.lib()      # fails loudly if libecho.so was not built
    return E


def gpu_run(E, g, sc, R, *, timelines=True, digest=True, graph=None):
    G = graph or E.Graph(g, 0)
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, R, timelines=timelines, digest=digest)
    res = {"step": out["step"].cpu().numpy()}
    if digest:
        res["digest"] = out["digest"].cpu().numpy().view(np.uint64)
    if timelines:
        res["start"] = out["start"].cpu().numpy()
        res["finish"] = out["finish"].cpu().numpy()
    if graph is None:
        G.close()
    return res


def assert_same(gpu, ref, cols=None):
    """gpu: [n_ops, n_scen] arrays; ref: oracle output [n_scen', n_ops] for scenarios `cols`."""
    cols = list(range(ref["step"].shape[0])) if cols is None else list(cols)
    np.testing.assert_array_equal(gpu["step"][cols], ref["step"])
    if "digest" in gpu:
        np.testing.assert_array_equal(gpu["digest"][cols], ref["digest"])
    if "start" in gpu and "start" in ref:
        for j, c in enumerate(cols):
            np.testing.assert_array_equal(gpu["start"][:, c], ref["start"][j], err_msg=f"start, scenario {c}")
            np.testing.assert_array_equal(gpu["finish"][:, c], ref["finish"][j], err_msg=f"finish, scenario {c}")


# ---------------------------------------------------------------- small graphs, everything compared
TINY = _tiny_cases()


@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("R", [0, 1, 2])
def test_tiny_graphs(E, name, R):
    g = TINY[name]
    sc = scenarios.draw(3, np.random.default_rng(7), bw_inter=(20000, 90000), alpha=(0, 5000),
                        ar_algo_random=True, slowdown=(65536, 140000))
    assert_same(gpu_run(E, g, sc, R), oracle.run(g, sc, R))


def _random_graph(rng, n_ranks, ops_per_rank, n_coll, p_comm=0.3, comm_streams=4):
    b = Builder(n_ranks, gpus_per_node=int(rng.integers(1, 5)))
    colls = []
    for _ in range(n_coll):
        t = int(rng.integers(0, 4 if n_ranks > 1 else 3))
        k = 2 if t == P2P else int(rng.integers(1, n_ranks + 1))
        members = sorted(rng.choice(n_ranks, size=min(k, n_ranks), replace=False).tolist())
        if t == P2P and len(members) < 2:
            continue
        colls.append((b.collective(t, int(rng.integers(0, 64 << 20))), members,
                      int(rng.integers(1, 1 + comm_streams))))
    # every rank issues its collectives in collective-id order on a per-collective stream
    for r in range(n_ranks):
        ids = []
        mine = [(c, s) for c, m, s in colls if r in m]
        for k in range(ops_per_rank):
            preds = [int(u) for u in ids[-6:] if rng.random() < 0.25]
            if mine and rng.random() < p_comm:
                c, s = mine.pop(0)
                ids.append(b.comm(r, c, stream=s, preds=preds))
            elif rng.random() < 0.1:
                ids.append(b.op(r, stream=5, kind=2, dur=int(rng.integers(0, 4000)), preds=preds))
            else:
                ids.append(b.compute(r, int(rng.integers(0, 90000)), stream=int(rng.integers(0, 2)) * 6,
                                     cls=int(rng.integers(0, 8)), preds=preds))
        for c, s in mine:
            b.comm(r, c, stream=s, preds=ids[-1:])
    return b.graph()


def test_maximum_refinement_count(E):
    """R = 64, the largest count the ABI takes: 65 walk passes and 64 overlap detections
    over one workspace, on a random 12-rank graph with two ragged tiles of scenarios and
    slowdowns strong enough that the timelines keep moving for several refinements."""
    g = _random_graph(np.random.default_rng(5), 12, 40, 20)
    sc = scenarios.draw(70, np.random.default_rng(64), bw_inter=(20000, 90000), alpha=(0, 5000),
                        ar_algo_random=True, slowdown=(65536, 200000), jitter=(3000, 4))
    assert_same(gpu_run(E, g, sc, 64), oracle.run(g, sc, 64, threads=THREADS))


@pytest.mark.parametrize("seed", range(12))
def test_random_graphs(E, seed):
    rng = np.random.default_rng(1000 + seed)
    g = _random_graph(rng, int(rng.integers(1, 17)), int(rng.integers(5, 60)), int(rng.integers(0, 30)))
    n = [1, 5, 64, 70, 130][seed % 5]
    sc = scenarios.draw(n, rng, bw_inter=(20000, 400000), bw_intra=(50000, 400000), alpha=(0, 20000),
                        ar_algo_random=True, slowdown=(65536, 150000),
                        jitter=(int(rng.integers(0, 20000)), int(seed)) if seed % 2 else None)
    try:
        ref = {R: oracle.run(g, sc, R, threads=THREADS) for R in (0, 1, 2)}
    except oracle.OracleError as e:      # generator made a deadlock: the library must agree
        assert e.code == -4
        with pytest.raises(E.EchoError) as x:
            E.Graph(g, 0)
        assert x.value.code in (E.ECHO_ERR_CYCLE, E.ECHO_ERR_MATCH)
        return
    G = E.Graph(g, 0)
    for R in (0, 1, 2):
        assert_same(gpu_run(E, g, sc, R, graph=G), ref[R])
    G.close()


# ---------------------------------------------------------------- several ranks per wavefront
# A graph with more ranks than the device holds wavefronts is walked with
# several ranks per wavefront; these tests force that layout on small graphs.
@pytest.mark.parametrize("rpw", [2, 3, 8])
def test_walkers_of_several_ranks_tiny(E, rpw):
    sc = scenarios.draw(3, np.random.default_rng(8), bw_inter=(20000, 90000), alpha=(0, 5000),
                        ar_algo_random=True, slowdown=(65536, 140000), jitter=(3000, 5))
    for name in sorted(TINY):
        g = TINY[name]
        G = E.Graph(g, 0, ranks_per_walker=rpw)
        for R in (0, 2):
            assert_same(gpu_run(E, g, sc, R, graph=G), oracle.run(g, sc, R))
        G.close()


def test_random_graphs_every_final_pass_variant(E):
    """300 random graphs with 65-256 scenarios (two to four tiles), one or two refinements or
    the fixed-point and prorated validators, some with one to three tiles per walk launch:
    the final pass runs with flagged mask rows, whole rows and flagged extra times.  Every
    start, finish, step and digest against the oracle."""
    for seed in range(300):
        rng = np.random.default_rng(90_000 + seed)
        g = _random_graph(rng, int(rng.integers(2, 40)), int(rng.integers(5, 60)), int(rng.integers(0, 40)))
        n = int(rng.choice([65, 100, 130, 192, 256]))
        sc = scenarios.draw(n, rng, bw_inter=(20000, 400000), bw_intra=(50000, 400000), alpha=(0, 20000),
                            ar_algo_random=True, slowdown=(65536, 150000), jitter=(5000, seed))
        R = int(rng.integers(1, 3))
        variant = int(rng.integers(0, 3))
        kw = [{}, {"until_stable": True}, {"prorate": True}][variant]
        if variant == 1:
            R = 6
        ref = oracle.run(g, sc, R, threads=THREADS, **kw)
        G = E.Graph(g, 0)
        try:
            if rng.integers(0, 2):
                G.set_launch_tiles(int(rng.integers(1, 4)))
            d, ns = E.scenarios_to_device(sc)
            out = G.compose(d, ns, R, timelines=True, digest=True, refinements=variant > 0, **kw)
            gpu = {"step": out["step"].cpu().numpy(), "digest": out["digest"].cpu().numpy().view(np.uint64),
                   "start": out["start"].cpu().numpy(), "finish": out["finish"].cpu().numpy()}
            assert_same(gpu, ref)
            if variant > 0:
                np.testing.assert_array_equal(out["refinements"].cpu().numpy(), ref["refinements"],
                                              err_msg=f"refinements, seed {seed}")
        finally:
            G.close()


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("rpw", [2, 5, 16])
def test_walkers_of_several_ranks_random(E, seed, rpw):
    rng = np.random.default_rng(2000 + seed)
    g = _random_graph(rng, int(rng.integers(2, 40)), int(rng.integers(5, 60)), int(rng.integers(0, 40)))
    sc = scenarios.draw(70, rng, bw_inter=(20000, 400000), bw_intra=(50000, 400000), alpha=(0, 20000),
                        ar_algo_random=True, slowdown=(65536, 150000), jitter=(5000, seed))
    try:
        ref = oracle.run(g, sc, 1, threads=THREADS)
    except oracle.OracleError as e:
        assert e.code == -4
        return
    G = E.Graph(g, 0, ranks_per_walker=rpw)
    assert_same(gpu_run(E, g, sc, 1, graph=G), ref)
    G.close()


@pytest.mark.parametrize("rpw", [2, 3])
def test_walkers_of_several_ranks_config1(E, rpw):
    g, sc = configs.graph(1), scenarios.take(configs.scenario_batch(4), slice(0, 130))
    G = E.Graph(g, 0, ranks_per_walker=rpw)
    assert_same(gpu_run(E, g, sc, 1, graph=G), oracle.run(g, sc, 1, threads=THREADS))
    G.close()


def test_1f1b_pipeline_closed_form(E):
    g = tinygraph.pipeline_1f1b(8, 16, 1000, 2100)
    sc = scenarios.default_scenarios(2)
    sc["alpha_ns"][:] = 0
    res = gpu_run(E, g, sc, 1)
    assert (res["step"] == (16 + 8 - 1) * 3100).all()


# ---------------------------------------------------------------- benchmark configurations
@pytest.mark.parametrize("R", [0, 1, 2])
def test_config1_tiny(E, R):
    g, sc = configs.graph(1), configs.scenario_batch(1)
    assert_same(gpu_run(E, g, sc, R), oracle.run(g, sc, R))


def test_config4_enumeration_4096(E):
    g, sc = configs.graph(4), configs.scenario_batch(4)
    assert_same(gpu_run(E, g, sc, 1), oracle.run(g, sc, 1, threads=THREADS))


def test_config2_gpt175b_96ranks(E):
    g, sc = configs.graph(2), configs.scenario_batch(2)
    ref = oracle.run(g, sc, 1, threads=THREADS)
    assert_same(gpu_run(E, g, sc, 1), ref)


def _sampled(E, g, sc, R, cols, *, digest=True):
    """Compose every scenario on the GPU; compare the sampled columns in full."""
    import torch
    G = E.Graph(g, 0)
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, R, timelines=True, digest=digest)
    idx = torch.tensor(cols, device=out["start"].device)
    gpu = {"step": out["step"].cpu().numpy(),
           "start": out["start"].index_select(1, idx).cpu().numpy(),
           "finish": out["finish"].index_select(1, idx).cpu().numpy()}
    if digest:
        gpu["digest"] = out["digest"].cpu().numpy().view(np.uint64)
    del out
    G.close()
    ref = oracle.run(g, scenarios.take(sc, cols), R, threads=min(THREADS, len(cols)))
    np.testing.assert_array_equal(gpu["step"][cols], ref["step"])
    if digest:
        np.testing.assert_array_equal(gpu["digest"][cols], ref["digest"])
    for j, c in enumerate(cols):
        np.testing.assert_array_equal(gpu["start"][:, j], ref["start"][j], err_msg=f"start, scenario {c}")
        np.testing.assert_array_equal(gpu["finish"][:, j], ref["finish"][j], err_msg=f"finish, scenario {c}")
    return gpu


def _stored(config, index, g, sc):
    """The oracle's step times and digests of every scenario (tests/golden), after
    checking that they were made from these very inputs."""
    from tests.golden import make_full_digests as fd
    h, step, dig = fd.load(config)[index]
    assert h == fd.input_hash(g, sc), \
        f"stored digests of config {config} graph {index} were made from other inputs: rerun {fd.__file__}"
    return step, dig


def _all_digests(E, g, sc, R):
    """Step time and digest of every scenario (digest variant, no timelines)."""
    G = E.Graph(g, 0)
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, R, timelines=False, digest=True)
    res = out["step"].cpu().numpy(), out["digest"].cpu().numpy().view(np.uint64)
    G.close()
    return res


def test_config3_gpt175b_1024ranks_sampled(E):
    """The benchmark's launch configuration (timelines out, no digest): every
    scenario's step time against the oracle's stored values, four scenarios'
    timelines in full against the oracle run here."""
    g, sc = configs.graph(3), configs.scenario_batch(3)
    n = scenarios.count(sc)
    step, _ = _stored(3, 0, g, sc)
    cols = sorted({0, n - 1, *np.random.default_rng(3).choice(n, 2, replace=False).tolist()})
    gpu = _sampled(E, g, sc, 1, cols, digest=False)
    np.testing.assert_array_equal(gpu["step"], step)
    assert (gpu["step"] > 0).all()


def test_config3_gpt175b_1024ranks_all_digests(E):
    g, sc = configs.graph(3), configs.scenario_batch(3)
    step, dig = _stored(3, 0, g, sc)
    gs, gd = _all_digests(E, g, sc, 1)
    np.testing.assert_array_equal(gs, step)
    np.testing.assert_array_equal(gd, dig)


def test_config3_every_pass_is_one_launch(E):
    """All 256 scenarios (four tiles) of the 1024-rank graph fit the device at once in
    every walk variant of a plain and a digest compose: a kernel that outgrew its register
    or LDS budget would split a pass into several launches and double its time."""
    import torch
    g = configs.graph(3)
    d, n = E.scenarios_to_device(configs.scenario_batch(3))
    G = E.Graph(g, 0)
    try:
        G.set_timing(True)
        for digest in (False, True):
            out = G.compose(d, n, 1, timelines=True, digest=digest)
            torch.cuda.synchronize()
            kinds = [k for k, _ in G.kernel_times()]
            assert kinds.count("walk") == 2, kinds
            del out
    finally:
        G.close()


# every graph of the extrapolation batch; graphs 6, 14 and 15 have 8192 ranks: more
# than the device holds wavefronts, so they are walked with several ranks per wavefront
@pytest.mark.parametrize("index", list(range(16)))
def test_config5_extrapolation_sampled(E, index):
    g, sc = configs.graph(5, index), configs.scenario_batch(5, index)
    step, dig = _stored(5, index, g, sc)
    gpu = _sampled(E, g, sc, 1, [0, scenarios.count(sc) - 1], digest=False)
    np.testing.assert_array_equal(gpu["step"], step)
    gs, gd = _all_digests(E, g, sc, 1)
    np.testing.assert_array_equal(gs, step)
    np.testing.assert_array_equal(gd, dig)


# ---------------------------------------------------------------- properties and edge cases
def test_batch_invariance(E):
    """A scenario composes to the same timeline alone or inside a wide batch."""
    g = configs.graph(1)
    sc = scenarios.draw(200, np.random.default_rng(9), bw_inter=(50000, 400000), slowdown=(65536, 91750),
                        jitter=(6554, 3), ar_algo_random=True)
    full = gpu_run(E, g, sc, 1)
    for cols in ([0], [199], [63, 64, 65], list(range(120, 200))):
        part = gpu_run(E, g, scenarios.take(sc, cols), 1)
        for j, c in enumerate(cols):
            np.testing.assert_array_equal(part["finish"][:, j], full["finish"][:, c])
            assert part["digest"][j] == full["digest"][c]


@pytest.mark.parametrize("n", [1, 63, 65, 127])
def test_ragged_scenario_counts(E, n):
    g = configs.graph(1)
    sc = scenarios.take(configs.scenario_batch(4), slice(0, n))
    assert_same(gpu_run(E, g, sc, 1), oracle.run(g, sc, 1, threads=THREADS))


def test_outputs_without_timelines(E):
    g = configs.graph(1)
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 100))
    a = gpu_run(E, g, sc, 1, timelines=False)
    ref = oracle.run(g, sc, 1, threads=THREADS, timelines=False)
    np.testing.assert_array_equal(a["step"], ref["step"])
    np.testing.assert_array_equal(a["digest"], ref["digest"])


def test_cc_costs_match_oracle(E):
    for cfg in (2, 4):
        g, sc = configs.graph(cfg), configs.scenario_batch(cfg)
        sc = scenarios.take(sc, slice(0, 64))
        G = E.Graph(g, 0)
        d, n = E.scenarios_to_device(sc)
        cost = G.cc_cost(d, n).cpu().numpy()
        G.close()
        ref = oracle.run(g, sc, 0, threads=THREADS, timelines=False, costs=True)
        np.testing.assert_array_equal(cost.T, ref["cost"])


def test_unfit_buffers_rejected_before_launch(E):
    """Output and scenario tensors that do not fit the call are refused on the host
    (no kernel sees them); the graph stays usable."""
    import torch
    g = configs.graph(1)
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 70))
    G = E.Graph(g, 0)
    try:
        d, n = E.scenarios_to_device(sc)
        dev = d.device
        small = torch.empty((G.n_ops, n - 1), dtype=torch.int64, device=dev)
        with pytest.raises(E.EchoError, match="start holds"):
            G.compose(d, n, 1, out={"start": small})
        with pytest.raises(E.EchoError, match="contiguous"):
            G.compose(d, n, 1, out={"finish": torch.empty((n, G.n_ops), dtype=torch.int64, device=dev).t()})
        with pytest.raises(E.EchoError, match="int64"):
            G.compose(d, n, 1, out={"step": torch.empty(n, dtype=torch.int32, device=dev)})
        with pytest.raises(E.EchoError, match="scenarios holds"):
            G.compose(d[: 192 * (n - 1)], n, 1)
        with pytest.raises(E.EchoError, match="scenarios is on"):
            G.compose(d.cpu(), n, 1)
        # the C ABI itself refuses the counts it cannot run (the binding checks them first)
        step = torch.empty(n, dtype=torch.int64, device=dev)
        for n_scen, n_refine in ((0, 1), (-1, 1), (n, -1), (n, 65)):
            rc = E.lib().echo_compose_batch(G.handle, d.data_ptr(), n_scen, n_refine, None, None,
                                            step.data_ptr(), None, None)
            assert rc == E.ECHO_ERR_ARG, (n_scen, n_refine, rc)
        rc = E.lib().echo_compose_batch(G.handle, None, n, 1, None, None, step.data_ptr(), None, None)
        assert rc == E.ECHO_ERR_ARG
        ref = oracle.run(g, sc, 1, threads=THREADS)
        assert_same(gpu_run(E, g, sc, 1, graph=G), ref)
    finally:
        G.close()


@pytest.mark.parametrize("until_stable", [False, True])
def test_compose_captured_in_a_hip_graph(E, until_stable):
    """After one eager call has sized the workspace, a compose call can be captured in a
    HIP graph: every replay (with eager work between replays) reproduces the eager
    outputs bit for bit."""
    import torch
    g = configs.graph(1)
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 130))
    G = E.Graph(g, 0)
    try:
        d, n = E.scenarios_to_device(sc)
        dev = d.device
        out = {"step": torch.empty(n, dtype=torch.int64, device=dev),
               "start": torch.empty((G.n_ops, n), dtype=torch.int64, device=dev),
               "finish": torch.empty((G.n_ops, n), dtype=torch.int64, device=dev),
               "digest": torch.empty(n, dtype=torch.int64, device=dev)}
        kw = dict(out=out, digest=True, check=False, until_stable=until_stable)
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            G.compose(d, n, 4, **kw)
        torch.cuda.synchronize()
        G.sync_status()
        ref = {k: v.clone() for k, v in out.items()}
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=s):
            G.compose(d, n, 4, **kw)
        for _ in range(3):
            for v in out.values():
                v.fill_(-1)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            for k in out:
                assert torch.equal(out[k], ref[k]), k
            assert out["start"].sum().item() == ref["start"].sum().item()     # eager work between
        G.sync_status()
        want = oracle.run(g, sc, 4, threads=THREADS, until_stable=until_stable)
        np.testing.assert_array_equal(ref["step"].cpu().numpy(), want["step"])
        np.testing.assert_array_equal(ref["digest"].cpu().numpy().view(np.uint64), want["digest"])
        del graph
    finally:
        G.close()


def test_graph_without_ops(E):
    g = Builder(4).graph()
    res = gpu_run(E, g, scenarios.default_scenarios(3), 1)
    assert (res["step"] == 0).all()


def test_single_member_collectives_and_empty_ranks(E):
    b = Builder(5, gpus_per_node=2)
    c = b.collective(AR, 5 << 20)
    d = b.collective(AG, 0)
    w = b.compute(1, 400)
    v = b.comm(1, c, preds=[w])
    b.compute(1, 30, preds=[v])
    b.comm(3, d)
    b.compute(3, 7)
    g = b.graph()
    sc = scenarios.default_scenarios(2)
    assert_same(gpu_run(E, g, sc, 1), oracle.run(g, sc, 1))


def test_out_of_range_scenario_reported(E):
    g = configs.graph(1)
    sc = scenarios.default_scenarios(4)
    sc["bw_inter_MBps"][2] = 0
    G = E.Graph(g, 0)
    d, n = E.scenarios_to_device(sc)
    with pytest.raises(E.EchoError) as x:
        G.compose(d, n, 1)
    assert x.value.code == E.ECHO_ERR_RANGE
    sc["bw_inter_MBps"][2] = 1000          # the graph stays usable afterwards
    d, n = E.scenarios_to_device(sc)
    G.compose(d, n, 1)
    G.close()


def test_time_limit_reported(E):
    big = (1 << 50) - 1
    b = Builder(2)
    c1, c2 = b.collective(AR, big), b.collective(AR, big)
    for r in range(2):
        b.comm(r, c1)
        b.comm(r, c2)
    sc = scenarios.default_scenarios(1)
    for k in ("bw_intra_MBps", "bw_inter_MBps", "reduce_MBps"):
        sc[k][:] = 1
    G = E.Graph(b.graph(), 0)
    d, n = E.scenarios_to_device(sc)
    with pytest.raises(E.EchoError) as x:
        G.compose(d, n, 0)
    assert x.value.code == E.ECHO_ERR_RANGE
    G.close()


# ---------------------------------------------------------------- DP-replica symmetry reduction
# One data-parallel replica composed alone (collectives costed at their whole
# group's size, barriers met by the members present) against the oracle, and
# against the GPU's own sweep over every replica.
from tests.test_oracle_pins import REPLICA_CASES, _replica_scen   # noqa: E402


def _replica_pair(params):
    g = gpt1f1b.gpt_graph(**params, replica_invariant=True)
    rg, op_map = gpt1f1b.dp_replica(g, params["tp"], params["dp"])
    return g, rg, op_map


def _full_vs_replica(E, g, rg, op_map, sc, R):
    """GPU sweep over all replicas and over one replica; the replica's rows must agree."""
    import torch
    d, n = E.scenarios_to_device(sc)
    Gf, Gr = E.Graph(g, 0), E.Graph(rg, 0)
    full = Gf.compose(d, n, R, timelines=True)
    red = Gr.compose(d, n, R, timelines=True)
    idx = torch.as_tensor(op_map, device=full["finish"].device)
    np.testing.assert_array_equal(full["step"].cpu().numpy(), red["step"].cpu().numpy())
    for key in ("start", "finish"):
        assert torch.equal(full[key].index_select(0, idx), red[key]), key
    Gf.close()
    Gr.close()
    return {"step": red["step"].cpu().numpy(), "start": red["start"].cpu().numpy(),
            "finish": red["finish"].cpu().numpy()}


@pytest.mark.parametrize("case", range(len(REPLICA_CASES)))
def test_dp_replica_small(E, case):
    g, rg, op_map = _replica_pair(REPLICA_CASES[case])
    sc = _replica_scen(case, 70)
    for R in (0, 1, 2):
        red = _full_vs_replica(E, g, rg, op_map, sc, R)
        assert_same(red, oracle.run(rg, sc, R, threads=THREADS))


def test_dp_replica_gpt175b_tp8pp4dp3(E):
    p = configs.graph_params(2)
    g, rg, op_map = _replica_pair(p)
    sc = configs.scenario_batch(2)
    red = _full_vs_replica(E, g, rg, op_map, sc, 1)
    assert_same(red, oracle.run(rg, sc, 1, threads=THREADS))


def test_dp_replica_gpt175b_8192_ranks(E):
    """GPT-175B TP8 x PP16 x DP64 (8192 ranks): the full sweep needs two ranks per
    wavefront; its DP replica has 128 ranks."""
    p = configs.graph_params(5, 15)
    g, rg, op_map = _replica_pair(p)
    sc = configs.scenario_batch(5, 15)
    red = _full_vs_replica(E, g, rg, op_map, sc, 1)
    cols = [0, scenarios.count(sc) - 1]
    ref = oracle.run(rg, scenarios.take(sc, cols), 1, threads=2)
    np.testing.assert_array_equal(red["step"][cols], ref["step"])
    for j, c in enumerate(cols):
        np.testing.assert_array_equal(red["finish"][:, c], ref["finish"][j])
        np.testing.assert_array_equal(red["start"][:, c], ref["start"][j])


# ---------------------------------------------------------------- validator variants
def _variant_run(E, g, sc, R, until_stable, prorate, graph=None):
    G = graph or E.Graph(g, 0)
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, R, timelines=True, digest=True, until_stable=until_stable, prorate=prorate,
                    refinements=True)
    res = {"step": out["step"].cpu().numpy(), "digest": out["digest"].cpu().numpy().view(np.uint64),
           "start": out["start"].cpu().numpy(), "finish": out["finish"].cpu().numpy(),
           "refinements": out["refinements"].cpu().numpy()}
    if graph is None:
        G.close()
    return res


VARIANTS = [(True, False), (False, True), (True, True)]


@pytest.mark.parametrize("until_stable,prorate", VARIANTS)
@pytest.mark.parametrize("seed", range(8))
def test_validator_variants_random_graphs(E, seed, until_stable, prorate):
    rng = np.random.default_rng(3000 + seed)
    g = _random_graph(rng, int(rng.integers(2, 14)), int(rng.integers(10, 60)), int(rng.integers(3, 30)))
    sc = scenarios.draw([1, 64, 70, 130][seed % 4], rng, bw_inter=(20000, 400000), alpha=(0, 20000),
                        slowdown=(65536, 300000), jitter=(4000, seed) if seed % 2 else None)
    try:
        ref = oracle.run(g, sc, 8, threads=THREADS, until_stable=until_stable, prorate=prorate)
    except oracle.OracleError as e:
        assert e.code == -4
        return
    gpu = _variant_run(E, g, sc, 8, until_stable, prorate)
    assert_same(gpu, ref)
    np.testing.assert_array_equal(gpu["refinements"], ref["refinements"])


@pytest.mark.parametrize("until_stable,prorate", VARIANTS)
def test_validator_variants_tiny(E, until_stable, prorate):
    sc = scenarios.draw(5, np.random.default_rng(21), bw_inter=(20000, 90000), alpha=(0, 5000),
                        slowdown=(65536, 200000))
    for name in sorted(TINY):
        g = TINY[name]
        ref = oracle.run(g, sc, 4, until_stable=until_stable, prorate=prorate)
        gpu = _variant_run(E, g, sc, 4, until_stable, prorate)
        assert_same(gpu, ref)
        np.testing.assert_array_equal(gpu["refinements"], ref["refinements"])


@pytest.mark.parametrize("seed", range(4))
def test_more_than_four_comm_streams(E, seed):
    """Ranks with up to seven comm streams (overlap detection's wide variant) under
    every validator."""
    rng = np.random.default_rng(7000 + seed)
    g = _random_graph(rng, int(rng.integers(2, 9)), int(rng.integers(60, 160)), int(rng.integers(12, 30)),
                      p_comm=0.15, comm_streams=7)
    per_rank = [len({int(s) for s, k, r in zip(g["op_stream"], g["op_kind"], g["op_rank"]) if k == 1 and r == q})
                for q in range(g["n_ranks"])]
    assert max(per_rank) > 4
    sc = scenarios.draw(70, rng, bw_inter=(20000, 400000), alpha=(0, 40000), slowdown=(65536, 196608),
                        jitter=(4000, seed) if seed % 2 else None)
    try:
        oracle.run(g, scenarios.take(sc, [0]), 0)
    except oracle.OracleError as e:
        assert e.code == -4
        return
    for R in (0, 2):
        assert_same(gpu_run(E, g, sc, R), oracle.run(g, sc, R, threads=THREADS))
    for until_stable, prorate in VARIANTS:
        ref = oracle.run(g, sc, 8, threads=THREADS, until_stable=until_stable, prorate=prorate)
        gpu = _variant_run(E, g, sc, 8, until_stable, prorate)
        assert_same(gpu, ref)
        np.testing.assert_array_equal(gpu["refinements"], ref["refinements"])


@pytest.mark.parametrize("prorate", [False, True])
@pytest.mark.parametrize("seed", range(4))
def test_fixed_point_with_strong_slowdowns(E, seed, prorate):
    """Long compute runs between sparse collectives and slowdowns up to 3x: ops move in
    and out of overlap from one refinement to the next (2 to 16 refinements), so blocks
    of ops that overlapped on the previous timeline are skipped whole by overlap
    detection on the next one, where returning to the plain duration is a change."""
    rng = np.random.default_rng(5000 + seed)
    g = _random_graph(rng, int(rng.integers(2, 9)), int(rng.integers(100, 200)), int(rng.integers(8, 24)),
                      p_comm=0.08)
    sc = scenarios.draw(130, rng, bw_inter=(20000, 400000), alpha=(0, 40000), slowdown=(65536, 196608),
                        jitter=(4000, seed) if seed % 2 else None)
    ref = oracle.run(g, sc, 16, threads=THREADS, until_stable=True, prorate=prorate)
    gpu = _variant_run(E, g, sc, 16, True, prorate)
    assert_same(gpu, ref)
    np.testing.assert_array_equal(gpu["refinements"], ref["refinements"])
    assert ref["refinements"].max() >= 3


@pytest.mark.parametrize("until_stable,prorate", VARIANTS)
def test_validator_variants_config1_and_2(E, until_stable, prorate):
    g, sc = configs.graph(1), scenarios.take(configs.scenario_batch(4), slice(0, 130))
    ref = oracle.run(g, sc, 10, threads=THREADS, until_stable=until_stable, prorate=prorate)
    gpu = _variant_run(E, g, sc, 10, until_stable, prorate)
    assert_same(gpu, ref)
    np.testing.assert_array_equal(gpu["refinements"], ref["refinements"])
    g, sc = configs.graph(2), configs.scenario_batch(2)
    cols = [0, 1, 2, 63]
    G = E.Graph(g, 0)
    gpu = _variant_run(E, g, sc, 10, until_stable, prorate, graph=G)
    G.close()
    ref = oracle.run(g, scenarios.take(sc, cols), 10, threads=4, until_stable=until_stable, prorate=prorate,
                     jitter_stream=cols)
    np.testing.assert_array_equal(gpu["refinements"][cols], ref["refinements"])
    np.testing.assert_array_equal(gpu["step"][cols], ref["step"])
    np.testing.assert_array_equal(gpu["digest"][cols], ref["digest"])
    for j, c in enumerate(cols):
        np.testing.assert_array_equal(gpu["finish"][:, c], ref["finish"][j])


def test_plain_refinement_reports_its_count(E):
    g, sc = configs.graph(1), scenarios.default_scenarios(3)
    res = _variant_run(E, g, sc, 3, False, False)
    assert (res["refinements"] == 3).all()
    assert_same(res, oracle.run(g, sc, 3))


def test_prorated_extra_time_limit_reported(E):
    """A prorated extra time of 2^32 ns or more does not fit its staging slot."""
    b = Builder(2)
    c = b.collective(AR, (1 << 50) - 1)
    lead = b.compute(0, 10, stream=2)
    b.comm(0, c, preds=[lead])
    b.compute(0, (1 << 40), cls=0)
    b.comm(1, c)
    sc = scenarios.default_scenarios(1)
    sc["slowdown_q16"][:] = 131072
    G = E.Graph(b.graph(), 0)
    d, n = E.scenarios_to_device(sc)
    with pytest.raises(E.EchoError) as x:
        G.compose(d, n, 1, prorate=True)
    assert x.value.code == E.ECHO_ERR_RANGE
    G.close()


# ---------------------------------------------------------------- CC model variants
def _mixed_cc_scenarios(sc, rng, n_tables):
    n = scenarios.count(sc)
    sc = dict(sc)
    sc["cc_model"] = (rng.random(n) < 0.3).astype(np.uint8)
    sc["cc_table"] = rng.integers(0, n_tables + 1, n).astype(np.int32)
    return sc


def test_cc_models_and_tables_costs(E):
    rng = np.random.default_rng(77)
    tables = scenarios.draw_cc_tables(3, rng)
    for cfg in (2, 4):
        g = configs.graph(cfg)
        sc = _mixed_cc_scenarios(scenarios.take(configs.scenario_batch(cfg), slice(0, 70)), rng, 3)
        G = E.Graph(g, 0)
        G.set_cc_tables(tables)
        d, n = E.scenarios_to_device(sc)
        cost = G.cc_cost(d, n).cpu().numpy()
        G.close()
        ref = oracle.run(g, sc, 0, threads=THREADS, timelines=False, costs=True, cc_tables=tables)
        np.testing.assert_array_equal(cost.T, ref["cost"])


def test_cc_models_and_tables_compose(E):
    rng = np.random.default_rng(78)
    tables = scenarios.draw_cc_tables(4, rng)
    g = configs.graph(1)
    sc = _mixed_cc_scenarios(scenarios.take(configs.scenario_batch(4), slice(0, 130)), rng, 4)
    G = E.Graph(g, 0)
    G.set_cc_tables(tables)
    assert_same(gpu_run(E, g, sc, 1, graph=G), oracle.run(g, sc, 1, threads=THREADS, cc_tables=tables))
    G.close()
    g, sc = configs.graph(2), _mixed_cc_scenarios(configs.scenario_batch(2), rng, 4)
    G = E.Graph(g, 0)
    G.set_cc_tables(tables)
    gpu = gpu_run(E, g, sc, 1, graph=G)
    G.close()
    cols = [0, 5, 63]
    ref = oracle.run(g, scenarios.take(sc, cols), 1, threads=3, cc_tables=tables, jitter_stream=cols)
    np.testing.assert_array_equal(gpu["step"][cols], ref["step"])
    np.testing.assert_array_equal(gpu["digest"][cols], ref["digest"])
    for j, c in enumerate(cols):
        np.testing.assert_array_equal(gpu["finish"][:, c], ref["finish"][j])


def test_cc_table_errors_reported(E):
    g = configs.graph(1)
    G = E.Graph(g, 0)
    bad = scenarios.draw_cc_tables(1, np.random.default_rng(1))
    bad[0, 1, 2] = 0                                   # chunk 0
    with pytest.raises(E.EchoError) as x:
        G.set_cc_tables(bad)
    assert x.value.code == E.ECHO_ERR_RANGE
    bad = scenarios.draw_cc_tables(1, np.random.default_rng(1))
    bad[0, 0, 5] = 0                                   # max_bytes decreases
    with pytest.raises(E.EchoError) as x:
        G.set_cc_tables(bad)
    assert x.value.code == E.ECHO_ERR_ARG
    G.set_cc_tables(scenarios.draw_cc_tables(2, np.random.default_rng(1)))
    sc = dict(scenarios.default_scenarios(3), cc_table=np.array([0, 2, 3], np.int32))   # table 3 is missing
    d, n = E.scenarios_to_device(sc)
    with pytest.raises(E.EchoError) as x:
        G.compose(d, n, 1)
    assert x.value.code == E.ECHO_ERR_RANGE
    G.set_cc_tables(None)
    sc = dict(scenarios.default_scenarios(2), cc_table=np.array([0, 1], np.int32))
    d, n = E.scenarios_to_device(sc)
    with pytest.raises(E.EchoError) as x:
        G.compose(d, n, 1)
    assert x.value.code == E.ECHO_ERR_RANGE
    G.close()


# ---------------------------------------------------------------- tree-ensemble slowdown
from workloads import slowdown_forest   # noqa: E402


@pytest.mark.parametrize("until_stable,prorate", [(False, False), (True, False), (False, True)])
@pytest.mark.parametrize("seed", range(6))
def test_forest_random_graphs(E, seed, until_stable, prorate):
    rng = np.random.default_rng(4000 + seed)
    g = _random_graph(rng, int(rng.integers(2, 14)), int(rng.integers(10, 60)), int(rng.integers(3, 30)))
    sc = scenarios.draw([1, 64, 70, 130][seed % 4], rng, bw_inter=(20000, 400000), bw_intra=(50000, 400000),
                        alpha=(0, 20000), ar_algo_random=True, jitter=(4000, seed) if seed % 2 else None)
    fo = slowdown_forest.synthetic_forest(seed)
    try:
        ref = oracle.run(g, sc, 6, threads=THREADS, until_stable=until_stable, prorate=prorate, forest=fo)
    except oracle.OracleError as e:
        assert e.code == -4
        return
    G = E.Graph(g, 0)
    G.set_forest(fo)
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, 6, timelines=True, digest=True, until_stable=until_stable, prorate=prorate,
                    forest=True, refinements=True)
    gpu = {"step": out["step"].cpu().numpy(), "digest": out["digest"].cpu().numpy().view(np.uint64),
           "start": out["start"].cpu().numpy(), "finish": out["finish"].cpu().numpy()}
    G.close()
    assert_same(gpu, ref)
    np.testing.assert_array_equal(out["refinements"].cpu().numpy(), ref["refinements"])


def test_forest_config1_and_2(E):
    fo = slowdown_forest.synthetic_forest(7)
    g, sc = configs.graph(1), scenarios.take(configs.scenario_batch(4), slice(0, 130))
    G = E.Graph(g, 0)
    G.set_forest(fo)
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, 2, timelines=True, digest=True, forest=True)
    G.close()
    gpu = {"step": out["step"].cpu().numpy(), "digest": out["digest"].cpu().numpy().view(np.uint64),
           "start": out["start"].cpu().numpy(), "finish": out["finish"].cpu().numpy()}
    assert_same(gpu, oracle.run(g, sc, 2, threads=THREADS, forest=fo))
    g, sc = configs.graph(2), configs.scenario_batch(2)
    G = E.Graph(g, 0)
    G.set_forest(fo)
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, 1, timelines=True, digest=True, forest=True)
    G.close()
    cols = [0, 31, 63]
    ref = oracle.run(g, scenarios.take(sc, cols), 1, threads=3, forest=fo, jitter_stream=cols)
    np.testing.assert_array_equal(out["step"].cpu().numpy()[cols], ref["step"])
    np.testing.assert_array_equal(out["digest"].cpu().numpy().view(np.uint64)[cols], ref["digest"])
    fin = out["finish"].cpu().numpy()
    for j, c in enumerate(cols):
        np.testing.assert_array_equal(fin[:, c], ref["finish"][j])


def test_forest_reproducing_the_table(E):
    g = configs.graph(1)
    rng = np.random.default_rng(12)
    table = rng.integers(65536, 200000, (8, 4)).astype(np.uint32)
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 70))
    sc["slowdown_q16"] = np.broadcast_to(table, (70, 8, 4)).copy()
    G = E.Graph(g, 0)
    G.set_forest(slowdown_forest.table_forest(table))
    d, n = E.scenarios_to_device(sc)
    a = G.compose(d, n, 2, timelines=True)
    b = G.compose(d, n, 2, timelines=True, forest=True)
    import torch
    assert torch.equal(a["finish"], b["finish"]) and torch.equal(a["start"], b["start"])
    G.close()


def test_forest_errors(E):
    g = configs.graph(1)
    G = E.Graph(g, 0)
    d, n = E.scenarios_to_device(scenarios.default_scenarios(2))
    with pytest.raises(E.EchoError) as x:            # no ensemble yet
        G.compose(d, n, 1, forest=True)
    assert x.value.code == E.ECHO_ERR_ARG
    deep = {"nodes": np.zeros(14, slowdown_forest.TREE_NODE_DTYPE), "roots": np.array([0], np.int32),
            "base": 65536, "class_metrics": np.zeros((8, 4), np.int64)}
    for i in range(13):
        deep["nodes"][i] = (0, i + 1, i + 1, 0, 1)
    deep["nodes"][13] = (-1, 0, 0, 5, 0)
    with pytest.raises(E.EchoError) as x:
        G.set_forest(deep)
    assert x.value.code == E.ECHO_ERR_ARG
    # nodes shared along every path: 13 nodes describe a full tree of depth 12 (8191 nodes
    # once laid out), and 8200 such trees pass the 2^26-node limit; the previous ensemble stays
    good = slowdown_forest.synthetic_forest(3, n_trees=8)
    G.set_forest(good)
    shared = {"nodes": np.zeros(13, slowdown_forest.TREE_NODE_DTYPE), "roots": np.zeros(8200, np.int32),
              "base": 65536, "class_metrics": np.zeros((8, 4), np.int64)}
    for i in range(12):
        shared["nodes"][i] = (i % 4, i + 1, i + 1, 0, 1000)
    shared["nodes"][12] = (-1, 0, 0, 7, 0)
    with pytest.raises(E.EchoError) as x:
        G.set_forest(shared)
    assert x.value.code == E.ECHO_ERR_RANGE
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 70))
    d, n = E.scenarios_to_device(sc)
    out = G.compose(d, n, 1, timelines=True, digest=True, forest=True)
    ref = oracle.run(g, sc, 1, threads=THREADS, forest=good)
    assert_same({"step": out["step"].cpu().numpy(), "digest": out["digest"].cpu().numpy().view(np.uint64),
                 "start": out["start"].cpu().numpy(), "finish": out["finish"].cpu().numpy()}, ref)
    G.close()


@pytest.mark.parametrize("ensemble", ["compact", "device"])
@pytest.mark.parametrize("knobs", ["uniform", "varied"])
def test_forest_walk_paths(E, ensemble, knobs):
    """Both ways the ensemble is walked, against the oracle: a 64-tree ensemble
    (about 11k nodes) fits the compact LDS form, a 128-tree one (about 23k) is walked
    from device memory; with the scenario knobs shared by every lane (only jitter and
    slowdown tables vary, as in the 1024-rank workload) the compact walk follows one
    path per wavefront wherever the lanes' features agree, with varied bandwidths and
    algorithms every lane walks its own."""
    fo = slowdown_forest.synthetic_forest(0, n_trees=64 if ensemble == "compact" else 128)
    assert (len(fo["nodes"]) + len(fo["roots"]) <= 12 * 1024) == (ensemble == "compact")
    rng = np.random.default_rng(77)
    graphs = [configs.graph(1), _random_graph(np.random.default_rng(5), 12, 40, 20)]
    for g in graphs:
        if knobs == "uniform":
            sc = scenarios.draw(130, rng, slowdown=(65536, 91750), jitter=(6554, 5))
        else:
            sc = scenarios.draw(130, rng, bw_inter=(20000, 400000), bw_intra=(50000, 400000), alpha=(0, 20000),
                                ar_algo_random=True, jitter=(4000, 9))
        for until_stable, prorate in [(False, False), (True, True)]:
            try:
                ref = oracle.run(g, sc, 4, threads=THREADS, until_stable=until_stable, prorate=prorate, forest=fo)
            except oracle.OracleError as e:
                assert e.code == -4
                continue
            G = E.Graph(g, 0)
            try:
                G.set_forest(fo)
                d, n = E.scenarios_to_device(sc)
                out = G.compose(d, n, 4, timelines=True, digest=True, until_stable=until_stable, prorate=prorate,
                                forest=True, refinements=True)
                gpu = {"step": out["step"].cpu().numpy(), "digest": out["digest"].cpu().numpy().view(np.uint64),
                       "start": out["start"].cpu().numpy(), "finish": out["finish"].cpu().numpy()}
                assert_same(gpu, ref)
                np.testing.assert_array_equal(out["refinements"].cpu().numpy(), ref["refinements"])
            finally:
                G.close()


def test_jittered_durations_beyond_32_bits(E):
    """Base durations on both sides of 2^32 ns (the jitter draw multiplies short ones in
    one 32-bit step) and up to the 2^43 limit, jittered with amplitudes up to 65535,
    through every pass: timelines against the oracle."""
    rng = np.random.default_rng(41)
    b = Builder(2)
    c = b.collective(AR, 1 << 20)
    for r in range(2):
        prev = []
        for k in range(40):
            d = int(rng.choice([rng.integers(1, 1 << 32), rng.integers(1 << 32, 1 << 42), (1 << 32) - 1, 1 << 32]))
            prev = [b.compute(r, d, preds=prev, cls=k % 8)]
        x = b.comm(r, c, preds=prev)
        b.compute(r, 1000, preds=[x])
    g = b.graph()
    sc = scenarios.draw(70, rng, slowdown=(65536, 91750), jitter=(6554, 3))
    sc["jitter_amp_q16"][::3] = 65535
    sc["jitter_amp_q16"][1::3] = 1
    assert_same(gpu_run(E, g, sc, 1), oracle.run(g, sc, 1))
