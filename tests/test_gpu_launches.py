"""GPU tests of the composer's launch layout and bounded waits, through the C ABI.

- A pass whose scenario tiles do not all fit one cooperative launch runs as
  several walk launches (each launch takes a range of tiles, every walker of
  a tile resident): results stay bit-identical to the oracle, both when the
  device's own capacity splits the pass and when the caller caps the tiles
  per launch.
- A tiny spin limit makes the bounded barrier waits give up: every kernel
  still runs to its end, the call reports ECHO_ERR_DEVICE, and the same graph
  composes bit-exactly again at the default limit.
- The walk-chain analysis runs on a graph resident on the GPU.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from tests.test_gpu_parity import THREADS, assert_same, gpu_run
from tests import tinygraph
from workloads import configs, gpt1f1b, scenarios

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2412_12487_amd as E
    E.lib()
    return E


def _gpt64():
    """A small GPT graph of 64 ranks (TP2 x PP4 x DP8, 4 layers, 4 microbatches): eight
    walk workgroups per scenario tile, P2P and data-parallel barriers across them."""
    return gpt1f1b.gpt_graph(n_layers=4, hidden=1024, seq=512, tp=2, pp=4, dp=8, microbatches=4, seed=11)


def _walk_launches_per_pass(G):
    passes = [[]]
    for kind, _ in G.kernel_times():
        if kind == "overlap":
            passes.append([])
        elif kind == "walk":
            passes[-1].append(kind)
    return [len(p) for p in passes]


def test_pass_split_by_device_capacity(E):
    """65 scenario tiles x 8 workgroups = 520 workgroups, more than the 512 an MI355X
    holds co-resident of the final (timeline-producing) walk variant, two
    eight-wavefront workgroups per compute unit: that pass runs as two launches (the
    lighter first pass may fit more workgroups per compute unit).  All step times
    and digests, and six scenarios' timelines (both launches' tiles and the ragged
    last one) against the oracle."""
    import torch
    g = _gpt64()
    n = 65 * 64 - 7
    sc = scenarios.draw(n, np.random.default_rng(21), bw_inter=(50_000, 400_000), alpha=(2_000, 20_000),
                        slowdown=(65536, 91750), ar_algo_random=True)
    G = E.Graph(g, 0)
    try:
        G.set_timing(True)
        d, n = E.scenarios_to_device(sc)
        out = G.compose(d, n, 1, timelines=True, digest=True)
        torch.cuda.synchronize()
        per_pass = _walk_launches_per_pass(G)
        assert len(per_pass) == 2 and per_pass[-1] == 2, per_pass
        cols = [0, 63, 64 * 64 - 1, 64 * 64, 64 * 64 + 5, n - 1]
        idx = torch.tensor(cols, device=out["start"].device)
        gpu = {"step": out["step"].cpu().numpy(), "digest": out["digest"].cpu().numpy().view(np.uint64),
               "start": out["start"].index_select(1, idx).cpu().numpy(),
               "finish": out["finish"].index_select(1, idx).cpu().numpy()}
        del out
    finally:
        G.close()
    ref = oracle.run(g, sc, 1, threads=THREADS, timelines=False)
    np.testing.assert_array_equal(gpu["step"], ref["step"])
    np.testing.assert_array_equal(gpu["digest"], ref["digest"])
    full = oracle.run(g, scenarios.take(sc, cols), 1, threads=len(cols), jitter_stream=cols)
    for j, c in enumerate(cols):
        np.testing.assert_array_equal(gpu["start"][:, j], full["start"][j], err_msg=f"start, scenario {c}")
        np.testing.assert_array_equal(gpu["finish"][:, j], full["finish"][j], err_msg=f"finish, scenario {c}")


@pytest.mark.parametrize("max_tiles", [1, 2])
@pytest.mark.parametrize("R", [0, 1, 2])
def test_pass_split_by_tile_cap(E, max_tiles, R):
    """Config 1 with 130 scenarios (three tiles, the last ragged) and at most one or
    two tiles per walk launch: every start, finish, step and digest."""
    import torch
    g = configs.graph(1)
    sc = scenarios.draw(130, np.random.default_rng(22), bw_inter=(50_000, 400_000), bw_intra=(50_000, 400_000),
                        alpha=(2_000, 20_000), slowdown=(65536, 91750), jitter=(6554, 7), ar_algo_random=True)
    G = E.Graph(g, 0)
    try:
        G.set_launch_tiles(max_tiles)
        G.set_timing(True)
        gpu = gpu_run(E, g, sc, R, graph=G)
        torch.cuda.synchronize()
        per_pass = _walk_launches_per_pass(G)
        assert per_pass == [-(-3 // max_tiles)] * (R + 1), per_pass
        assert_same(gpu, oracle.run(g, sc, R, threads=THREADS))
        G.set_launch_tiles(0)
        gpu_run(E, g, sc, R, graph=G)
        assert _walk_launches_per_pass(G) == [1] * (R + 1)
    finally:
        G.close()


@pytest.mark.parametrize("max_tiles", [2, 3])
def test_final_mask_variants_across_split_launches(E, max_tiles):
    """Config 1 with 520 scenarios (nine tiles, the last ragged), one refinement.  The final
    pass fetches only flagged mask rows when its launches average two tiles or more: at
    most three tiles per launch (3 + 3 + 3) it does, at most two (2 + 2 + 2 + 2 + 1) it
    fetches whole rows.  Both give every start, finish, step and digest of the oracle."""
    import torch
    g = configs.graph(1)
    sc = scenarios.draw(520, np.random.default_rng(23), bw_inter=(50_000, 400_000), bw_intra=(50_000, 400_000),
                        alpha=(2_000, 20_000), slowdown=(65536, 91750), jitter=(6554, 9), ar_algo_random=True)
    G = E.Graph(g, 0)
    try:
        G.set_launch_tiles(max_tiles)
        G.set_timing(True)
        gpu = gpu_run(E, g, sc, 1, graph=G)
        torch.cuda.synchronize()
        assert _walk_launches_per_pass(G) == [-(-9 // max_tiles)] * 2
        assert_same(gpu, oracle.run(g, sc, 1, threads=THREADS))
    finally:
        G.close()


def test_launch_tile_cap_rejects_negative(E):
    G = E.Graph(configs.graph(1), 0)
    try:
        with pytest.raises(E.EchoError) as x:
            G.set_launch_tiles(-1)
        assert x.value.code == E.ECHO_ERR_ARG
    finally:
        G.close()


def test_tiny_spin_limit_gives_up_every_wait_and_the_graph_recovers(E):
    """A 10 ns limit: a wait for collective members that outlasts its first clock
    check gives up at the next one (the pipeline's receives wait far longer), every
    other wait gives up on seeing the abort bit, every kernel runs to its end and the
    call reports ECHO_ERR_DEVICE; at the default limit the same graph composes
    bit-exactly again."""
    g = _gpt64()
    sc = scenarios.draw(130, np.random.default_rng(23), bw_inter=(50_000, 400_000), alpha=(2_000, 20_000),
                        slowdown=(65536, 91750), jitter=(6554, 9))
    G = E.Graph(g, 0)
    try:
        d, n = E.scenarios_to_device(sc)
        G.set_spin_limit(10)
        G.compose(d, n, 1, timelines=True, digest=True, check=False)
        with pytest.raises(E.EchoError) as x:
            G.sync_status()
        assert x.value.code == E.ECHO_ERR_DEVICE
        G.set_spin_limit(20 * 10**9)
        assert_same(gpu_run(E, g, sc, 1, graph=G), oracle.run(g, sc, 1, threads=THREADS))
        for bad in (0, 9, (1 << 40) + 1):
            with pytest.raises(E.EchoError) as y:
                G.set_spin_limit(bad)
            assert y.value.code == E.ECHO_ERR_ARG
    finally:
        G.close()


def test_walk_chain_of_a_resident_graph(E):
    g = configs.graph(1)
    G = E.Graph(g, 0)
    try:
        ch = G.walk_chain(1, 0, 0)
        per_rank = np.bincount(g["op_rank"], minlength=g["n_ranks"])
        comm_per_rank = np.bincount(g["op_rank"][g["op_kind"] == 1], minlength=g["n_ranks"])
        assert ch["items"] >= int((per_rank + comm_per_rank).max())
        assert ch["ps"] == ch["items"]
        ch2 = G.walk_chain(1000, 5000, 9000)
        assert ch2["ps"] == 1000 * ch2["items"] + 5000 * ch2["lds_barriers"] + 9000 * ch2["global_barriers"]
    finally:
        G.close()


def test_every_walk_variant_keeps_two_workgroups_per_cu(E):
    """The loader sizes walkers to the fewest co-resident walk workgroups of any kernel
    variant.  Every variant fits two eight-wavefront workgroups per compute unit, so a
    graph of 2 x 8 x 2 x CUs ranks (8192 on an MI355X) walks two ranks per wavefront, as
    when two are asked for, not three (one variant over 128 registers would make it three:
    every pass of the largest graphs would then take half as long again).  Each rank is a
    chain of three compute ops, so the walk's longest chain is 3 x ranks per wavefront."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    R = 2 * 8 * 2 * cus
    b = tinygraph.Builder(R)
    for r in range(R):
        u = b.compute(r, 1000 + r)
        u = b.compute(r, 2000, preds=(u,))
        b.compute(r, 3000, preds=(u,))
    g = b.graph()
    chains = {}
    for rpw in (0, 2, 3):
        G = E.Graph(g, 0, ranks_per_walker=rpw)
        try:
            chains[rpw] = G.walk_chain(1, 0, 0)["items"]
        finally:
            G.close()
    assert chains[2] == 6 and chains[3] == 9
    assert chains[0] == chains[2]


def test_library_loaded_before_torch_touches_the_gpu():
    """A fresh process that loads a graph before any torch call, then hands torch-allocated
    scenarios to it: the binding loads torch's HIP runtime before libecho.so, so both share
    one runtime, and the collective costs (a plain launch) match the oracle.  (The child
    runs no walk: once this process has made cooperative launches, the runtime refuses
    another process's on the same GPU.)"""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = (
        "import numpy as np, oracle\n"
        "import paper_2412_12487_amd as E\n"
        "from workloads import configs, scenarios\n"
        "g = configs.graph(2)\n"
        "G = E.Graph(g, 0)\n"
        "sc = scenarios.take(configs.scenario_batch(2), slice(0, 16))\n"
        "d, n = E.scenarios_to_device(sc)\n"
        "cost = G.cc_cost(d, n).cpu().numpy()\n"
        "ref = oracle.run(g, sc, 0, timelines=False, costs=True)\n"
        "assert np.array_equal(cost.T, ref['cost'])\n"
        "G.close()\n"
        "print('ok')\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=110)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
