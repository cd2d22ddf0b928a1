"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test ties one part of the oracle to something other than itself:
printed tables (chunk sizes), hand-worked values of Eq. 2-5, published
SplitMix64 outputs, brute-force longest paths on tiny graphs, the 1F1B
pipeline closed form, and structural invariants of any composed timeline.
"""
from __future__ import annotations

import itertools
import os

import numpy as np
import pytest

import oracle
from tests import bruteforce, tinygraph
from tests.tinygraph import AG, AR, P2P, RS, Builder
from workloads import configs, gpt1f1b, scenarios

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    out = []
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#")[0].strip()
        if line:
            out.append(line.split())
    return out


_ALIAS = {"alpha": "alpha_ns", "bw_intra": "bw_intra_MBps", "bw_inter": "bw_inter_MBps",
          "reduce": "reduce_MBps"}


def _scen(n=1, **kw):
    sc = scenarios.default_scenarios(n)
    for k, v in kw.items():
        k = _ALIAS.get(k, k)
        sc[k] = np.full_like(sc[k], v) if np.isscalar(v) else np.asarray(v, sc[k].dtype)
    return sc


# ---------------------------------------------------------------- CC estimator
@pytest.mark.parametrize("row", _rows("table6_chunk_sizes.txt"), ids=lambda r: r[0])
def test_chunk_size_table6(row):
    assert oracle.chunk_bytes(int(row[0])) == int(row[1])


@pytest.mark.parametrize("row", _rows("cc_costs.txt"), ids=lambda r: "-".join(r[:4]))
def test_cc_cost_hand_values(row):
    t, algo, S, N, M, K, alpha, bwa, bwe, red, want = map(int, row)
    got = oracle.cc_time(t, S, N, M, K, alpha=alpha, bw_intra=bwa, bw_inter=bwe, reduce=red, algo=algo)
    assert got == want


@pytest.mark.parametrize("S,N,M,K", [(4194304, 8, 1, 8), (26214400, 4, 4, 1), (50331648, 16, 2, 8),
                                     (123456789, 24, 3, 8), (1, 2, 2, 1)])
def test_ring_allreduce_is_reduce_scatter_plus_all_gather(S, N, M, K):
    """Eq. 4 (ring AR) carries 2(N-1) slow hops per round where Eq. 3 (ring RS)
    carries N-1, and Eq. 2 (ring AG) is exactly those N-1 hops: a ring all-reduce
    is a reduce-scatter plus an all-gather with one connection set-up, so
    T_AR = T_RS + T_AG - alpha.  A dropped or doubled term breaks this."""
    kw = dict(alpha=7000, bw_intra=300000, bw_inter=40000, reduce=150000)
    ar = oracle.cc_time(AR, S, N, M, K, **kw)
    rs = oracle.cc_time(RS, S, N, M, K, **kw)
    ag = oracle.cc_time(AG, S, N, M, K, **kw)
    assert ar == rs + ag - 7000


def test_cc_cost_monotone_in_knobs():
    base = dict(alpha=10000, bw_intra=400000, bw_inter=50000, reduce=160000)
    for t, algo in [(AR, 0), (AR, 1), (AG, 0), (RS, 0), (P2P, 0)]:
        for S, N, M, K in [(26214400, 8, 2, 4), (4194304, 8, 1, 8), (50331648, 2, 2, 1)]:
            if t == P2P and N != 2:
                continue
            t0 = oracle.cc_time(t, S, N, M, K, algo=algo, **base)
            assert oracle.cc_time(t, S, N, M, K, algo=algo, **dict(base, alpha=20000)) == t0 + 10000
            for knob in ("bw_intra", "bw_inter", "reduce"):
                assert oracle.cc_time(t, S, N, M, K, algo=algo, **dict(base, **{knob: base[knob] * 2})) <= t0
            assert oracle.cc_time(t, 2 * S, N, M, K, algo=algo, **base) >= t0


def test_time_limit_reported():
    """The largest single collective allowed by the input ranges stays below 2^62 ns,
    but two of them in a row do not: the composer reports a range error."""
    big = (1 << 50) - 1
    t = oracle.cc_time(AR, big, 4096, 512, 8, alpha=0, bw_intra=1, bw_inter=1, reduce=1)
    assert (1 << 61) < t < (1 << 62)
    b = Builder(2)
    c1, c2 = b.collective(AR, big), b.collective(AR, big)
    for r in range(2):
        b.comm(r, c1)
        b.comm(r, c2)
    g = b.graph()
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(g, _scen(1, bw_intra_MBps=1, bw_inter_MBps=1, reduce_MBps=1), 0)
    assert e.value.code == -2


# ---------------------------------------------------------------- fixed-point and jitter
@pytest.mark.parametrize("row", _rows("q16_worked.txt"), ids=lambda r: "-".join(r[:2]))
def test_q16_worked_values(row):
    d, f, want = map(int, row)
    assert oracle.q16(d, f) == want


@pytest.mark.parametrize("row", _rows("splitmix64_seed0.txt"), ids=lambda r: r[0])
def test_splitmix64_published_outputs(row):
    k, want = int(row[0]), int(row[1], 16)
    assert oracle.splitmix64_at(0, k) == want
    # the digest's mixing function is SplitMix64's output function
    golden = 0x9E3779B97F4A7C15
    assert oracle.mix64((k * golden) % (1 << 64)) == want


def _chain_graph(durs):
    b = Builder(1)
    prev = []
    for d in durs:
        prev = [b.compute(0, int(d), preds=prev)]
    return b.graph()


def test_jitter_amplitude_zero_is_identity_and_bounds_hold():
    durs = np.random.default_rng(5).integers(1, 200_000, 400)
    g = _chain_graph(durs)
    r = oracle.run(g, _scen(1), 0)
    assert r["step"][0] == durs.sum()
    A = 6554
    sc = _scen(3, jitter_amp_q16=A, jitter_seed=3)
    r = oracle.run(g, sc, 0)
    d = r["finish"] - r["start"]
    lo = np.floor(durs * (65536 - A) / 65536) - 1
    hi = np.ceil(durs * (65536 + A) / 65536) + 1
    assert (d >= lo).all() and (d <= hi).all()
    rel = (d / durs - 1.0)
    assert abs(rel.mean()) < 0.02 and rel.max() > 0.08 and rel.min() < -0.08
    assert not np.array_equal(d[0], d[1])          # each scenario has its own stream


def _jitter_rows():
    """Rows of jitter_worked.txt grouped by scenario and base duration: {(seed, stream, A, d0): {v: D}}."""
    groups = {}
    for r in _rows("jitter_worked.txt"):
        seed, stream, v, A, d0 = int(r[0], 16), int(r[1]), int(r[2]), int(r[3]), int(r[4])
        groups.setdefault((seed, stream, A, d0), {})[v] = int(r[11])
    return groups


@pytest.mark.parametrize("key", sorted(_jitter_rows()), ids=lambda k: "s%d-A%d-d%d" % (k[1], k[2], k[3]))
def test_jittered_durations_hand_worked(key):
    """D(v) of a three-op chain (ops v = 0, 1, 2, each of base duration d0) under a
    jittered scenario equals the values worked by hand from published SplitMix64
    outputs (the draw's sub-stream offset 2^36, k = v + 1, the high half of u and
    the 2A + 1 levels each change some of them)."""
    seed, stream, A, d0 = key
    want = _jitter_rows()[key]
    g = _chain_graph([d0] * 3)
    sc = _scen(1, jitter_amp_q16=A)
    sc["jitter_seed"] = np.array([seed], np.uint64)
    sc["jitter_stream"] = np.array([stream], np.uint32)
    r = oracle.run(g, sc, 0)
    got = (r["finish"][0] - r["start"][0]).tolist()
    assert got == [want[v] for v in range(3)]
    assert r["step"][0] == sum(want.values())


def test_jitter_table_refutes_plausible_slips():
    """Each plausible slip in the draw changes at least one hand-worked D: k = v
    instead of v + 1, the low instead of the high half of u, 2A instead of 2A + 1
    levels, a 2^32 instead of a 2^36 sub-stream offset (u computed here from the
    published generator definition; the table's u column is the published list)."""
    M = (1 << 64) - 1
    golden = 0x9E3779B97F4A7C15

    def mix(z):
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
        return z ^ (z >> 31)

    def draw(seed, stream, v, A, d0, k_off=1, low=False, levels=1, shift=36):
        u = mix((seed + ((stream << shift) + v + k_off) * golden) & M)
        x = (u & 0xFFFFFFFF) if low else (u >> 32)
        J = ((x * (2 * A + levels)) >> 32) - A
        return (d0 * (65536 + J) + 32768) >> 16

    rows = [(k, v, D) for k, vs in _jitter_rows().items() for v, D in vs.items()]
    assert all(draw(*k[:2], v, *k[2:]) == D for k, v, D in rows)     # the table is self-consistent
    for slip in (dict(k_off=0), dict(low=True), dict(levels=0), dict(shift=32)):
        assert any(draw(*k[:2], v, *k[2:], **slip) != D for k, v, D in rows), slip


# ---------------------------------------------------------------- composer vs brute force
def _dur_cost(g, sc, si=0):
    r = oracle.run(g, scenarios.take(sc, [si]), 0, costs=True, jitter_stream=[si])
    base = np.where(g["op_kind"] == 1, 0, r["finish"][0] - r["start"][0])
    return base, r["cost"][0]


def _tiny_cases():
    cases = {}
    b = Builder(1)
    a = b.compute(0, 5)
    b.compute(0, 7, preds=[a])
    cases["chain"] = b.graph()

    b = Builder(1)
    a = b.compute(0, 3)
    x = b.compute(0, 10, stream=1, preds=[a])
    y = b.compute(0, 4, stream=2, preds=[a])
    b.compute(0, 2, preds=[x, y])
    cases["diamond_streams"] = b.graph()

    b = Builder(4)
    c = b.collective(AR, 4 << 20)
    for r in range(4):
        w = b.compute(r, 1000 * (r + 1))
        v = b.comm(r, c, preds=[w])
        b.compute(r, 50, preds=[v])
    cases["skewed_allreduce"] = b.graph()

    b = Builder(2, gpus_per_node=1)
    c1 = b.collective(P2P, 1 << 20)
    c2 = b.collective(P2P, 1 << 20)
    w = b.compute(0, 300)
    b.comm(0, c1, stream=3, preds=[w])
    b.compute(0, 900, preds=[w])
    v = b.comm(0, c2, stream=4, preds=[w])
    b.compute(0, 40, preds=[v])
    x = b.compute(1, 700)
    y = b.comm(1, c1, stream=4, preds=[x])
    z = b.compute(1, 200, preds=[y])
    b.comm(1, c2, stream=3, preds=[z])
    cases["p2p_pair_two_servers"] = b.graph()

    b = Builder(3, gpus_per_node=2)
    c1 = b.collective(AR, 8 << 20)
    c2 = b.collective(RS, 30 << 20)
    c3 = b.collective(AG, 30 << 20)
    for r in range(3):
        w = b.compute(r, 100 * (3 - r), cls=r)
        v1 = b.comm(r, c1, stream=1, preds=[w])
        u = b.compute(r, 20000 + 7 * r, cls=0, preds=[w])
        v2 = b.comm(r, c2, stream=2, preds=[u])
        b.compute(r, 15000, cls=3, preds=[u])
        b.comm(r, c3, stream=2, preds=[v1])
        b.compute(r, 500, cls=4, preds=[v2])
    cases["three_collectives_overlap"] = b.graph()
    return cases


TINY = _tiny_cases()


@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("algo", [0, 1])
def test_composer_matches_path_enumeration(name, algo):
    g = TINY[name]
    sc = _scen(1, ar_algo=algo, bw_inter=60000, alpha=3000)
    base, cost = _dur_cost(g, sc)
    s, f = bruteforce.compose(g, base, cost)
    r = oracle.run(g, sc, 0)
    np.testing.assert_array_equal(r["start"][0], s)
    np.testing.assert_array_equal(r["finish"][0], f)


@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("n_refine", [1, 2])
def test_validator_matches_pairwise_overlap(name, n_refine):
    g = TINY[name]
    rng = np.random.default_rng(11)
    table = rng.integers(65536, 140000, (8, 4)).astype(np.uint32)
    sc = _scen(1, alpha=2500)
    sc["slowdown_q16"] = table[None].copy()
    base, cost = _dur_cost(g, sc)
    s, f = bruteforce.compose_validated(g, base, cost, table, n_refine)
    r = oracle.run(g, sc, n_refine)
    np.testing.assert_array_equal(r["start"][0], s)
    np.testing.assert_array_equal(r["finish"][0], f)


def test_skewed_collective_finishes_at_last_launch_plus_cost():
    g = TINY["skewed_allreduce"]
    sc = _scen(1)
    r = oracle.run(g, sc, 0, costs=True)
    T = 64565                        # 4 MiB ring AR on one server, default knobs (cc_costs.txt case A, N=8)
    T4 = oracle.cc_time(AR, 4 << 20, 4, 1, 4, alpha=10000, bw_intra=400000, bw_inter=50000, reduce=160000)
    assert r["cost"][0][0] == T4 and T4 < T
    comm = np.flatnonzero(g["op_kind"] == 1)
    assert (r["finish"][0][comm] == 4000 + T4).all()
    assert list(r["start"][0][comm]) == [1000, 2000, 3000, 4000]
    assert r["step"][0] == 4000 + T4 + 50


def test_random_small_dags_match_path_enumeration():
    rng = np.random.default_rng(123)
    for trial in range(40):
        n_ranks = int(rng.integers(1, 4))
        b = Builder(n_ranks, gpus_per_node=int(rng.integers(1, 3)))
        n_coll = int(rng.integers(0, 3))
        colls = [b.collective(int(rng.integers(0, 3)), int(rng.integers(0, 50 << 20))) for _ in range(n_coll)]
        for r in range(n_ranks):
            ids = []
            order = list(rng.permutation(n_coll))
            for k in range(int(rng.integers(2, 6))):
                preds = [int(u) for u in ids if rng.random() < 0.3]
                if order and rng.random() < 0.4:
                    ids.append(b.comm(r, colls[order.pop()], stream=int(rng.integers(1, 4)), preds=preds))
                else:
                    ids.append(b.compute(r, int(rng.integers(0, 5000)), stream=int(rng.integers(0, 2)),
                                         cls=int(rng.integers(0, 8)), preds=preds))
            for c in order:           # every rank joins every collective
                b.comm(r, colls[c], stream=int(rng.integers(1, 4)), preds=ids[-1:])
        g = b.graph()
        if len(g["op_rank"]) > 26:
            continue
        sc = _scen(1, ar_algo=trial % 2, alpha=int(rng.integers(0, 5000)))
        sc["slowdown_q16"] = rng.integers(65536, 100000, (1, 8, 4)).astype(np.uint32)
        try:
            base, cost = _dur_cost(g, sc)
        except oracle.OracleError as e:
            assert e.code == -4                               # oracle says deadlock ...
            with pytest.raises(bruteforce.Cycle):             # ... and the merged graph has a cycle
                bruteforce.compose(g, g["op_dur"], np.zeros(n_coll, np.int64))
            continue
        for R in (0, 1):
            s, f = bruteforce.compose_validated(g, base, cost, sc["slowdown_q16"][0], R)
            r = oracle.run(g, sc, R)
            np.testing.assert_array_equal(r["start"][0], s)
            np.testing.assert_array_equal(r["finish"][0], f)


# ---------------------------------------------------------------- closed forms
@pytest.mark.parametrize("P,m", [(1, 1), (1, 4), (2, 1), (2, 4), (3, 5), (4, 4), (4, 8), (8, 16)])
def test_1f1b_makespan_closed_form(P, m):
    """Uniform stages, free communication: a 1F1B step takes (m + P - 1)(t_f + t_b)."""
    tf, tb = 1000, 2100
    g = tinygraph.pipeline_1f1b(P, m, tf, tb)
    sc = _scen(1, alpha=0)
    r = oracle.run(g, sc, 0)
    assert r["step"][0] == (m + P - 1) * (tf + tb)
    if P <= 4 and m <= 8 and len(g["op_rank"]) <= 60:
        base, cost = _dur_cost(g, sc)
        assert (cost == 0).all()
        s, f = bruteforce.compose(g, base, cost)
        np.testing.assert_array_equal(r["finish"][0], f)


def test_single_collective_step_equals_its_cost():
    for t, S in [(AR, 4 << 20), (AG, 100 << 20), (RS, 3 << 20)]:
        b = Builder(8)
        c = b.collective(t, S)
        for r in range(8):
            b.comm(r, c)
        g = b.graph()
        r = oracle.run(g, _scen(1), 1, costs=True)
        assert r["step"][0] == r["cost"][0][0]
        assert (r["start"][0] == 0).all()


# ---------------------------------------------------------------- invariants on real-shaped graphs
def _check_invariants(g, r, si=0):
    s, f = r["start"][si], r["finish"][si]
    assert (s >= 0).all() and (f >= s).all()
    preds = bruteforce._preds(g) if len(g["op_rank"]) < 5000 else None
    n = len(g["op_rank"])
    # stream FIFO and explicit dependencies: s(v) >= f(u); non-comm s(v) = max pred f
    key = g["op_rank"].astype(np.int64) * 8 + g["op_stream"]
    order = np.lexsort((np.arange(n), key))
    same = key[order][1:] == key[order][:-1]
    assert (s[order][1:][same] >= f[order][:-1][same]).all()
    src = np.repeat(np.arange(n), np.diff(g["pred_off"]))
    assert (s[src] >= f[g["pred_idx"]]).all()
    comm = g["op_kind"] == 1
    cf = {}
    for v in np.flatnonzero(comm):
        cf.setdefault(int(g["op_coll"][v]), set()).add(int(f[v]))
    assert all(len(x) == 1 for x in cf.values())
    assert r["step"][si] == f.max()
    if preds is not None:
        for v in range(n):
            want = max([f[u] for u in preds[v]], default=0)
            assert s[v] == want


def test_invariants_config1():
    g = configs.graph(1)
    sc = configs.scenario_batch(4)
    sub = scenarios.take(sc, slice(0, 8))
    for R in (0, 1, 2):
        r = oracle.run(g, sub, R, threads=4)
        for si in range(8):
            _check_invariants(g, r, si)


def test_all_unit_factors_make_refinement_a_no_op():
    g = configs.graph(1)
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 4))
    sc["slowdown_q16"][:] = 65536
    r0 = oracle.run(g, sc, 0, threads=4)
    r1 = oracle.run(g, sc, 1, threads=4)
    for k in ("start", "finish", "step", "digest"):
        np.testing.assert_array_equal(r0[k], r1[k])


def test_refinement_never_shortens_the_step():
    """q16(d, F) >= d for F >= 1.0, so the validated step is at least the
    interference-free critical path; with gradient buckets overlapping later
    layers' backward kernels it is strictly longer."""
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 8))
    g = configs.graph(1)
    r0 = oracle.run(g, sc, 0, threads=4, timelines=False)
    r1 = oracle.run(g, sc, 1, threads=4, timelines=False)
    assert (r1["step"] >= r0["step"]).all()
    g = gpt1f1b.gpt_graph(n_layers=8, hidden=1024, seq=512, tp=2, pp=2, dp=2, microbatches=4, seed=0)
    r0 = oracle.run(g, sc, 0, threads=4, timelines=False)
    r1 = oracle.run(g, sc, 1, threads=4, timelines=False)
    r2 = oracle.run(g, sc, 2, threads=4, timelines=False)
    assert (r1["step"] > r0["step"]).all() and (r2["step"] >= r0["step"]).all()


@pytest.mark.parametrize("knob,direction", [("bw_intra_MBps", -1), ("bw_inter_MBps", -1),
                                             ("reduce_MBps", -1), ("alpha_ns", +1)])
def test_step_monotone_in_network_knobs_without_interference(knob, direction):
    g = configs.graph(1, 0)
    g = dict(g, gpus_per_node=2)          # spread the 8 ranks over 4 servers
    vals = [2_000, 9_000, 50_000, 120_000, 400_000]
    sc = _scen(len(vals))
    sc[knob] = np.array(vals, np.int64)
    r = oracle.run(g, sc, 0, threads=4, timelines=False)
    steps = r["step"]
    assert (np.diff(steps) * direction >= 0).all()
    assert steps[0] != steps[-1]


def test_renumbering_servers_keeps_every_op_time():
    g = dict(configs.graph(1), gpus_per_node=2)
    sc = scenarios.take(configs.scenario_batch(4), slice(0, 4))
    sc["jitter_amp_q16"][:] = 0
    perm = [2, 0, 3, 1]                    # server i -> perm[i]
    gpn = 2
    new_rank = np.array([perm[r // gpn] * gpn + r % gpn for r in range(8)])
    old_rank_of = np.argsort(new_rank)
    old_ids = np.concatenate([np.flatnonzero(g["op_rank"] == old_rank_of[r]) for r in range(8)])
    new_id = np.empty_like(old_ids)
    new_id[old_ids] = np.arange(len(old_ids))
    pc = np.diff(g["pred_off"])[old_ids]
    pred_lists = [g["pred_idx"][g["pred_off"][v]:g["pred_off"][v + 1]] for v in old_ids]
    h = dict(g)
    for k in ("op_stream", "op_kind", "op_class", "op_dur", "op_coll"):
        h[k] = g[k][old_ids]
    h["op_rank"] = new_rank[g["op_rank"][old_ids]].astype(np.int32)
    h["pred_off"] = np.concatenate([[0], np.cumsum(pc)]).astype(np.int64)
    h["pred_idx"] = np.concatenate([new_id[p] for p in pred_lists]).astype(np.int32)
    a = oracle.run(g, sc, 1, threads=4)
    b = oracle.run(h, sc, 1, threads=4)
    np.testing.assert_array_equal(a["start"][:, old_ids], b["start"])
    np.testing.assert_array_equal(a["finish"][:, old_ids], b["finish"])
    np.testing.assert_array_equal(a["step"], b["step"])


def test_scenario_alone_equals_scenario_in_batch():
    g = configs.graph(1)
    sc = configs.scenario_batch(3)      # jittered scenarios
    full = oracle.run(configs.graph(1), scenarios.take(sc, slice(0, 6)), 1, threads=3)
    for si in (0, 5):
        one = oracle.run(g, scenarios.take(sc, [si]), 1, jitter_stream=[si])
        np.testing.assert_array_equal(one["finish"][0], full["finish"][si])
        assert one["digest"][0] == full["digest"][si]


def test_digest_is_sum_of_mixed_op_records():
    g = TINY["three_collectives_overlap"]
    r = oracle.run(g, _scen(1), 1)
    s, f = r["start"][0], r["finish"][0]
    want = 0
    for v in range(len(s)):
        want = (want + oracle.mix64(oracle.mix64(v ^ int(s[v])) ^ int(f[v]))) % (1 << 64)
    assert int(r["digest"][0]) == want


# ---------------------------------------------------------------- error behaviour
def test_deadlock_detected():
    b = Builder(2)
    c1, c2 = b.collective(AR, 1024), b.collective(AR, 1024)
    b.comm(0, c1, stream=1)
    b.comm(0, c2, stream=1)
    b.comm(1, c2, stream=1)
    b.comm(1, c1, stream=1)
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(b.graph(), _scen(1), 0)
    assert e.value.code == -4


@pytest.mark.parametrize("mutate,code", [
    (lambda g: g["pred_idx"].__setitem__(0, 5), -1),       # dependency on a later op
    (lambda g: g["op_dur"].__setitem__(0, 1 << 43), -2),  # duration out of range
    (lambda g: g["coll_bytes"].__setitem__(0, 1 << 50), -2),
    (lambda g: g["op_stream"].__setitem__(0, 8), -1),
    (lambda g: g["op_coll"].__setitem__(0, 0), -1),        # compute op naming a collective
])
def test_bad_graphs_rejected(mutate, code):
    g = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in TINY["skewed_allreduce"].items()}
    mutate(g)
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(g, _scen(1), 0)
    assert e.value.code == code


def test_bad_scenarios_rejected():
    g = TINY["chain"]
    for k, v in [("bw_inter_MBps", 0), ("reduce_MBps", 0), ("alpha_ns", -1), ("jitter_amp_q16", 65536)]:
        with pytest.raises(oracle.OracleError) as e:
            oracle.run(g, _scen(1, **{k: v}), 0)
        assert e.value.code == -2
    sc = _scen(1)
    sc["slowdown_q16"][0, 3, 1] = 65535
    with pytest.raises(oracle.OracleError):
        oracle.run(g, sc, 0)


def test_all_benchmark_graphs_small_enough_compose():
    for cfg in (1, 4):
        g = configs.graph(cfg)
        r = oracle.run(g, scenarios.take(configs.scenario_batch(cfg), slice(0, 2)), 1, timelines=False)
        assert (r["step"] > 0).all()


# ---------------------------------------------------------------- DP-replica symmetry reduction
# Sec. 8.5 (DDP mode): one copy of the workload per DP group.  Simulating one
# replica, with every collective costed at its whole group's size and its
# barrier met by the members present, must reproduce the sweep over all
# replicas op for op when every replica has the same durations.
REPLICA_CASES = [
    dict(configs.TINY, tp=2, pp=2, dp=2, microbatches=4, seed=0),
    dict(configs.TINY, tp=2, pp=2, dp=4, microbatches=3, seed=1, gpus_per_node=2),   # DP groups span servers
    dict(configs.TINY | dict(n_layers=4), tp=1, pp=4, dp=3, microbatches=4, seed=2, gpus_per_node=1),
    dict(configs.TINY, tp=2, pp=2, dp=3, microbatches=2, seed=3, distopt=True, gpus_per_node=2),   # RS + AG
]


def _replica_scen(seed, n=6):
    return scenarios.draw(n, np.random.default_rng(seed), bw_inter=(20000, 400000), bw_intra=(50000, 400000),
                          alpha=(0, 20000), ar_algo_random=True, slowdown=(65536, 150000))


@pytest.mark.parametrize("case", range(len(REPLICA_CASES)))
def test_dp_replica_equals_full_sweep(case):
    p = REPLICA_CASES[case]
    g = gpt1f1b.gpt_graph(**p, replica_invariant=True)
    rg, op_map = gpt1f1b.dp_replica(g, p["tp"], p["dp"])
    assert len(rg["op_rank"]) * p["dp"] == len(g["op_rank"])
    # precondition: the replicas are copies of each other, placement (hence costs) included
    for k in range(1, p["dp"]):
        rk, _ = gpt1f1b.dp_replica(g, p["tp"], p["dp"], replica=k)
        for key, val in rg.items():
            np.testing.assert_array_equal(np.asarray(rk[key]), np.asarray(val), err_msg=key)
    sc = _replica_scen(case)
    for R in (0, 1, 2):
        full, red = oracle.run(g, sc, R), oracle.run(rg, sc, R)
        np.testing.assert_array_equal(full["step"], red["step"])
        np.testing.assert_array_equal(full["start"][:, op_map], red["start"])
        np.testing.assert_array_equal(full["finish"][:, op_map], red["finish"])
    # every replica runs the same timeline
    for k in range(1, p["dp"]):
        _, m_k = gpt1f1b.dp_replica(g, p["tp"], p["dp"], replica=k)
        np.testing.assert_array_equal(full["finish"][:, m_k], red["finish"])


def test_dp_replica_of_asymmetric_placement_differs():
    """Replicas placed differently (a pipeline hop inside a server for one replica,
    across servers for another) are not copies: the reduction does not apply."""
    p = dict(configs.TINY | dict(n_layers=4), tp=1, pp=4, dp=3, microbatches=4, seed=2, gpus_per_node=4)
    g = gpt1f1b.gpt_graph(**p, replica_invariant=True)
    r0, _ = gpt1f1b.dp_replica(g, 1, 3, replica=0)
    r1, _ = gpt1f1b.dp_replica(g, 1, 3, replica=1)
    assert (r0["coll_M"] != r1["coll_M"]).any()
    sc = _replica_scen(2)
    assert (oracle.run(g, sc, 1)["step"] != oracle.run(r0, sc, 1)["step"]).any()


def test_dp_replica_needs_the_whole_group_membership():
    """Costing the replica's collectives at their local size (or drawing durations per
    replica) changes the result: the reduction is exact only as specified."""
    p = REPLICA_CASES[1]
    g = gpt1f1b.gpt_graph(**p, replica_invariant=True)
    rg, op_map = gpt1f1b.dp_replica(g, p["tp"], p["dp"])
    sc = _replica_scen(11)
    full = oracle.run(g, sc, 1)
    local = {k: v for k, v in rg.items() if k not in ("coll_N", "coll_M", "coll_K")}
    assert (oracle.run(local, sc, 1)["step"] != full["step"]).any()
    g2 = gpt1f1b.gpt_graph(**p)                       # durations differ between replicas
    rg2, _ = gpt1f1b.dp_replica(g2, p["tp"], p["dp"])
    assert (oracle.run(rg2, sc, 1)["step"] != oracle.run(g2, sc, 1)["step"]).any()


@pytest.mark.parametrize("bad", [dict(N=0), dict(M=0), dict(K=0), dict(MK=True), dict(P2P=3)])
def test_inconsistent_group_membership_rejected(bad):
    p = REPLICA_CASES[0]
    rg, _ = gpt1f1b.dp_replica(gpt1f1b.gpt_graph(**p, replica_invariant=True), p["tp"], p["dp"])
    rg = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in rg.items()}
    c = int(np.flatnonzero(rg["coll_type"] != P2P)[0])
    if "N" in bad:
        rg["coll_N"][c] = 0
    if "M" in bad:
        rg["coll_M"][c] = 0
    if "K" in bad:
        rg["coll_K"][c] = 0
    if "MK" in bad:
        rg["coll_N"][c], rg["coll_M"][c], rg["coll_K"][c] = 8, 2, 3
    if "P2P" in bad:
        q = int(np.flatnonzero(rg["coll_type"] == P2P)[0])
        rg["coll_N"][q], rg["coll_M"][q], rg["coll_K"][q] = 3, 1, 3
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(rg, scenarios.default_scenarios(1), 1)
    assert e.value.code == -1


# ---------------------------------------------------------------- validator variants
# Sec. 3 / Sec. 6 give no iteration rule: besides R fixed refinements, refine until
# the durations stop changing, and/or inflate only the overlapped part of an op.
@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("until_stable,prorate", [(True, False), (False, True), (True, True)])
def test_validator_variants_match_brute_force(name, until_stable, prorate):
    g = TINY[name]
    rng = np.random.default_rng(13)
    table = rng.integers(65536, 200000, (8, 4)).astype(np.uint32)
    sc = _scen(1, alpha=2500)
    sc["slowdown_q16"] = table[None].copy()
    base, cost = _dur_cost(g, sc)
    s, f, done = bruteforce.compose_variants(g, base, cost, table, 4, until_stable=until_stable, prorate=prorate)
    r = oracle.run(g, sc, 4, until_stable=until_stable, prorate=prorate)
    np.testing.assert_array_equal(r["start"][0], s)
    np.testing.assert_array_equal(r["finish"][0], f)
    assert r["refinements"][0] == done


def _overlap_pair(comm_start, comp_dur, coll_bytes):
    """Rank 0: a compute op (stream 0) and an all-reduce (stream 1) launched after a
    lead-in op of comm_start ns; rank 1 joins the all-reduce at once."""
    b = Builder(2)
    c = b.collective(AR, coll_bytes)
    lead = b.compute(0, comm_start, stream=2)
    b.comm(0, c, preds=[lead])
    v = b.compute(0, comp_dur, cls=3)
    b.comm(1, c)
    return b.graph(), v


def test_prorated_inflation_hand_value():
    """A 1000 ns compute op starting at 0, with an all-reduce running from 700 ns on:
    300 ns overlap; prorated d' = 700 + q16(300, F), whole-op d' = q16(1000, F)."""
    g, v = _overlap_pair(700, 1000, 1 << 20)
    sc = _scen(1)
    F = 98304                                   # 1.5
    sc["slowdown_q16"][:] = F
    whole = oracle.run(g, sc, 1)
    part = oracle.run(g, sc, 1, prorate=True)
    assert whole["finish"][0][v] == (1000 * F + 32768) >> 16 == 1500
    assert part["finish"][0][v] == 700 + ((300 * F + 32768) >> 16) == 1150


def test_prorating_a_fully_overlapped_op_equals_whole_inflation():
    g, v = _overlap_pair(0, 1000, 1 << 30)      # the all-reduce outlasts the compute op
    sc = _scen(1)
    sc["slowdown_q16"][:] = 80000
    assert oracle.run(g, sc, 1, prorate=True)["finish"][0][v] == oracle.run(g, sc, 1)["finish"][0][v]


def test_until_stable_equals_fixed_refinements_it_reports():
    """The result after `refinements` rounds is the fixed point: plain refinement with that
    many rounds, or one more, gives the same timeline."""
    g = configs.graph(1)
    sc = scenarios.draw(6, np.random.default_rng(17), bw_inter=(20000, 90000), slowdown=(65536, 200000),
                        jitter=(6554, 1))
    for prorate in (False, True):
        r = oracle.run(g, sc, 8, until_stable=True, prorate=prorate)
        assert (r["refinements"] >= 1).all()
        for j in range(6):
            k = int(r["refinements"][j])
            one = scenarios.take(sc, [j])
            for R in ({k, k + 1} if k < 8 else {k}):
                fixed = oracle.run(g, one, R, prorate=prorate, jitter_stream=[j])
                np.testing.assert_array_equal(fixed["finish"][0], r["finish"][j])


def test_random_small_dags_validator_variants():
    """Random tiny graphs with overlapping comm ops: the fixed-point and prorated validators
    against brute force (per-nanosecond coverage, repeated full path enumeration)."""
    rng = np.random.default_rng(321)
    deep = 0
    for trial in range(60):
        n_ranks = int(rng.integers(1, 4))
        b = Builder(n_ranks, gpus_per_node=int(rng.integers(1, 3)))
        n_coll = int(rng.integers(1, 4))
        colls = [b.collective(int(rng.integers(0, 3)), int(rng.integers(0, 256 << 10))) for _ in range(n_coll)]
        for r in range(n_ranks):
            ids = []
            order = list(rng.permutation(n_coll))
            for k in range(int(rng.integers(3, 7))):
                preds = [int(u) for u in ids if rng.random() < 0.25]
                if order and rng.random() < 0.4:
                    ids.append(b.comm(r, colls[order.pop()], stream=int(rng.integers(1, 4)), preds=preds))
                else:
                    ids.append(b.compute(r, int(rng.integers(1, 600)), stream=int(rng.integers(0, 2)),
                                         cls=int(rng.integers(0, 8)), preds=preds))
            for c in order:
                b.comm(r, colls[c], stream=int(rng.integers(1, 4)), preds=ids[-1:])
        g = b.graph()
        if len(g["op_rank"]) > 24:
            continue
        sc = _scen(1, alpha=int(rng.integers(0, 300)), bw_intra=400000, bw_inter=200000)
        sc["slowdown_q16"] = rng.integers(65536, 260000, (1, 8, 4)).astype(np.uint32)
        try:
            base, cost = _dur_cost(g, sc)
        except oracle.OracleError as e:
            assert e.code == -4
            continue
        for until_stable, prorate in ((True, False), (False, True), (True, True)):
            s, f, done = bruteforce.compose_variants(g, base, cost, sc["slowdown_q16"][0], 6,
                                                     until_stable=until_stable, prorate=prorate)
            r = oracle.run(g, sc, 6, until_stable=until_stable, prorate=prorate)
            np.testing.assert_array_equal(r["start"][0], s)
            np.testing.assert_array_equal(r["finish"][0], f)
            assert r["refinements"][0] == done
            deep += until_stable and done >= 2
    assert deep >= 5          # the fixed point is often reached only after several rounds


# ---------------------------------------------------------------- CC model variants
_AB = dict(alpha=10000, bw_intra=400000, bw_inter=50000, reduce=160000)


def _table_from_bandwidths(alpha_ns, bw_intra_MBps, bw_inter_MBps, reduce_MBps):
    """The CC parameter table holding what a table-less scenario with these knobs
    uses (reading 11): Table 6 bands and chunks, per-chunk times
    ceil(chunk * 1000 / bandwidth), alpha and the reduce throughput as given."""
    cdiv = lambda a, b: -(-a // b)
    chunk = scenarios.TABLE6_CHUNK
    return scenarios.cc_table(chunk=chunk, alpha=alpha_ns, beta=cdiv(chunk * 1000, bw_intra_MBps),
                              gamma=cdiv(chunk * 1000, bw_inter_MBps), reduce=reduce_MBps)


@pytest.mark.parametrize("row", _rows("cc_alpha_beta.txt"), ids=lambda r: "-".join(r[:5]))
def test_alpha_beta_hand_values(row):
    t, algo, S, N, M, K, want = (int(x) for x in row)
    assert oracle.cc_time(t, S, N, M, K, algo=algo, cc_model=1, **_AB) == want


@pytest.mark.parametrize("S,N,M", [(1, 2, 1), (4 << 20, 8, 1), (5 << 20, 16, 2), (300 << 20, 64, 8), (12345, 3, 3)])
def test_alpha_beta_ring_allreduce_is_reduce_scatter_plus_all_gather(S, N, M):
    K = -(-N // M)
    ar = oracle.cc_time(0, S, N, M, K, cc_model=1, **_AB)
    assert ar == oracle.cc_time(2, S, N, M, K, cc_model=1, **_AB) + oracle.cc_time(1, S, N, M, K, cc_model=1, **_AB)


def test_cc_table_equal_to_bandwidth_parameters_reproduces_every_cost():
    rng = np.random.default_rng(8)
    for _ in range(200):
        kn = dict(alpha=int(rng.integers(0, 30000)), bw_intra=int(rng.integers(1000, 500000)),
                  bw_inter=int(rng.integers(1000, 500000)), reduce=int(rng.integers(1000, 500000)))
        table = _table_from_bandwidths(kn["alpha"], kn["bw_intra"], kn["bw_inter"], kn["reduce"])
        S = int(rng.choice([0, 1, 4 << 20, (4 << 20) + 1, 16 << 20, (128 << 20) + 7, 1 << 30,
                            int(rng.integers(0, 1 << 31))]))
        N = int(rng.integers(1, 300))
        M = int(rng.integers(1, N + 1))
        K = -(-N // M)
        for t in range(4):
            if t == 3 and N != 2:
                continue
            for algo in (0, 1):
                assert oracle.cc_time(t, S, N, M, K, algo=algo, table=table, **kn) == \
                    oracle.cc_time(t, S, N, M, K, algo=algo, **kn)


def test_cc_table_row_selection_hand_values():
    """Rows serve S up to their bound; the last row every larger S.  P2P inside one server:
    alpha_row + ceil(S / chunk_row) * beta_row."""
    table = scenarios.cc_table(chunk=np.arange(1, 8) * 1000, alpha=np.arange(1, 8) * 100,
                               beta=np.arange(1, 8) * 10, gamma=np.arange(1, 8) * 50, reduce=100000)
    p2p = lambda S: oracle.cc_time(3, S, 2, 1, 2, table=table, **_AB)
    assert p2p(4 << 20) == 100 + 4195 * 10                 # row 0: ceil(4194304 / 1000) = 4195
    assert p2p((4 << 20) + 1) == 200 + 2098 * 20           # row 1: ceil(4194305 / 2000) = 2098
    assert p2p(300 << 20) == 700 + 44939 * 70              # past the last bound: row 6, ceil(314572800 / 7000)
    # across servers the hop is gamma
    assert oracle.cc_time(3, 1000, 2, 2, 1, table=table, **_AB) == 100 + 1 * 50


def test_compose_with_cc_tables_and_models():
    """A scenario whose table equals its bandwidth parameters composes exactly like the
    table-less scenario; the alpha-beta model changes the result."""
    g = configs.graph(1)
    sc = scenarios.draw(4, np.random.default_rng(31), bw_inter=(20000, 90000), bw_intra=(50000, 400000),
                        alpha=(0, 9000), ar_algo_random=True)
    tables = np.stack([_table_from_bandwidths(int(sc["alpha_ns"][i]), int(sc["bw_intra_MBps"][i]),
                                                          int(sc["bw_inter_MBps"][i]), int(sc["reduce_MBps"][i]))
                       for i in range(4)])
    plain = oracle.run(g, sc, 1)
    via = dict(sc, cc_table=np.arange(1, 5, dtype=np.int32))
    r = oracle.run(g, via, 1, cc_tables=tables)
    np.testing.assert_array_equal(r["finish"], plain["finish"])
    ab = oracle.run(g, dict(sc, cc_model=np.ones(4, np.uint8)), 1)
    assert (ab["step"] != plain["step"]).all()


def test_cc_table_errors():
    g = configs.graph(1)
    sc = dict(scenarios.default_scenarios(1), cc_table=np.array([2], np.int32))
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(g, sc, 1, cc_tables=scenarios.draw_cc_tables(1, np.random.default_rng(0)))
    assert e.value.code == -2
    bad = scenarios.draw_cc_tables(1, np.random.default_rng(0))
    bad[0, 0, 3] = bad[0, 0, 2] - 1                       # max_bytes decreases
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(g, scenarios.default_scenarios(1), 1, cc_tables=bad)
    assert e.value.code == -1


# ---------------------------------------------------------------- tree-ensemble slowdown
from workloads import slowdown_forest   # noqa: E402


def _stump(values):
    """One tree: AR (type 0) takes values[0], every other type values[1]."""
    nodes = np.zeros(3, slowdown_forest.TREE_NODE_DTYPE)
    nodes[0] = (2, 1, 2, 0, 1)
    nodes[1] = (-1, 0, 0, values[0], 0)
    nodes[2] = (-1, 0, 0, values[1], 0)
    return {"nodes": nodes, "roots": np.array([0], np.int32), "base": 65536,
            "class_metrics": np.zeros((8, 4), np.int64)}


def test_forest_stump_hand_value():
    g, v = _overlap_pair(700, 1000, 1 << 30)          # the all-reduce covers [700, ...)
    sc = _scen(1)
    r = oracle.run(g, sc, 1, forest=_stump([10000, 20000]))
    assert r["finish"][0][v] == (1000 * 75536 + 32768) >> 16 == 1153
    r = oracle.run(g, sc, 1, forest=_stump([10000, 20000]), prorate=True)
    assert r["finish"][0][v] == 700 + ((300 * 75536 + 32768) >> 16) == 1046


@pytest.mark.parametrize("prorate", [False, True])
def test_forest_reproducing_the_table_equals_table_factors(prorate):
    g = configs.graph(1)
    rng = np.random.default_rng(5)
    table = rng.integers(65536, 200000, (8, 4)).astype(np.uint32)
    sc = scenarios.draw(5, rng, bw_inter=(20000, 90000), alpha=(0, 5000), jitter=(4000, 2))
    sc["slowdown_q16"] = np.broadcast_to(table, (5, 8, 4)).copy()
    for R in (1, 3):
        a = oracle.run(g, sc, R, prorate=prorate)
        b = oracle.run(g, sc, R, prorate=prorate, forest=slowdown_forest.table_forest(table))
        np.testing.assert_array_equal(a["finish"], b["finish"])
        np.testing.assert_array_equal(a["start"], b["start"])


def test_forest_factors_match_brute_force_on_random_tiny_graphs():
    rng = np.random.default_rng(654)
    checked = 0
    for trial in range(40):
        n_ranks = int(rng.integers(1, 4))
        b = Builder(n_ranks, gpus_per_node=int(rng.integers(1, 3)))
        n_coll = int(rng.integers(1, 4))
        colls = [b.collective(int(rng.integers(0, 3)), int(rng.integers(0, 256 << 10))) for _ in range(n_coll)]
        for r in range(n_ranks):
            ids = []
            order = list(rng.permutation(n_coll))
            for k in range(int(rng.integers(3, 7))):
                preds = [int(u) for u in ids if rng.random() < 0.25]
                if order and rng.random() < 0.4:
                    ids.append(b.comm(r, colls[order.pop()], stream=int(rng.integers(1, 4)), preds=preds))
                else:
                    ids.append(b.compute(r, int(rng.integers(1, 600)), stream=int(rng.integers(0, 2)),
                                         cls=int(rng.integers(0, 8)), preds=preds))
            for c in order:
                b.comm(r, colls[c], stream=int(rng.integers(1, 4)), preds=ids[-1:])
        g = b.graph()
        if len(g["op_rank"]) > 24:
            continue
        sc = _scen(1, alpha=int(rng.integers(0, 300)), bw_intra=400000, bw_inter=200000, ar_algo=int(trial % 2))
        fo = slowdown_forest.synthetic_forest(trial, n_trees=8, max_depth=6, base=70000, leaf_mean=2000,
                                              leaf_sd=6000)
        try:
            base, cost = _dur_cost(g, sc)
        except oracle.OracleError as e:
            assert e.code == -4
            continue
        for until_stable, prorate in ((False, False), (True, False), (False, True)):
            s, f, done = bruteforce.compose_variants(g, base, cost, None, 4, until_stable=until_stable,
                                                     prorate=prorate, forest=fo, knobs=(trial % 2, 400000, 200000))
            r = oracle.run(g, sc, 4, until_stable=until_stable, prorate=prorate, forest=fo)
            np.testing.assert_array_equal(r["start"][0], s)
            np.testing.assert_array_equal(r["finish"][0], f)
            assert r["refinements"][0] == done
            checked += 1
    assert checked >= 60


def test_malformed_forests_rejected():
    g = configs.graph(1)
    sc = scenarios.default_scenarios(1)
    deep = {"nodes": np.zeros(14, slowdown_forest.TREE_NODE_DTYPE), "roots": np.array([0], np.int32),
            "base": 65536, "class_metrics": np.zeros((8, 4), np.int64)}
    for i in range(13):                                   # a chain of 13 splits
        deep["nodes"][i] = (0, i + 1, i + 1, 0, 1)
    deep["nodes"][13] = (-1, 0, 0, 5, 0)
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(g, sc, 1, forest=deep)
    assert e.value.code == -1
    bad = _stump([1, 2])
    bad["nodes"][0]["feature"] = 12
    with pytest.raises(oracle.OracleError) as e:
        oracle.run(g, sc, 1, forest=bad)
    assert e.value.code == -1


def test_stored_full_digests_are_whole():
    """The stored oracle digests of the two largest workloads (full-size parity
    tests) parse into every graph and scenario they cover."""
    from tests.golden import make_full_digests as fd
    c3, c5 = fd.load(3), fd.load(5)
    assert sorted(c3) == [0] and len(c3[0][1]) == 256
    assert sorted(c5) == list(range(16)) and all(len(s) == 32 and len(d) == 32 for _, s, d in c5.values())
    for h, step, dig in list(c3.values()) + list(c5.values()):
        assert len(h) == 16 and (step > 0).all() and dig.dtype == np.uint64


def test_stored_full_digests_match_their_inputs():
    """The smallest extrapolation graph: the stored block was made from exactly these
    inputs, and the oracle reproduces its first and last scenarios."""
    from tests.golden import make_full_digests as fd
    from workloads import configs, scenarios
    g, sc = configs.graph(5, 0), configs.scenario_batch(5, 0)
    h, step, dig = fd.load(5)[0]
    assert h == fd.input_hash(g, sc)
    n = scenarios.count(sc)
    ref = oracle.run(g, scenarios.take(sc, [0, n - 1]), 1, threads=2, timelines=False, jitter_stream=[0, n - 1])
    np.testing.assert_array_equal(ref["step"], step[[0, n - 1]])
    np.testing.assert_array_equal(ref["digest"], dig[[0, n - 1]])
