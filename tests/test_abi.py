"""C-ABI checks that need no GPU: exported symbols, record layout, loader validation.

The loader validates, matches and levels a graph before it touches the
device, so every rejection path runs on the CPU; a valid graph gets as far as
hipSetDevice (ECHO_ERR_HIP when no GPU is present).
"""
from __future__ import annotations

import os
import re

import numpy as np
import pytest

from tests.tinygraph import AG, AR, P2P, Builder
from workloads import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def E():
    import paper_2412_12487_amd as E
    if not os.path.exists(E.LIB_PATH):
        from paper_2412_12487_amd import build
        build.build()
    return E


def _gpu_present():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def _load_code(E, g):
    try:
        E.Graph(g).close()
        return E.ECHO_OK
    except E.EchoError as e:
        return e.code


def test_missing_library_fails_loudly(E, tmp_path):
    """No fallback: without libecho.so the binding raises instead of computing anything."""
    from paper_2412_12487_amd import echo as binding
    saved = (binding.LIB_PATH, binding._lib)
    try:
        binding.LIB_PATH, binding._lib = str(tmp_path / "libecho.so"), None
        with pytest.raises(ImportError, match="missing"):
            binding.lib()
        with pytest.raises(ImportError, match="missing"):
            binding.Graph(configs.graph(1))
    finally:
        binding.LIB_PATH, binding._lib = saved


def test_library_exports_every_declared_symbol(E):
    header = open(os.path.join(ROOT, "include", "echo.h")).read()
    declared = set(re.findall(r"\b(echo_[a-z_]+)\s*\(", header))
    assert declared == set(E.EXPORTS)
    L = E.lib()
    for name in declared:
        assert hasattr(L, name), name


def test_scenario_record_layout_matches_header(E):
    header = open(os.path.join(ROOT, "include", "echo.h")).read()
    body = header[header.index("typedef struct {\n    int64_t alpha_ns"):]
    body = body[:body.index("} echo_scenario;")]
    for field in ("alpha_ns", "bw_intra_MBps", "bw_inter_MBps", "reduce_MBps", "jitter_seed",
                  "jitter_stream", "jitter_amp_q16", "ar_algo", "slowdown_q16"):
        assert field in body
    dt = E.SCENARIO_DTYPE
    assert dt.itemsize == 192
    assert dt.fields["slowdown_q16"][1] == 64 and dt.fields["ar_algo"][1] == 48


def _valid_code(E):
    # the sanitizer run links the loader against a host-memory stand-in of the HIP runtime
    if os.environ.get("ECHO_HOST_STUB"):
        return E.ECHO_OK
    return E.ECHO_OK if _gpu_present() else E.ECHO_ERR_HIP


def test_valid_benchmark_graph_passes_validation(E):
    assert _load_code(E, configs.graph(1)) == _valid_code(E)


def test_issue_order_mismatch_is_a_match_error(E):
    b = Builder(2)
    c1, c2 = b.collective(AR, 1024), b.collective(AR, 1024)
    b.comm(0, c1)
    b.comm(0, c2)
    b.comm(1, c2)
    b.comm(1, c1)
    assert _load_code(E, b.graph()) == E.ECHO_ERR_MATCH


def test_cross_stream_deadlock_is_a_cycle(E):
    """Each communicator issues one collective (so the matching rule holds),
    but rank 0 needs c1 before it can launch c2 and rank 1 the reverse."""
    b = Builder(2)
    c1, c2 = b.collective(AR, 1024), b.collective(AG, 1024)
    v = b.comm(0, c1, stream=1)
    w = b.compute(0, 10, preds=[v])
    b.comm(0, c2, stream=2, preds=[w])
    v = b.comm(1, c2, stream=2)
    w = b.compute(1, 10, preds=[v])
    b.comm(1, c1, stream=1, preds=[w])
    assert _load_code(E, b.graph()) == E.ECHO_ERR_CYCLE


def test_independent_streams_in_opposite_order_are_valid(E):
    b = Builder(2)
    c1, c2 = b.collective(AR, 1024), b.collective(AR, 1024)
    b.comm(0, c1, stream=1)
    b.comm(0, c2, stream=2)
    b.comm(1, c2, stream=2)
    b.comm(1, c1, stream=1)
    assert _load_code(E, b.graph()) == _valid_code(E)


@pytest.mark.parametrize("case", ["p2p3", "twice", "empty", "badpred", "dur", "bytes", "rankorder",
                                  "stream", "collid"])
def test_malformed_graphs_rejected(E, case):
    b = Builder(3)
    c = b.collective(P2P if case == "p2p3" else AR, 1024)
    if case == "empty":
        b.collective(AR, 10)
    for r in range(3):
        w = b.compute(r, 5)
        b.comm(r, c, preds=[w])
        if case == "twice" and r == 1:
            b.comm(r, c, stream=2)
    g = b.graph()
    want = E.ECHO_ERR_MATCH
    if case == "badpred":
        g["pred_idx"][0] = 3
        want = E.ECHO_ERR_ARG
    elif case == "dur":
        g["op_dur"][0] = 1 << 43
        want = E.ECHO_ERR_RANGE
    elif case == "bytes":
        g["coll_bytes"][0] = 1 << 50
        want = E.ECHO_ERR_RANGE
    elif case == "rankorder":
        g["op_rank"][0] = 2
        want = E.ECHO_ERR_ARG
    elif case == "stream":
        g["op_stream"][2] = 8
        want = E.ECHO_ERR_ARG
    elif case == "collid":
        g["op_coll"][1] = 7
        want = E.ECHO_ERR_ARG
    assert _load_code(E, g) == want


def test_generated_graphs_all_load(E):
    """Every config's generator output is acyclic and matches (config 5: the smaller graphs)."""
    for cfg, idx in [(1, 0), (2, 0), (5, 0), (5, 3), (5, 8), (5, 11)]:
        assert _load_code(E, configs.graph(cfg, idx)) == _valid_code(E), (cfg, idx)


def test_walker_width_out_of_range_is_an_argument_error(E):
    g = configs.graph(1)
    for bad in (-1, 17):
        with pytest.raises(E.EchoError) as x:
            E.Graph(g, 0, ranks_per_walker=bad)
        assert x.value.code == E.ECHO_ERR_ARG


def _replica_graph():
    from workloads import gpt1f1b
    p = dict(configs.TINY, tp=2, pp=2, dp=2, microbatches=2, seed=0)
    rg, _ = gpt1f1b.dp_replica(gpt1f1b.gpt_graph(**p, replica_invariant=True), 2, 2)
    return {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in rg.items()}


def test_replica_graph_with_group_membership_passes_validation(E):
    assert _load_code(E, _replica_graph()) == _valid_code(E)


@pytest.mark.parametrize("what", ["partial", "N_below_members", "M_zero", "MK_short", "p2p_not_two"])
def test_inconsistent_group_membership_is_an_argument_error(E, what):
    g = _replica_graph()
    c = int(np.flatnonzero(g["coll_type"] != P2P)[0])
    if what == "partial":
        g["coll_K"] = None
    elif what == "N_below_members":
        q = int(np.flatnonzero(g["coll_type"] == P2P)[0])
        g["coll_N"][q], g["coll_M"][q], g["coll_K"][q] = 1, 1, 1
    elif what == "M_zero":
        g["coll_M"][c] = 0
    elif what == "MK_short":
        g["coll_N"][c], g["coll_M"][c], g["coll_K"][c] = 9, 2, 4
    else:
        q = int(np.flatnonzero(g["coll_type"] == P2P)[0])
        g["coll_N"][q], g["coll_M"][q], g["coll_K"][q] = 4, 2, 2
    assert _load_code(E, g) == E.ECHO_ERR_ARG


def test_binding_rejects_unfit_buffers(E):
    """Output and scenario tensors are checked on the host before their pointers
    reach the library: device, contiguity, dtype and size."""
    import torch
    from paper_2412_12487_amd import echo as B
    cpu = torch.device("cpu")
    ok = torch.zeros((4, 8), dtype=torch.int64)
    assert B._device_buffer(ok, "start", cpu, 4 * 8 * 8, torch.int64).value == ok.data_ptr()
    bad = [
        (ok.t(), "contiguous"),
        (ok.to(torch.int32), "must be torch.int64"),
        (ok[:3], "needs 256"),
        ([0] * 32, "torch tensor"),
    ]
    for t, msg in bad:
        with pytest.raises(B.EchoError, match=msg):
            B._device_buffer(t, "start", cpu, 4 * 8 * 8, torch.int64)
    with pytest.raises(B.EchoError, match="the graph on"):
        B._device_buffer(ok, "start", torch.device("meta"), 8)
